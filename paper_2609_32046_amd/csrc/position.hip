// The paper's position-level selector after the score kernel (gfx950):
//
//   position_terms   per sender and position, over every unit of the sender
//                    (fixed order): the layer sum of the per-layer query mean
//                    (Q before pooling), the correction numerator (from the
//                    score kernel's pooled per-token terms) and denominator
//                    (Pool_7 of each unit's mean weight, raised to p), then
//                    C_{p,t}; fp64 accumulation.
//   position_output  Q_t = Pool_7 of the layer sum, S_t = Q_t * C_t^alpha.
//   spans_kernel     the span rule, one workgroup per sender.
//   gather_rows      continuous rows at the selected positions.
//
// Appendix C.1 (mean-query-attention and CacheBack-correction equations),
// Appendix D.2 (general score), Appendix C.2 (budgets and span selection),
// Appendix C.3 and section 3.1.2 (continuous-row messages).
#include <math.h>

#include "kernels.h"
#include "position.h"

namespace cb {
namespace {

constexpr int kPool = 3;          // Pool_7: positions t-3 .. t+3
constexpr int kTermWaves = 8;     // waves sharing one block of positions
constexpr int kTermLanes = 64;    // positions per block
constexpr int kTermBatch = 4;     // units whose loads are in flight together

struct TermArgs {
  const float* importance;   // [U][T]
  const float* numer;        // [U][T]
  double* qpre;              // [S][T]
  double* corr;              // [S][T]
  int64_t T;
  int LH;                    // units per sender
  int pow_mode;
  double p, inv_mG, num_scale, q_scale;
};

// Block: 8 waves x 64 positions; wave w takes the sender's units w, w+8, ...
__global__ __launch_bounds__(kTermWaves * kTermLanes) void position_terms(TermArgs a) {
  __shared__ double part[3][kTermWaves][kTermLanes];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int s = blockIdx.y;
  const int64_t t = (int64_t)blockIdx.x * kTermLanes + lane;
  const bool in = t < a.T;
  const int64_t lo = t - kPool < 0 ? 0 : t - kPool;
  const int64_t hi = t + kPool < a.T - 1 ? t + kPool : a.T - 1;
  double q = 0.0, num = 0.0, den = 0.0;
  if (in) {
    // Units wave, wave + 8, ... in that order; the loads of kTermBatch units
    // are issued before any of them is used (the loop is latency-bound).
    // The window's 7 loads are clamped into [lo, hi], which repeats an end
    // value near the sequence ends and leaves the maximum unchanged.
    for (int j0 = wave; j0 < a.LH; j0 += kTermBatch * kTermWaves) {
      float win[kTermBatch][2 * kPool + 1], nu[kTermBatch];
#pragma unroll
      for (int b = 0; b < kTermBatch; ++b) {
        const int j = j0 + b * kTermWaves;
        if (j >= a.LH) continue;
        const size_t u = (size_t)s * a.LH + j;
        const float* row = a.importance + u * (size_t)a.T;
#pragma unroll
        for (int d = -kPool; d <= kPool; ++d) {
          const int64_t x = t + d < lo ? lo : (t + d > hi ? hi : t + d);
          win[b][d + kPool] = row[x];
        }
        nu[b] = a.numer[u * (size_t)a.T + t];
      }
#pragma unroll
      for (int b = 0; b < kTermBatch; ++b) {
        if (j0 + b * kTermWaves >= a.LH) continue;
        float pooled = win[b][0];
#pragma unroll
        for (int d = 1; d <= 2 * kPool; ++d) pooled = fmaxf(pooled, win[b][d]);
        const double x = (double)pooled * a.inv_mG;   // Pool_7 of the unit's token mean
        q += (double)win[b][kPool];
        if (a.pow_mode == kPowMax) {
          num = fmax(num, (double)nu[b]);
          den = fmax(den, x);
        } else {
          num += (double)nu[b];
          den += a.pow_mode == kPowSquare ? x * x : pow(x, a.p);
        }
      }
    }
  }
  part[0][wave][lane] = q;
  part[1][wave][lane] = num;
  part[2][wave][lane] = den;
  __syncthreads();
  if (wave != 0 || !in) return;
  q = num = den = 0.0;
  for (int w = 0; w < kTermWaves; ++w) {
    q += part[0][w][lane];
    if (a.pow_mode == kPowMax) {
      num = fmax(num, part[1][w][lane]);
      den = fmax(den, part[2][w][lane]);
    } else {
      num += part[1][w][lane];
      den += part[2][w][lane];
    }
  }
  num *= a.num_scale;
  double c;
  if (num == 0.0 && den == 0.0) {
    c = 1.0;
  } else if (a.pow_mode == kPowMax) {
    c = num / den;
  } else if (a.pow_mode == kPowSquare) {
    c = num / den;
  } else {
    c = pow(num / den, 1.0 / (a.p - 1.0));
  }
  // C >= 1 in exact arithmetic (mean of pooled powers >= power of pooled
  // mean); fp32 underflow of the smallest per-token terms can only lower
  // the numerator, so the bound is restored here.
  if (!(c >= 1.0)) c = 1.0;
  a.qpre[(size_t)s * a.T + t] = q * a.q_scale;
  a.corr[(size_t)s * a.T + t] = c;
}

__global__ void position_output(const double* __restrict__ qpre, const double* __restrict__ corr,
                                int64_t T, int64_t n, double alpha, float* __restrict__ score,
                                float* __restrict__ qscore, float* __restrict__ corr_out) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const int64_t s = i / T, t = i - s * T;
  const int64_t lo = t - kPool < 0 ? 0 : t - kPool;
  const int64_t hi = t + kPool < T - 1 ? t + kPool : T - 1;
  const double* row = qpre + s * T;
  double qv = row[lo];
  for (int64_t d = lo + 1; d <= hi; ++d) qv = fmax(qv, row[d]);
  const double c = corr[i];
  const double w = alpha == 0.0 ? 1.0 : alpha == 2.0 ? c * c : pow(c, alpha);
  score[i] = (float)(qv * w);
  if (qscore) qscore[i] = (float)qv;
  if (corr_out) corr_out[i] = (float)c;
}

// ---- span rule ----------------------------------------------------------------

constexpr int kSpanThreads = 1024;
constexpr int kSpanWaves = kSpanThreads / 64;

// Order-preserving map of a double onto uint64 (larger key, larger value;
// -0 == +0, NaN lowest).
__device__ __forceinline__ uint64_t order_key64(double x) {
  if (x != x) return 0ull;
  if (x == 0.0) x = 0.0;
  const uint64_t b = (uint64_t)__double_as_longlong(x);
  return (b >> 63) ? ~b : (b | 0x8000000000000000ull);
}

__device__ __forceinline__ bool forced(int64_t t, int64_t T, int64_t n_latent) {
  return t == 0 || t >= T - n_latent;
}

// Positions of span j not forced.
__device__ __forceinline__ int64_t fresh(int64_t j, int64_t T, int width, int64_t n_latent) {
  const int64_t lo = j * width, hi = lo + width < T ? lo + width : T;
  const int64_t f_lo = T - n_latent;   // forced tail [f_lo, T)
  int64_t n = hi - lo;
  const int64_t a = lo > f_lo ? lo : f_lo;
  if (hi > a) n -= hi - a;
  if (lo == 0 && f_lo > 0) n -= 1;     // position 0 (not already in the tail)
  return n;
}

// Block-wide exclusive scan of one uint64 per thread; returns the prefix,
// writes the total.
__device__ uint64_t scan64(uint64_t v, uint64_t* scratch, uint64_t* total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  uint64_t incl = v;
  for (int off = 1; off < 64; off <<= 1) {
    const uint64_t o = __shfl_up(incl, off);
    if (lane >= off) incl += o;
  }
  if (lane == 63) scratch[wave] = incl;
  __syncthreads();
  if (wave == 0) {
    const uint64_t x = lane < kSpanWaves ? scratch[lane] : 0;
    uint64_t run = x;
    for (int off = 1; off < kSpanWaves; off <<= 1) {
      const uint64_t o = __shfl_up(run, off);
      if (lane >= off) run += o;
    }
    if (lane < kSpanWaves) scratch[lane] = run - x;
    if (lane == kSpanWaves - 1) scratch[kSpanWaves] = run;
  }
  __syncthreads();
  const uint64_t res = scratch[wave] + incl - v;
  *total = scratch[kSpanWaves];
  __syncthreads();
  return res;
}

struct SpanArgs {
  const float* score;   // [S][T]
  uint64_t* keys;       // [S][nspan] workspace, used when nspan > kLdsSpans
  int32_t* idx;         // [S][out_count]
  int64_t T, nspan, n_latent, rem, out_count;
  int width;
};

// Span keys of up to kLdsSpans spans stay in LDS; more go to the workspace.
constexpr int kLdsSpans = 4096;
// Histogram copies (one per pair of waves); a bin holds the spans with that
// digit in its high half and their unforced positions in its low half.
constexpr int kHistCopies = kSpanWaves / 2;

// One workgroup per sender.  LK: the keys live in LDS.
template <bool LK>
__global__ __launch_bounds__(kSpanThreads) void spans_kernel(SpanArgs a) {
  __shared__ uint64_t hist[kHistCopies][256];
  __shared__ uint64_t s_keys[LK ? kLdsSpans : 1];
  __shared__ uint64_t scratch[kSpanWaves + 1];
  __shared__ float fred[kSpanWaves];
  __shared__ uint64_t s_prefix, s_need;
  __shared__ uint32_t s_holders;
  __shared__ int64_t s_cut, s_cut_take;
  __shared__ uint64_t s_mask;   // positions of the cut span taken (bit i: lo + i)
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int64_t T = a.T, nspan = a.nspan;
  const int width = a.width;
  const float* sc = a.score + (size_t)blockIdx.x * T;
  uint64_t* keys;
  if constexpr (LK)
    keys = s_keys;
  else
    keys = a.keys + (size_t)blockIdx.x * nspan;
  int32_t* out = a.idx + (size_t)blockIdx.x * a.out_count;

  // 1-2. span means (fp64 sums in position order over the fp32 scores) with
  //      the maximum score in place of position 0's.  The spans cover every
  //      position, so one read gives both the maximum and the other spans'
  //      sums; span 0 is summed once the maximum is known.
  float mx = -INFINITY;
  for (int64_t j = tid; j < nspan; j += kSpanThreads) {
    const int64_t lo = j * width, hi = lo + width < T ? lo + width : T;
    double sum = 0.0;
#pragma unroll 8
    for (int64_t t = lo; t < hi; ++t) {
      const float v = sc[t];
      mx = fmaxf(mx, v);
      sum += (double)v;
    }
    if (j > 0) keys[j] = order_key64(sum / (double)(hi - lo));
  }
  for (int off = 32; off > 0; off >>= 1) mx = fmaxf(mx, __shfl_xor(mx, off));
  if (lane == 0) fred[wave] = mx;
  __syncthreads();
  mx = fred[0];
  for (int w = 1; w < kSpanWaves; ++w) mx = fmaxf(mx, fred[w]);
  if (tid == 0) {
    const int64_t hi = width < T ? width : T;
    double sum = 0.0;
    for (int64_t t = 0; t < hi; ++t) sum += (double)(t == 0 ? mx : sc[t]);
    keys[0] = order_key64(sum / (double)hi);
  }
  if constexpr (!LK) __threadfence_block();
  __syncthreads();

  // 3. the cut: the first span in rank order (mean descending, index
  //    ascending) at which the running count of unforced positions passes
  //    `rem`.  Radix passes over the 64-bit keys with histograms of those
  //    counts narrow it to one key theta (ending early once one span is left
  //    with the chosen prefix); an ordered pass over the spans holding theta
  //    finds the span itself.  Counts fit 32 bits: they sum to at most T.
  const int64_t n_forced = a.n_latent + 1 < T ? a.n_latent + 1 : T;   // {0} and the tail
  const bool take_all = a.rem >= T - n_forced;
  uint64_t prefix = 0;
  uint32_t need = (uint32_t)a.rem;
  if (!take_all && a.rem > 0) {
    for (int pass = 0; pass < 8; ++pass) {
      const int shift = 56 - 8 * pass;
      const uint64_t hi_mask = pass == 0 ? 0ull : (~0ull << (shift + 8));
      for (int i = tid; i < kHistCopies * 256; i += kSpanThreads) (&hist[0][0])[i] = 0;
      __syncthreads();
      for (int64_t j = tid; j < nspan; j += kSpanThreads) {
        const uint64_t k = keys[j];
        if ((k & hi_mask) == prefix)
          atomicAdd((unsigned long long*)&hist[wave >> 1][(k >> shift) & 255],
                    (1ull << 32) | (unsigned long long)fresh(j, T, width, a.n_latent));
      }
      __syncthreads();
      if (wave == 0) {
        // lane owns digits 4*lane .. 4*lane+3; digits above d rank before it
        uint32_t c[4], n[4];
        for (int q = 0; q < 4; ++q) {
          uint64_t b = 0;
          for (int w = 0; w < kHistCopies; ++w) b += hist[w][4 * lane + q];
          c[q] = (uint32_t)b;
          n[q] = (uint32_t)(b >> 32);
        }
        const uint32_t own = c[0] + c[1] + c[2] + c[3];
        uint32_t suffix = own;
        for (int off = 1; off < 64; off <<= 1) {
          const uint32_t o = __shfl_down(suffix, off);
          if (lane + off < 64) suffix += o;
        }
        uint32_t above = suffix - own;
        for (int q = 3; q >= 0; --q) {
          if (above <= need && above + c[q] > need) {
            s_prefix = prefix | ((uint64_t)(4 * lane + q) << shift);
            s_need = need - above;
            s_holders = n[q];
          }
          above += c[q];
        }
      }
      __syncthreads();
      prefix = s_prefix;
      need = (uint32_t)s_need;
      // Usually a few passes leave one span with the chosen prefix: its key
      // is theta, and the later passes would keep `need` as it is.
      if (pass < 7 && s_holders == 1) {
        const uint64_t fixed = ~0ull << shift;
        uint64_t found = 0;
        bool hit = false;
        for (int64_t j = tid; j < nspan; j += kSpanThreads)
          if ((keys[j] & fixed) == prefix) {
            found = keys[j];
            hit = true;
          }
        __syncthreads();   // every thread has read s_prefix
        if (hit) s_prefix = found;
        __syncthreads();
        prefix = s_prefix;
        break;
      }
    }
  }
  const uint64_t theta = prefix;

  // 4. the cut span among the spans with key theta, in index order
  const int64_t per = (nspan + kSpanThreads - 1) / kSpanThreads;
  const int64_t j0 = tid * per < nspan ? tid * per : nspan;
  const int64_t j1 = j0 + per < nspan ? j0 + per : nspan;
  if (tid == 0) {
    s_cut = -1;
    s_cut_take = 0;
    s_mask = 0;
  }
  __syncthreads();
  if (!take_all && a.rem > 0) {
    uint64_t mine = 0;
    for (int64_t j = j0; j < j1; ++j)
      if (keys[j] == theta) mine += fresh(j, T, width, a.n_latent);
    uint64_t total;
    uint64_t before = scan64(mine, scratch, &total);
    for (int64_t j = j0; j < j1; ++j) {
      if (keys[j] != theta) continue;
      const int64_t f = fresh(j, T, width, a.n_latent);
      if (before <= need && before + f > need) {   // exactly one span of the block
        s_cut = j;
        s_cut_take = (int64_t)(need - before);
        break;
      }
      before += f;
    }
    __syncthreads();
    // the interval of the cut span: its unselected positions nearest its top
    // position (right first at equal distance), clipped to the span.  The
    // top is the first position holding the span's largest score (NaNs
    // skipped, unless the span's first score is NaN: then that position);
    // wave 0 finds it with one lane per position.
    if (wave == 0 && s_cut >= 0 && s_cut_take > 0) {
      const int64_t lo = s_cut * width, hi = lo + width < T ? lo + width : T;
      const int64_t t = lo + lane;
      float v = -INFINITY;
      if (t < hi) {
        v = t == 0 ? mx : sc[t];
        if (v != v) v = lane == 0 ? INFINITY : -INFINITY;
      }
      int at = lane;
      for (int off = 1; off < 64; off <<= 1) {
        const float ov = __shfl_xor(v, off);
        const int oat = __shfl_xor(at, off);
        if (ov > v || (ov == v && oat < at)) {
          v = ov;
          at = oat;
        }
      }
      if (lane == 0) {
        const int64_t top = lo + at;
        uint64_t mask = 0;
        int64_t taken = 0;
        for (int64_t d = 0; taken < s_cut_take && d < width; ++d) {
          const int64_t r = top + d, l = top - d;
          if (r < hi && !forced(r, T, a.n_latent)) {
            mask |= 1ull << (r - lo);
            ++taken;
          }
          if (d > 0 && taken < s_cut_take && l >= lo && !forced(l, T, a.n_latent)) {
            mask |= 1ull << (l - lo);
            ++taken;
          }
        }
        s_mask = mask;
      }
    }
  }
  __syncthreads();
  const int64_t cut = s_cut;
  const uint64_t mask = s_mask;
  // position t = j*width + off
  auto selected = [&](int64_t t, int64_t j, int off) -> bool {
    if (forced(t, T, a.n_latent) || take_all) return true;
    if (a.rem == 0) return false;
    const uint64_t k = keys[j];
    if (k > theta) return true;
    if (k < theta) return false;
    if (j < cut) return true;
    if (j > cut) return false;
    return (mask >> off) & 1ull;
  };

  // 5. selected positions in source order
  const int64_t tper = (T + kSpanThreads - 1) / kSpanThreads;
  const int64_t t0 = tid * tper < T ? tid * tper : T;
  const int64_t t1 = t0 + tper < T ? t0 + tper : T;
  const int64_t js = (int64_t)((uint32_t)t0 / (uint32_t)width);   // T < 2^31
  const int offs = (int)(t0 - js * width);
  uint64_t cnt = 0;
  for (int64_t t = t0, j = js, off = offs; t < t1; ++t) {
    cnt += selected(t, j, (int)off);
    if (++off == width) off = 0, ++j;
  }
  uint64_t total;
  uint64_t pos = scan64(cnt, scratch, &total);
  for (int64_t t = t0, j = js, off = offs; t < t1; ++t) {
    if (selected(t, j, (int)off) && pos < (uint64_t)a.out_count) out[pos++] = (int32_t)t;
    if (++off == width) off = 0, ++j;
  }
}

// ---- continuous rows --------------------------------------------------------------

// out[r] = rows[s][idx[r]] for r = s*count + j; an index outside [0, T)
// gives a zero row.  `lanes` bytes per thread and pass (16 or 4).  I: the
// index type of the element and row divisions (32 bits when n fits).
template <typename V, typename I>
__global__ __launch_bounds__(256) void gather_rows_kernel(const unsigned char* __restrict__ rows,
                                                          const int32_t* __restrict__ idx,
                                                          unsigned char* __restrict__ out,
                                                          int64_t T, int64_t count, int64_t vecs,
                                                          int64_t n) {
  constexpr int kUnroll = 4;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i0 < n;
       i0 += stride * kUnroll) {
    V v[kUnroll];
    int64_t dst[kUnroll];
#pragma unroll
    for (int k = 0; k < kUnroll; ++k) {
      const int64_t i = i0 + k * stride;
      const int64_t r = i < n ? (int64_t)((I)i / (I)vecs) : 0, c = i < n ? i - r * vecs : 0;
      const int64_t s = (int64_t)((I)r / (I)count);
      const int64_t t = idx[r];
      const bool ok = i < n && t >= 0 && t < T;
      dst[k] = i < n ? i : -1;
      // out-of-range entries read row 0 of the sender (valid memory) and store zeros
      const V x = reinterpret_cast<const V*>(rows)[(s * T + (ok ? t : 0)) * vecs + c];
      v[k] = ok ? x : V{};
    }
#pragma unroll
    for (int k = 0; k < kUnroll; ++k)
      if (dst[k] >= 0) __builtin_nontemporal_store(v[k], reinterpret_cast<V*>(out) + dst[k]);
  }
}

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

int compute_units_here() {
  int dev = 0, n = 256;
  if (hipGetDevice(&dev) != hipSuccess) return 256;
  if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
    n = 256;
  return n;
}

}  // namespace

hipError_t launch_position_finish(const PositionFinish& f, hipStream_t s) {
  TermArgs a;
  a.importance = f.importance;
  a.numer = f.numer;
  a.qpre = f.qpre;
  a.corr = f.corr64;
  a.T = f.T;
  a.LH = f.LH;
  a.pow_mode = f.pow_mode;
  a.p = f.p;
  a.inv_mG = 1.0 / ((double)f.m * f.G);
  a.num_scale = f.num_scale;
  a.q_scale = 1.0 / ((double)f.m * f.Hq);
  const dim3 grid((unsigned)((f.T + kTermLanes - 1) / kTermLanes), (unsigned)f.S);
  position_terms<<<grid, kTermWaves * kTermLanes, 0, s>>>(a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int64_t n = (int64_t)f.S * f.T;
  position_output<<<(unsigned)((n + 255) / 256), 256, 0, s>>>(f.qpre, f.corr64, f.T, n, f.alpha,
                                                              f.score, f.qscore, f.corr);
  return hipGetLastError();
}

hipError_t launch_spans(const float* score, int64_t S, int64_t T, int width, int64_t n_latent,
                        int64_t rem, int64_t out_count, uint64_t* keys, int32_t* idx,
                        hipStream_t s) {
  SpanArgs a;
  a.score = score;
  a.keys = keys;
  a.idx = idx;
  a.T = T;
  a.nspan = (T + width - 1) / width;
  a.n_latent = n_latent;
  a.rem = rem;
  a.out_count = out_count;
  a.width = width;
  if (a.nspan <= kLdsSpans)
    spans_kernel<true><<<(unsigned)S, kSpanThreads, 0, s>>>(a);
  else
    spans_kernel<false><<<(unsigned)S, kSpanThreads, 0, s>>>(a);
  return hipGetLastError();
}

hipError_t launch_gather_rows(const void* rows, int64_t S, int64_t T, int64_t row_bytes,
                              const int32_t* idx, int64_t count, void* out, hipStream_t s) {
  const int64_t total = S * count;
  if (total == 0) return hipSuccess;
  const int64_t blocks_cap = (int64_t)compute_units_here() * 8;
  if (row_bytes % 16 == 0) {
    const int64_t vecs = row_bytes / 16, n = total * vecs;
    const int64_t blocks = (n + 255) / 256 < blocks_cap ? (n + 255) / 256 : blocks_cap;
    if (n + blocks * 256 * 4 < ((int64_t)1 << 32))
      gather_rows_kernel<u32x4, uint32_t><<<(unsigned)blocks, 256, 0, s>>>(
          static_cast<const unsigned char*>(rows), idx, static_cast<unsigned char*>(out), T,
          count, vecs, n);
    else
      gather_rows_kernel<u32x4, uint64_t><<<(unsigned)blocks, 256, 0, s>>>(
          static_cast<const unsigned char*>(rows), idx, static_cast<unsigned char*>(out), T,
          count, vecs, n);
  } else {
    const int64_t vecs = row_bytes / 4, n = total * vecs;
    const int64_t blocks = (n + 255) / 256 < blocks_cap ? (n + 255) / 256 : blocks_cap;
    if (n + blocks * 256 * 4 < ((int64_t)1 << 32))
      gather_rows_kernel<uint32_t, uint32_t><<<(unsigned)blocks, 256, 0, s>>>(
          static_cast<const unsigned char*>(rows), idx, static_cast<unsigned char*>(out), T,
          count, vecs, n);
    else
      gather_rows_kernel<uint32_t, uint64_t><<<(unsigned)blocks, 256, 0, s>>>(
          static_cast<const unsigned char*>(rows), idx, static_cast<unsigned char*>(out), T,
          count, vecs, n);
  }
  return hipGetLastError();
}

}  // namespace cb
