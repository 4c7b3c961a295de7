// Per-unit top-k with the (score descending, index ascending) rule, output in
// source order: the device-side body of the select kernels.
//
// Scores are mapped to uint32 keys whose unsigned order is the float order
// (-0 -> +0, NaN -> 0, the lowest).  An MSB-first radix select over four
// 8-bit digits finds the keep-th largest key theta and how many keys equal to
// theta must be taken (`need`); each digit pass builds per-wave histograms in
// LDS (flat score distributions put most keys in one bin, so one shared
// histogram would serialise).  A final ordered pass flags every key above
// theta plus the first `need` keys equal to theta, and a block-wide
// exclusive scan turns the flags into output positions, which are therefore
// ascending in index.  Integer work only: exact and deterministic.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace cb {

__device__ __forceinline__ uint32_t order_key(float f) {
  uint32_t b = __float_as_uint(f);
  if ((b & 0x7f800000u) == 0x7f800000u && (b & 0x007fffffu)) return 0u;   // NaN
  if (b == 0x80000000u) b = 0u;                                            // -0 == +0
  return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}

// LDS a select_unit<NT> call needs besides the keys, in uint32 words.
template <int NT>
struct SelectLds {
  static constexpr int kWaves = NT / 64;
  // two histogram buffers [kWaves][256], scan scratch, two (prefix, need)
  static constexpr int kWords = 2 * kWaves * 256 + kWaves + 1 + 4;
};

// Exclusive scan of one value per thread over the NT-thread block; returns
// the prefix and writes the total to *total.  `scratch` holds NT/64 + 1 words.
template <int NT>
__device__ __forceinline__ uint32_t block_exclusive_scan(uint32_t v, uint32_t* scratch,
                                                          uint32_t* total) {
  constexpr int kWaves = NT / 64;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  uint32_t incl = v;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const uint32_t o = __shfl_up(incl, off);
    if (lane >= off) incl += o;
  }
  if (lane == 63) scratch[wave] = incl;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t run = 0;
    for (int w = 0; w < kWaves; ++w) {
      const uint32_t x = scratch[w];
      scratch[w] = run;
      run += x;
    }
    scratch[kWaves] = run;
  }
  __syncthreads();
  const uint32_t res = scratch[wave] + incl - v;
  *total = scratch[kWaves];
  __syncthreads();
  return res;
}

// Histogram counting with a two-entry cache of (digit, count) per thread,
// flushed by one LDS atomic per eviction instead of one per key: near-uniform
// scores put almost every key of a row into the same one or two bins (for
// example on both sides of a power of two), where per-key atomics from all 64
// lanes of a wave would serialise on one address.
struct DigitRuns {
  // d0 != d1 unless both are the empty marker, which no digit (< 256) equals.
  uint32_t d0 = 0xffffffffu, c0 = 0, d1 = 0xffffffffu, c1 = 0;
  // Counts digit d when `take`.  Hits only bump a register (no branch); a
  // miss evicts the older entry with one atomic.
  __device__ __forceinline__ void add(uint32_t* h, uint32_t d, bool take) {
    const bool h0 = d == d0, h1 = d == d1;
    c0 += (take && h0) ? 1u : 0u;
    c1 += (take && h1) ? 1u : 0u;
    if (take && !h0 && !h1) {
      if (c1) atomicAdd(&h[d1], c1);
      d1 = d0;
      c1 = c0;
      d0 = d;
      c0 = 1;
    }
  }
  __device__ __forceinline__ void flush(uint32_t* h) {
    if (c0) atomicAdd(&h[d0], c0);
    if (c1) atomicAdd(&h[d1], c1);
  }
};

// Radix-select driver shared by both key sources below.  `digit_pass`
// adds this thread's keys that match `prefix` on the digits above `shift`
// into hist[wave][digit]; `count` and `emit` walk this thread's contiguous
// span of positions for the ordered output.
template <int NT, typename DigitPass, typename Count, typename Emit>
__device__ __forceinline__ void radix_select(int keep, uint32_t* work, DigitPass&& digit_pass,
                                             Count&& count, Emit&& emit, bool packed_scan = false) {
  constexpr int kWaves = NT / 64;
  uint32_t* hists = work;                             // [2][kWaves][256]
  uint32_t* scan_scratch = work + 2 * kWaves * 256;   // kWaves + 1
  uint32_t* s_vars = scan_scratch + kWaves + 1;       // [2] x (prefix, need)
  const int tid = threadIdx.x, wave = tid >> 6;

  // Pass p counts into buffer p & 1 and clears the other one for pass p+1;
  // that buffer was last read (by wave 0) before the previous pass's final
  // barrier.  Two barriers per pass: histograms complete, digit chosen.
  for (int i = tid; i < kWaves * 256; i += NT) hists[i] = 0;
  __syncthreads();
  uint32_t prefix = 0, need = (uint32_t)keep;
  for (int pass = 0; pass < 4; ++pass) {
    const int shift = 24 - 8 * pass;
    const uint32_t hi_mask = pass == 0 ? 0u : (0xffffffffu << (shift + 8));
    uint32_t* hist = hists + (pass & 1) * (kWaves * 256);
    uint32_t* other = hists + ((pass + 1) & 1) * (kWaves * 256);
    digit_pass(hist + wave * 256, prefix, hi_mask, shift);
    if (pass < 3)
      for (int i = tid; i < kWaves * 256; i += NT) other[i] = 0;
    __syncthreads();
    if (wave == 0) {
      // The digit d with (count of digits > d) < need <= (count of digits >= d).
      // Lane j owns digits 4j..4j+3 and sums them over the waves' histograms;
      // a suffix scan over lanes counts the digits above each lane.  Exactly
      // one (lane, digit) satisfies the test.
      const int lane = tid;
      uint32_t c[4] = {0, 0, 0, 0};
#pragma unroll
      for (int w = 0; w < kWaves; ++w) {
        const uint4 v = *reinterpret_cast<const uint4*>(hist + w * 256 + 4 * lane);
        c[0] += v.x;
        c[1] += v.y;
        c[2] += v.z;
        c[3] += v.w;
      }
      const uint32_t own = c[0] + c[1] + c[2] + c[3];
      uint32_t suffix = own;
#pragma unroll
      for (int off = 1; off < 64; off <<= 1) {
        const uint32_t o = __shfl_down(suffix, off);
        if (lane + off < 64) suffix += o;
      }
      uint32_t above = suffix - own;
#pragma unroll
      for (int q = 3; q >= 0; --q) {
        if (above < need && above + c[q] >= need) {
          s_vars[2 * (pass & 1)] = prefix | ((uint32_t)(4 * lane + q) << shift);
          s_vars[2 * (pass & 1) + 1] = need - above;
        }
        above += c[q];
      }
    }
    __syncthreads();
    prefix = s_vars[2 * (pass & 1)];
    need = s_vars[2 * (pass & 1) + 1];
  }
  const uint32_t theta = prefix;

  // Ordered output: every key above theta, plus the first `need` keys equal
  // to theta in position order.
  // Block scans give each thread's first slot.  With T < 2^16 both counts
  // travel in one scan as 16-bit fields (no carry between them).
  uint32_t gt = 0, eq = 0;
  count(theta, gt, eq);
  uint32_t gt_before, eq_before, total;
  if (packed_scan) {
    const uint32_t both = block_exclusive_scan<NT>((gt << 16) | eq, scan_scratch, &total);
    gt_before = both >> 16;
    eq_before = both & 0xffffu;
  } else {
    gt_before = block_exclusive_scan<NT>(gt, scan_scratch, &total);
    eq_before = block_exclusive_scan<NT>(eq, scan_scratch, &total);
  }
  emit(theta, need, eq_before, gt_before + (eq_before < need ? eq_before : need));
}

// Words of LDS that stage a row of T scores for the register path: one pad
// word after every 32, so that threads reading their own contiguous spans
// (a stride of `per` words between lanes) spread over the banks.
__host__ __device__ constexpr int64_t select_stage_words(int64_t T) { return T + (T >> 5) + 1; }
__device__ __forceinline__ int stage_slot(int p) { return p + (p >> 5); }
// Scores per LDS chunk in the ordered passes of long rows.
constexpr int kLongChunk = 16384;

// Select `keep` of the T scores in `row` into out[0..keep), ascending.  All
// NT threads of the workgroup call it; `work` holds SelectLds<NT>::kWords
// words of LDS.  Thread i owns the contiguous positions [i*per, (i+1)*per),
// per = ceil(T / NT).
//
// With per <= KPT (`stage` then holds select_stage_words(T) words of LDS) the
// row is read once, coalesced, into LDS, and every thread copies its span into
// registers; the selected positions are gathered in LDS and written out
// coalesced.  Otherwise every pass re-reads the scores from global memory
// (L2): the digit passes read the row coalesced; the ordered passes walk
// each thread's span, either eight keys at a time from L2 (`stage` unused) or,
// with STAGE_LONG (`stage` holds select_stage_words(kLongChunk) words), from
// chunks of kLongChunk scores staged through LDS with coalesced loads.
template <int NT, int KPT, bool STAGE_LONG = false>
__device__ __forceinline__ void select_unit(const float* __restrict__ row, int T, int keep,
                                            int32_t* __restrict__ out, uint32_t* work,
                                            uint32_t* stage) {
  const int tid = threadIdx.x;
  const int per = (T + NT - 1) / NT;
  const int lo = tid * per < T ? tid * per : T;
  const int hi = lo + per < T ? lo + per : T;
  const int n = hi - lo;

  // Loads first, unconditionally (addresses clamped into the row), so that
  // they are all in flight together; conversion and masking afterwards.
  auto at = [&](int j) { return row + (lo + j < T ? lo + j : T - 1); };
  if (per <= KPT) {
    {
      uint32_t v[KPT];
#pragma unroll
      for (int j = 0; j < KPT; ++j) {
        const int p = tid + j * NT;
        v[j] = __float_as_uint(row[p < T ? p : T - 1]);
      }
#pragma unroll
      for (int j = 0; j < KPT; ++j) {
        const int p = tid + j * NT;
        if (p < T) stage[stage_slot(p)] = v[j];
      }
    }
    __syncthreads();
    uint32_t key[KPT];
#pragma unroll
    for (int j = 0; j < KPT; ++j)
      key[j] = j < n ? order_key(__uint_as_float(stage[stage_slot(lo + j < T ? lo + j : T - 1)]))
                     : 0u;
    radix_select<NT>(
        keep, work,
        [&](uint32_t* h, uint32_t prefix, uint32_t hi_mask, int shift) {
          DigitRuns runs;
#pragma unroll
          for (int j = 0; j < KPT; ++j)
            runs.add(h, (key[j] >> shift) & 255u, j < n && (key[j] & hi_mask) == prefix);
          runs.flush(h);
        },
        [&](uint32_t theta, uint32_t& gt, uint32_t& eq) {
#pragma unroll
          for (int j = 0; j < KPT; ++j) {
            gt += j < n && key[j] > theta;
            eq += j < n && key[j] == theta;
          }
        },
        [&](uint32_t theta, uint32_t need, uint32_t eq_seen, uint32_t pos) {
          // The staged scores are dead: the slots hold the output instead.
#pragma unroll
          for (int j = 0; j < KPT; ++j) {
            if (j >= n) continue;
            bool take = key[j] > theta;
            if (key[j] == theta) {
              take = eq_seen < need;
              ++eq_seen;
            }
            if (take && pos < (uint32_t)keep) stage[pos++] = (uint32_t)(lo + j);
          }
        },
        /*packed_scan=*/true);
    __syncthreads();
    for (int i = tid; i < keep; i += NT) out[i] = (int32_t)stage[i];
    return;
  }

  // Long rows.  The digit passes read the row coalesced, in 16-byte loads
  // when rows are 16-byte aligned (T % 4 == 0), since a histogram does not
  // depend on the order of the keys; the ordered count and output passes
  // walk each thread's span, eight keys at a time.
  constexpr int B = 8;
  const bool vec = (T & 3) == 0;
  auto span_batch = [&](int j0, uint32_t (&kb)[B]) {
    if (vec && (per & 3) == 0 && lo + j0 + B <= T) {
      const uint4 a = *reinterpret_cast<const uint4*>(row + lo + j0);
      const uint4 b = *reinterpret_cast<const uint4*>(row + lo + j0 + 4);
      kb[0] = a.x; kb[1] = a.y; kb[2] = a.z; kb[3] = a.w;
      kb[4] = b.x; kb[5] = b.y; kb[6] = b.z; kb[7] = b.w;
    } else {
#pragma unroll
      for (int j = 0; j < B; ++j) kb[j] = __float_as_uint(*at(j0 + j));
    }
#pragma unroll
    for (int j = 0; j < B; ++j) kb[j] = j0 + j < n ? order_key(__uint_as_float(kb[j])) : 0u;
  };
  // Ordered passes over LDS chunks: all threads stage scores [c0, c1)
  // coalesced, then each thread visits its span's part [a0, a1) of the chunk.
  // Every thread runs the same number of chunks, so the barriers are uniform.
  auto for_chunks = [&](auto&& body) {
    for (int c0 = 0; c0 < T; c0 += kLongChunk) {
      const int c1 = c0 + kLongChunk < T ? c0 + kLongChunk : T;
      __syncthreads();   // the previous chunk's readers are done
      if (vec) {
        for (int p = c0 + 4 * tid; p < c1; p += 4 * NT) {   // c0, c1 multiples of 4
          const uint4 v = *reinterpret_cast<const uint4*>(row + p);
          const int q = p - c0;
          stage[stage_slot(q)] = v.x;
          stage[stage_slot(q + 1)] = v.y;
          stage[stage_slot(q + 2)] = v.z;
          stage[stage_slot(q + 3)] = v.w;
        }
      } else {
        for (int p = c0 + tid; p < c1; p += NT) stage[stage_slot(p - c0)] = __float_as_uint(row[p]);
      }
      __syncthreads();
      body(lo > c0 ? lo : c0, hi < c1 ? hi : c1, c0);
    }
  };
  radix_select<NT>(
      keep, work,
      [&](uint32_t* h, uint32_t prefix, uint32_t hi_mask, int shift) {
        DigitRuns runs;
        auto add = [&](uint32_t raw, bool valid) {
          const uint32_t key = order_key(__uint_as_float(raw));
          runs.add(h, (key >> shift) & 255u, valid && (key & hi_mask) == prefix);
        };
        if (vec) {
          const uint4* r4 = reinterpret_cast<const uint4*>(row);
          const int n4 = T >> 2;
          for (int i = tid; i < n4; i += 4 * NT) {
            uint4 v[4];
            bool ok[4];
#pragma unroll
            for (int k = 0; k < 4; ++k) {
              ok[k] = i + k * NT < n4;
              v[k] = r4[ok[k] ? i + k * NT : i];
            }
#pragma unroll
            for (int k = 0; k < 4; ++k) {
              add(v[k].x, ok[k]);
              add(v[k].y, ok[k]);
              add(v[k].z, ok[k]);
              add(v[k].w, ok[k]);
            }
          }
        } else {
          for (int p = tid; p < T; p += NT) add(__float_as_uint(row[p]), true);
        }
        runs.flush(h);
      },
      [&](uint32_t theta, uint32_t& gt, uint32_t& eq) {
        if constexpr (STAGE_LONG) {
          for_chunks([&](int a0, int a1, int c0) {
            for (int p = a0; p < a1; ++p) {
              const uint32_t key = order_key(__uint_as_float(stage[stage_slot(p - c0)]));
              gt += key > theta;
              eq += key == theta;
            }
          });
          return;
        }
        for (int j0 = 0; j0 < n; j0 += B) {
          uint32_t kb[B];
          span_batch(j0, kb);
#pragma unroll
          for (int j = 0; j < B; ++j) {
            gt += j0 + j < n && kb[j] > theta;
            eq += j0 + j < n && kb[j] == theta;
          }
        }
      },
      [&](uint32_t theta, uint32_t need, uint32_t eq_seen, uint32_t pos) {
        if constexpr (STAGE_LONG) {
          for_chunks([&](int a0, int a1, int c0) {
            for (int p = a0; p < a1; ++p) {
              const uint32_t key = order_key(__uint_as_float(stage[stage_slot(p - c0)]));
              bool take = key > theta;
              if (key == theta) {
                take = eq_seen < need;
                ++eq_seen;
              }
              if (take && pos < (uint32_t)keep) out[pos++] = p;
            }
          });
          return;
        }
        for (int j0 = 0; j0 < n; j0 += B) {
          uint32_t kb[B];
          span_batch(j0, kb);
#pragma unroll
          for (int j = 0; j < B; ++j) {
            if (j0 + j >= n) continue;
            bool take = kb[j] > theta;
            if (kb[j] == theta) {
              take = eq_seen < need;
              ++eq_seen;
            }
            if (take && pos < (uint32_t)keep) out[pos++] = lo + j0 + j;
          }
        }
      });
}

}  // namespace cb
