// Query-attention importance of sender positions (gfx950 / CDNA4).
//
// For one unit (sender s, layer l, KV head g) the query rows are the m tokens
// of every query head in the group: R = G*m rows of D values, and the logits
// are S = scale * Q K^T (R x T).  Importance is the column sum of the row
// softmax, I[t] = sum_r exp(S[r,t] - lse_r).  Because every row carries its
// own normaliser, no column sum can start before the whole row is known, so
// K is traversed twice:
//
//   pass 1 (stats):  per row and per T-chunk, the running max and sum of
//                    exp2 in log2 units; the last workgroup of a unit to
//                    finish folds the chunks in fixed order into lse2 (log2
//                    of the row normaliser).  No waiting, no float atomics.
//   pass 2 (reduce): recompute the logits, add exp2(x - lse2) over the rows.
//
// Both passes run the contraction on bf16 (fp32 for fp32 inputs) MFMA with
// fp32 accumulation.  Each wavefront keeps 64 query rows in registers for the
// whole kernel; 64-token K tiles are staged through LDS (double-buffered,
// XOR-swizzled 16-byte chunks so B-fragment reads are bank-conflict free)
// and shared by every wave of the workgroup.  The contraction index is
// permuted consistently for Q and K: lane group j (lanes 16j..16j+15) holds a
// contiguous quarter of each row, so every fragment is one 16-byte load.
// The scale is applied in fp32 to the accumulator (folded with log2 e), never
// to bf16 operands.
//
// Workgroups are mapped XCD-contiguously: blockIdx b runs on XCD b % 8, and
// consecutive work items (the chunks of one unit) go to the same XCD so the
// unit's query block is fetched into one L2 only.
#include <math.h>

#include "kernels.h"

namespace cb {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kMaxChunkTokens = 512;

template <int ESZ, int D>
struct Geo {
  static constexpr int kRowBytes = D * ESZ;
  static constexpr int kChunks = kRowBytes / 16;          // 16-byte chunks per K row
  static constexpr int kSegs = kChunks / 4;               // chunks per lane group
  static constexpr int kSwz = kChunks >= 16 ? 15 : kChunks - 1;
  static constexpr int kTileBytes = kTileTokens * kRowBytes;
  static constexpr int kTileChunks = kTileTokens * kChunks;
};

__device__ __forceinline__ int swz_offset(int row, int c, int row_bytes, int swz) {
  return row * row_bytes + ((c ^ (row & swz)) << 4);
}

// One 16-byte segment of the contraction for a 16x16 output block.
template <int ESZ>
__device__ __forceinline__ void mfma_seg(const u32x4& a, const u32x4& b, f32x4& acc);

template <>
__device__ __forceinline__ void mfma_seg<2>(const u32x4& a, const u32x4& b, f32x4& acc) {
  acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                __builtin_bit_cast(bf16x8, b), acc, 0, 0, 0);
}

template <>
__device__ __forceinline__ void mfma_seg<4>(const u32x4& a, const u32x4& b, f32x4& acc) {
#pragma unroll
  for (int e = 0; e < 4; ++e)
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a[e]), __uint_as_float(b[e]),
                                               acc, 0, 0, 0);
}

// Combine two (max, sum) pairs of exp2 partial sums.
__device__ __forceinline__ void lse_merge(float& m, float& z, float mo, float zo) {
  const float mn = fmaxf(m, mo);
  const float ms = (mn == -INFINITY) ? 0.f : mn;
  z = z * __builtin_amdgcn_exp2f(m - ms) + zo * __builtin_amdgcn_exp2f(mo - ms);
  m = mn;
}

template <int ESZ, int D, int W, bool PASS2>
__global__ __launch_bounds__(W * 64) void score_kernel(ScoreArgs a) {
  using Gm = Geo<ESZ, D>;
  constexpr int kPer = Gm::kTileChunks / (W * 64);   // staged chunks per thread per tile
  constexpr int kBatch = kPer < 8 ? kPer : 8;
  static_assert(Gm::kTileChunks % (W * 64) == 0, "tile must split evenly");
  static_assert(kPer % kBatch == 0, "batches must split evenly");

  __shared__ __attribute__((aligned(16))) unsigned char ktile[2][Gm::kTileBytes];
  __shared__ float imp_lds[PASS2 ? W * kMaxChunkTokens : 1];
  __shared__ int s_last;

  const int item = (blockIdx.x & 7) * a.per_xcd + (blockIdx.x >> 3);
  if (item >= a.items) return;
  const int chunk = item % a.chunks;
  const int rest = item / a.chunks;
  const int rg = rest % a.row_groups;
  const int u = a.unit0 + rest / a.row_groups;
  const int layer = (u / a.Hkv) % a.L;
  const int kvh = u % a.Hkv;

  const int tid = threadIdx.x;
  const int wave = tid >> 6;
  const int lane = tid & 63;
  const int lg = lane >> 4;   // lane group: which quarter of the contraction / which 4 rows
  const int lc = lane & 15;   // lane column: token within a 16-token block / Q row

  const unsigned char* qb = static_cast<const unsigned char*>(a.q) +
                            (size_t)((layer * a.Hq + kvh * a.G) * a.m) * Gm::kRowBytes;
  const unsigned char* kb = static_cast<const unsigned char*>(a.k) +
                            (size_t)u * (size_t)a.T * Gm::kRowBytes;

  const int wrow0 = rg * kRowsPerGroup + wave * kRowsPerWave;
  const bool wave_active = wrow0 < a.R;

  // ---- query rows of this wave, resident in registers -----------------------
  u32x4 qf[4][Gm::kSegs];
#pragma unroll
  for (int rb = 0; rb < 4; ++rb) {
    const int row = wrow0 + rb * 16 + lc;
    const u32x4* src = reinterpret_cast<const u32x4*>(qb + (size_t)row * Gm::kRowBytes) +
                       lg * Gm::kSegs;
#pragma unroll
    for (int sg = 0; sg < Gm::kSegs; ++sg) qf[rb][sg] = (row < a.R) ? src[sg] : u32x4{0, 0, 0, 0};
  }

  // ---- per-lane row state -----------------------------------------------------
  // Rows held by this lane: wrow0 + rb*16 + 4*lg + i.
  float st_m[4][4], st_z[4][4];   // pass 1: running max / sum (log2 units)
  float row_l2[4][4];             // pass 2: lse2 of the row (+inf for padding rows)
#pragma unroll
  for (int rb = 0; rb < 4; ++rb)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      st_m[rb][i] = -INFINITY;
      st_z[rb][i] = 0.f;
      if (PASS2) {
        const int row = wrow0 + rb * 16 + 4 * lg + i;
        row_l2[rb][i] = (row < a.R) ? a.lse2[(size_t)u * a.R + row] : INFINITY;
      }
    }

  const int64_t t_begin = (int64_t)chunk * a.chunk_tokens;
  const int64_t t_end = (t_begin + a.chunk_tokens < a.T) ? t_begin + a.chunk_tokens : a.T;
  const int ntiles = (int)((t_end - t_begin + kTileTokens - 1) / kTileTokens);

  // ---- K tile staging: global -> registers -> LDS (swizzled) ------------------
  u32x4 stage[kBatch];
  auto stage_load = [&](int tile, int batch) {
#pragma unroll
    for (int j = 0; j < kBatch; ++j) {
      const int cidx = (batch * kBatch + j) * (W * 64) + tid;
      const int row = cidx / Gm::kChunks;
      const int c = cidx % Gm::kChunks;
      const int64_t t = t_begin + (int64_t)tile * kTileTokens + row;
      stage[j] = (t < t_end)
                     ? *reinterpret_cast<const u32x4*>(kb + (size_t)t * Gm::kRowBytes + c * 16)
                     : u32x4{0, 0, 0, 0};
    }
  };
  auto stage_store = [&](int buf, int batch) {
#pragma unroll
    for (int j = 0; j < kBatch; ++j) {
      const int cidx = (batch * kBatch + j) * (W * 64) + tid;
      const int row = cidx / Gm::kChunks;
      const int c = cidx % Gm::kChunks;
      *reinterpret_cast<u32x4*>(&ktile[buf][swz_offset(row, c, Gm::kRowBytes, Gm::kSwz)]) =
          stage[j];
    }
  };

  for (int b = 0; b < kPer / kBatch; ++b) {
    stage_load(0, b);
    stage_store(0, b);
  }
  __syncthreads();

  for (int tile = 0; tile < ntiles; ++tile) {
    const int buf = tile & 1;
    const bool has_next = tile + 1 < ntiles;
    if (has_next) stage_load(tile + 1, 0);

    if (wave_active) {
      f32x4 acc[4][4];
#pragma unroll
      for (int rb = 0; rb < 4; ++rb)
#pragma unroll
        for (int tb = 0; tb < 4; ++tb) acc[rb][tb] = f32x4{0.f, 0.f, 0.f, 0.f};

#pragma unroll
      for (int sg = 0; sg < Gm::kSegs; ++sg) {
        u32x4 kf[4];
#pragma unroll
        for (int tb = 0; tb < 4; ++tb) {
          const int row = tb * 16 + lc;
          kf[tb] = *reinterpret_cast<const u32x4*>(
              &ktile[buf][swz_offset(row, lg * Gm::kSegs + sg, Gm::kRowBytes, Gm::kSwz)]);
        }
#pragma unroll
        for (int rb = 0; rb < 4; ++rb)
#pragma unroll
          for (int tb = 0; tb < 4; ++tb) mfma_seg<ESZ>(qf[rb][sg], kf[tb], acc[rb][tb]);
      }

      // Token of column tb for this lane; padding tokens are masked.
      const int64_t tok0 = t_begin + (int64_t)tile * kTileTokens + lc;
      bool valid[4];
#pragma unroll
      for (int tb = 0; tb < 4; ++tb) valid[tb] = tok0 + tb * 16 < t_end;

      if (!PASS2) {
#pragma unroll
        for (int rb = 0; rb < 4; ++rb)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            float raw[4];
#pragma unroll
            for (int tb = 0; tb < 4; ++tb) raw[tb] = valid[tb] ? acc[rb][tb][i] : -INFINITY;
            const float tmax = fmaxf(fmaxf(raw[0], raw[1]), fmaxf(raw[2], raw[3])) * a.c2;
            const float mn = fmaxf(st_m[rb][i], tmax);
            const float ms = (mn == -INFINITY) ? 0.f : mn;
            float z = st_z[rb][i] * __builtin_amdgcn_exp2f(st_m[rb][i] - ms);
#pragma unroll
            for (int tb = 0; tb < 4; ++tb) z += __builtin_amdgcn_exp2f(__builtin_fmaf(raw[tb], a.c2, -ms));
            st_z[rb][i] = z;
            st_m[rb][i] = mn;
          }
      } else {
        const int tloc0 = tile * kTileTokens;
#pragma unroll
        for (int tb = 0; tb < 4; ++tb) {
          float s = 0.f;
#pragma unroll
          for (int rb = 0; rb < 4; ++rb)
#pragma unroll
            for (int i = 0; i < 4; ++i)
              s += __builtin_amdgcn_exp2f(__builtin_fmaf(acc[rb][tb][i], a.c2, -row_l2[rb][i]));
          s += __shfl_xor(s, 16);
          s += __shfl_xor(s, 32);
          if (lg == 0) imp_lds[wave * kMaxChunkTokens + tloc0 + tb * 16 + lc] = s;
        }
      }
    } else if (PASS2) {
      const int tloc0 = tile * kTileTokens;
      if (lg == 0)
#pragma unroll
        for (int tb = 0; tb < 4; ++tb) imp_lds[wave * kMaxChunkTokens + tloc0 + tb * 16 + lc] = 0.f;
    }

    if (has_next) {
      stage_store(buf ^ 1, 0);
      for (int b = 1; b < kPer / kBatch; ++b) {
        stage_load(tile + 1, b);
        stage_store(buf ^ 1, b);
      }
    }
    __syncthreads();
  }

  if (PASS2) {
    // Column sums over the waves, in wave order, then out to global memory.
    float* out = (a.row_groups > 1)
                     ? a.imp_partial + ((size_t)rg * a.units_total + u) * (size_t)a.T
                     : a.importance + (size_t)u * (size_t)a.T;
    const int n = (int)(t_end - t_begin);
    for (int t = tid; t < n; t += W * 64) {
      float s = 0.f;
#pragma unroll
      for (int w = 0; w < W; ++w) s += imp_lds[w * kMaxChunkTokens + t];
      out[t_begin + t] = s;
    }
    return;
  }

  // ---- pass 1: fold the 16 lane columns, publish per-chunk row statistics ----
#pragma unroll
  for (int rb = 0; rb < 4; ++rb)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float m = st_m[rb][i], z = st_z[rb][i];
#pragma unroll
      for (int off = 1; off < 16; off <<= 1) {
        const float mo = __shfl_xor(m, off);
        const float zo = __shfl_xor(z, off);
        lse_merge(m, z, mo, zo);
      }
      const int row = wrow0 + rb * 16 + 4 * lg + i;
      if (lc == 0 && row < a.R)
        a.partial[((size_t)u * a.chunks + chunk) * a.R + row] = make_float2(m, z);
    }

  // The last workgroup of this unit to arrive folds all chunks, in chunk order.
  __threadfence();
  __syncthreads();
  if (tid == 0) {
    const int prev = atomicAdd(&a.counters[u], 1);
    s_last = (prev == a.chunks * a.row_groups - 1);
  }
  __syncthreads();
  if (!s_last) return;
  __threadfence();
  for (int row = tid; row < a.R; row += W * 64) {
    float m = -INFINITY, z = 0.f;
    for (int c = 0; c < a.chunks; ++c) {
      const float2 p = a.partial[((size_t)u * a.chunks + c) * a.R + row];
      lse_merge(m, z, p.x, p.y);
    }
    const float l2 = m + __log2f(z);
    a.lse2[(size_t)u * a.R + row] = l2;
    if (a.row_lse) a.row_lse[(size_t)u * a.R + row] = l2 * 0.69314718055994530942f;
  }
  if (tid == 0) a.counters[u] = 0;
}

__global__ void zero_ints(int* p, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = 0;
}

// importance[u][t] = sum over row groups, in order.
__global__ void rowgroup_sum(const float* __restrict__ part, float* __restrict__ out,
                             int row_groups, int64_t per_group, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  float s = 0.f;
  for (int r = 0; r < row_groups; ++r) s += part[r * per_group + i];
  out[i] = s;
}

template <int ESZ, int D, bool PASS2>
hipError_t launch_w(const ScorePlan& p, const ScoreArgs& a, int waves, hipStream_t s) {
  const dim3 grid(8 * a.per_xcd);
  switch (waves) {
    case 1: score_kernel<ESZ, D, 1, PASS2><<<grid, 64, 0, s>>>(a); break;
    case 2: score_kernel<ESZ, D, 2, PASS2><<<grid, 128, 0, s>>>(a); break;
    case 4: score_kernel<ESZ, D, 4, PASS2><<<grid, 256, 0, s>>>(a); break;
    default: score_kernel<ESZ, D, 8, PASS2><<<grid, 512, 0, s>>>(a); break;
  }
  return hipGetLastError();
}

template <bool PASS2>
hipError_t launch_typed(const ScorePlan& p, const ScoreArgs& a, int waves, hipStream_t s) {
  if (p.dtype == 1)
    return p.D == 128 ? launch_w<2, 128, PASS2>(p, a, waves, s) : launch_w<2, 64, PASS2>(p, a, waves, s);
  return p.D == 128 ? launch_w<4, 128, PASS2>(p, a, waves, s) : launch_w<4, 64, PASS2>(p, a, waves, s);
}

}  // namespace

bool make_score_plan(int L, int Hq, int Hkv, int D, int m, int S, int64_t T, int dtype,
                     float scale, ScorePlan* p) {
  if (L < 1 || Hq < 1 || Hkv < 1 || m < 1 || S < 1 || T < 1) return false;
  if (Hq % Hkv != 0 || (D != 64 && D != 128) || T >= ((int64_t)1 << 31)) return false;
  if (!(scale >= 0.f) || !isfinite(scale)) return false;
  const int G = Hq / Hkv;
  if ((int64_t)G * m > kMaxRows) return false;
  p->T = T;
  p->L = L; p->Hq = Hq; p->Hkv = Hkv; p->G = G; p->m = m; p->R = G * m; p->D = D;
  p->dtype = dtype;
  p->units = S * L * Hkv;
  p->chunk_tokens = kMaxChunkTokens;
  p->chunks = (int)((T + p->chunk_tokens - 1) / p->chunk_tokens);
  p->row_groups = (p->R + kRowsPerGroup - 1) / kRowsPerGroup;
  const double esz = dtype == 1 ? 2.0 : 4.0;
  const double unit_k_bytes = (double)T * D * esz;
  const double budget = 96.0 * 1024 * 1024;
  int per = (int)(budget / unit_k_bytes);
  if (per < 1) per = 1;
  if (per > p->units) per = p->units;
  const int groups = (p->units + per - 1) / per;
  p->units_per_launch = (p->units + groups - 1) / groups;
  const float sc = scale > 0.f ? scale : (float)(1.0 / sqrt((double)D));
  p->c2 = (float)((double)sc * 1.4426950408889634);
  auto al = [](size_t x) { return (x + 255) & ~(size_t)255; };
  size_t off = 0;
  p->off_partial = off; off = al(off + (size_t)p->units * p->chunks * p->R * sizeof(float2));
  p->off_lse2 = off; off = al(off + (size_t)p->units * p->R * sizeof(float));
  p->off_counters = off; off = al(off + (size_t)p->units * sizeof(int));
  p->off_imp_partial = off;
  if (p->row_groups > 1) off = al(off + (size_t)p->row_groups * p->units * (size_t)T * sizeof(float));
  p->total_bytes = off;
  return true;
}

hipError_t launch_score_init(const ScorePlan& p, int* counters, hipStream_t s) {
  zero_ints<<<(p.units + 255) / 256, 256, 0, s>>>(counters, p.units);
  return hipGetLastError();
}

hipError_t launch_score_pass(const ScorePlan& p, const ScoreArgs& a, bool pass2, hipStream_t s) {
  const int rows0 = p.R < kRowsPerGroup ? p.R : kRowsPerGroup;
  const int need = (rows0 + kRowsPerWave - 1) / kRowsPerWave;
  const int waves = need <= 1 ? 1 : need <= 2 ? 2 : need <= 4 ? 4 : 8;
  return pass2 ? launch_typed<true>(p, a, waves, s) : launch_typed<false>(p, a, waves, s);
}

hipError_t launch_rowgroup_sum(const ScorePlan& p, const ScoreArgs& a, hipStream_t s) {
  const int64_t n = (int64_t)a.nunits * a.T;
  const int64_t per_group = (int64_t)a.units_total * a.T;
  // Partials for unit u and row group r live at imp_partial[r][u][:].
  const float* part = a.imp_partial + (size_t)a.unit0 * a.T;
  float* out = a.importance + (size_t)a.unit0 * a.T;
  rowgroup_sum<<<(unsigned)((n + 255) / 256), 256, 0, s>>>(part, out, p.row_groups, per_group, n);
  return hipGetLastError();
}

}  // namespace cb
