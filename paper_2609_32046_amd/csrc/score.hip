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
//                    exp2 in log2 units, written to the workspace.
//   pass 2 (reduce): fold the chunk statistics of the unit's rows in fixed
//                    chunk order into lse2 (log2 of the row normaliser), then
//                    recompute the logits and add exp2(x - lse2) over the
//                    rows.  No float atomics, no inter-workgroup waiting.
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

// LDS ring depth: as many 64-token K tiles as fit the workgroup's share of
// the 160 KiB LDS at two waves per SIMD (8/W workgroups per CU), between 2
// and 4, after the other LDS arrays.
template <int ESZ, int D, int W>
struct Stages {
  static constexpr int kTile = kTileTokens * D * ESZ;
  static constexpr int kOther = W * (kMaxChunkTokens + kRowsPerWave) * 4;
  static constexpr int kBudget = (W >= 2 ? 160 * 1024 * W / 8 : 40 * 1024) - kOther;
  static constexpr int kFit = kBudget / kTile;
  static constexpr int value = kFit < 2 ? 2 : (kFit > 4 ? 4 : kFit);
};

// s_waitcnt immediates (gfx9 encoding: vmcnt[3:0] and [15:14], expcnt[6:4],
// lgkmcnt[11:8]); counters not named are left at their maximum.
constexpr int vmcnt_imm(int n) { return (n & 15) | ((n >> 4) << 14) | (7 << 4) | (15 << 8); }
constexpr int kWaitVmcnt0 = vmcnt_imm(0);
constexpr int lgkmcnt_imm(int n) { return 15 | (3 << 14) | (7 << 4) | ((n & 15) << 8); }

// Wait until at most `later` tiles of kPer loads each are still in flight.
template <int kPer, int kStages>
__device__ __forceinline__ void wait_tiles(int later) {
  static_assert((kStages - 2) * kPer <= 63, "vmcnt holds at most 63");
  if (kStages >= 4 && later >= 2) {
    __builtin_amdgcn_s_waitcnt(vmcnt_imm(2 * kPer));
  } else if (kStages >= 3 && later >= 1) {
    __builtin_amdgcn_s_waitcnt(vmcnt_imm(kPer));
  } else {
    __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
  }
}

// One 16-byte-per-lane load from global memory straight into LDS: lane i
// writes lds_base + 16*i.  Issued through asm so that the compiler's own
// wait-count insertion, which cannot tell the ring's buffers apart and would
// drain every in-flight tile before each LDS read, stays out of the ring;
// completion is tracked explicitly with wait_tiles() below.
__device__ __forceinline__ void load_lds16(const void* gptr, uint32_t lds_base) {
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off"
               :
               : "v"(gptr), "s"(lds_base)
               : "memory", "m0");
}

// LDS offset of a shared-memory pointer (the low 32 bits of its flat address).
__device__ __forceinline__ uint32_t lds_offset(const void* p) {
  return (uint32_t)reinterpret_cast<uintptr_t>(p);
}

// Workgroup barrier that waits for this wave's LDS operations only; loads in
// flight to later ring stages stay in flight.
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_s_waitcnt(lgkmcnt_imm(0));
  __builtin_amdgcn_s_barrier();
}

// Sum of v over the four lanes l, l^16, l^32, l^48 (the four lane groups
// that hold the same token column), returned in every one of them.  Two
// cross-row swaps instead of LDS-routed shuffles; the addition order is the
// same in every lane, so all four hold bitwise-equal sums.
__device__ __forceinline__ float sum_lane_groups(float v) {
  const auto p = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v),
                                                  false, false);
  const float s = __uint_as_float(p[0]) + __uint_as_float(p[1]);
  const auto q = __builtin_amdgcn_permlane32_swap(__float_as_uint(s), __float_as_uint(s),
                                                  false, false);
  return __uint_as_float(q[0]) + __uint_as_float(q[1]);
}

// Scheduler hint: interleave one MFMA with `valu` VALU instructions, n times.
template <int N, int VALU>
__device__ __forceinline__ void interleave_mfma_valu() {
#pragma unroll
  for (int i = 0; i < N; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);      // MFMA
    __builtin_amdgcn_sched_group_barrier(0x002, VALU, 0);   // VALU
  }
}

// Combine two (max, sum) pairs of exp2 partial sums.
__device__ __forceinline__ void lse_merge(float& m, float& z, float mo, float zo) {
  const float mn = fmaxf(m, mo);
  const float ms = (mn == -INFINITY) ? 0.f : mn;
  z = z * __builtin_amdgcn_exp2f(m - ms) + zo * __builtin_amdgcn_exp2f(mo - ms);
  m = mn;
}

template <int ESZ, int D, int W, bool PASS2>
// bf16: two waves per SIMD (<= 256 registers per lane) so one wave's MFMAs
// overlap another's exp/VALU epilogue.
__global__ __launch_bounds__(W * 64, ESZ == 2 ? 2 : 1) void score_kernel(ScoreArgs a) {
  using Gm = Geo<ESZ, D>;
  constexpr int kPer = Gm::kTileChunks / (W * 64);   // 16-byte loads per thread per tile
  constexpr int kStages = Stages<ESZ, D, W>::value;  // K tiles resident/in flight in LDS
  static_assert(Gm::kTileChunks % (W * 64) == 0, "tile must split evenly");

  __shared__ __attribute__((aligned(16))) unsigned char ktile[kStages][Gm::kTileBytes];
  __shared__ float imp_lds[PASS2 ? W * kMaxChunkTokens : 1];
  __shared__ float lse_lds[PASS2 ? W * kRowsPerWave : 1];

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

  // ---- pass 2 prologue: fold the chunk statistics of this row group ---------
  // One thread per row; chunks are folded in ascending order, eight loads in
  // flight, so every workgroup of the unit derives bitwise-identical lse2.
  if (PASS2) {
    const int row_base = rg * kRowsPerGroup;
    const int nrows = (a.R - row_base < W * kRowsPerWave) ? a.R - row_base : W * kRowsPerWave;
    if (tid < nrows) {
      const int row = row_base + tid;
      const float2* p = a.partial + (size_t)u * a.chunks * a.R + row;
      float m = -INFINITY, z = 0.f;
      int c = 0;
      for (; c + 8 <= a.chunks; c += 8) {
        float2 v[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) v[j] = p[(size_t)(c + j) * a.R];
#pragma unroll
        for (int j = 0; j < 8; ++j) lse_merge(m, z, v[j].x, v[j].y);
      }
      for (; c < a.chunks; ++c) {
        const float2 v = p[(size_t)c * a.R];
        lse_merge(m, z, v.x, v.y);
      }
      const float l2 = m + __log2f(z);
      lse_lds[tid] = l2;
      if (chunk == 0 && a.row_lse)
        a.row_lse[(size_t)u * a.R + row] = l2 * 0.69314718055994530942f;
    }
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
      row_l2[rb][i] = INFINITY;
    }

  const int64_t t_begin = (int64_t)chunk * a.chunk_tokens;
  const int64_t t_end = (t_begin + a.chunk_tokens < a.T) ? t_begin + a.chunk_tokens : a.T;
  const int ntiles = (int)((t_end - t_begin + kTileTokens - 1) / kTileTokens);

  // ---- K tiles: direct global -> LDS loads into a kStages-deep ring -----------
  // Lane `tid` owns LDS slot j*(W*64) + tid of a tile and fetches the K chunk
  // whose swizzled position that slot is: every load instruction of a wave
  // writes one contiguous KiB of LDS, and the swizzle stays the one the
  // B-fragment reads expect.  Rows past the chunk end are clamped to its last
  // row (always valid memory); their logits are masked or never stored.
  int koff[kPer];   // byte offset of this lane's chunk inside a tile's rows
  int krow[kPer];   // its row inside the tile
#pragma unroll
  for (int j = 0; j < kPer; ++j) {
    const int slot = j * (W * 64) + tid;
    krow[j] = slot / Gm::kChunks;
    const int c = (slot % Gm::kChunks) ^ (krow[j] & Gm::kSwz);
    koff[j] = krow[j] * Gm::kRowBytes + c * 16;
  }
  const uint32_t lds_ring = lds_offset(&ktile[0][0]) + wave * 64 * 16;
  auto issue_tile = [&](int tile, int buf) {
    const int64_t tbase = t_begin + (int64_t)tile * kTileTokens;
    const unsigned char* src = kb + (size_t)tbase * Gm::kRowBytes;
    const uint32_t dst = lds_ring + buf * Gm::kTileBytes;
    if (tbase + kTileTokens <= t_end) {
#pragma unroll
      for (int j = 0; j < kPer; ++j)
        load_lds16(src + koff[j], __builtin_amdgcn_readfirstlane(dst + j * (W * 64) * 16));
    } else {
      const int last = (int)(t_end - 1 - tbase);
#pragma unroll
      for (int j = 0; j < kPer; ++j) {
        const int over = krow[j] > last ? (krow[j] - last) * Gm::kRowBytes : 0;
        load_lds16(src + koff[j] - over, __builtin_amdgcn_readfirstlane(dst + j * (W * 64) * 16));
      }
    }
  };

  // One 16-token column block: this wave's 64 rows against tokens
  // tb*16..tb*16+15 of the tile, as four 16x16 MFMA blocks (one per row
  // block) over the kSegs contraction segments.
  auto load_block = [&](const unsigned char* kt, int tb, u32x4 (&kf)[Gm::kSegs]) {
    const int row = tb * 16 + lc;
#pragma unroll
    for (int sg = 0; sg < Gm::kSegs; ++sg)
      kf[sg] = *reinterpret_cast<const u32x4*>(
          kt + swz_offset(row, lg * Gm::kSegs + sg, Gm::kRowBytes, Gm::kSwz));
  };
  auto mfma_block = [&](const u32x4 (&kf)[Gm::kSegs], f32x4 (&acc)[4]) {
#pragma unroll
    for (int rb = 0; rb < 4; ++rb) acc[rb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int sg = 0; sg < Gm::kSegs; ++sg)
#pragma unroll
      for (int rb = 0; rb < 4; ++rb) mfma_seg<ESZ>(qf[rb][sg], kf[sg], acc[rb]);
  };
  auto column_block = [&](const unsigned char* kt, int tb, f32x4 (&acc)[4]) {
    u32x4 kf[Gm::kSegs];
    load_block(kt, tb, kf);
    mfma_block(kf, acc);
  };
  // Software pipeline over the four column blocks of a tile: the LDS reads
  // and MFMAs of block tb+1 are issued ahead of block tb's exp epilogue, and
  // the scheduler is asked to interleave them, so the matrix unit and the
  // VALU work at the same time within one wave.
  constexpr int kMfmaPerBlock = 4 * Gm::kSegs * (ESZ == 4 ? 4 : 1);
  auto pipelined_tile = [&](const unsigned char* kt, auto&& epilogue) {
    u32x4 kf[2][Gm::kSegs];
    f32x4 acc[2][4];
    load_block(kt, 0, kf[0]);
    mfma_block(kf[0], acc[0]);
#pragma unroll
    for (int tb = 0; tb < 4; ++tb) {
      const int cur = tb & 1;
      if (tb < 3) {
        load_block(kt, tb + 1, kf[cur ^ 1]);
        mfma_block(kf[cur ^ 1], acc[cur ^ 1]);
      }
      epilogue(tb, acc[cur]);
      if (tb < 3) interleave_mfma_valu<kMfmaPerBlock, 3>();
    }
  };

  // Everything issued so far (query rows, chunk statistics) must land before
  // the ring's vmcnt bookkeeping starts.
  __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
  for (int j = 0; j < kStages - 1 && j < ntiles; ++j) issue_tile(j, j);

  for (int tile = 0; tile < ntiles; ++tile) {
    const int buf = tile % kStages;
    // Wait for this tile's loads (later tiles may stay in flight), then make
    // every wave's loads visible; the barrier also retires the previous
    // tile's buffer, which the next issue overwrites.
    const int later = ((ntiles - 1 < tile + kStages - 2) ? ntiles - 1 : tile + kStages - 2) - tile;
    wait_tiles<kPer, kStages>(later);
    lds_barrier();
    if (tile + kStages - 1 < ntiles) issue_tile(tile + kStages - 1, (tile + kStages - 1) % kStages);
    if (PASS2 && tile == 0) {
#pragma unroll
      for (int rb = 0; rb < 4; ++rb)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int row = wrow0 + rb * 16 + 4 * lg + i;
          row_l2[rb][i] =
              (row < a.R) ? lse_lds[wave * kRowsPerWave + rb * 16 + 4 * lg + i] : INFINITY;
        }
    }
    if (!wave_active) {
      if (PASS2 && lg == 0)
#pragma unroll
        for (int tb = 0; tb < 4; ++tb)
          imp_lds[wave * kMaxChunkTokens + tile * kTileTokens + tb * 16 + lc] = 0.f;
      continue;
    }
    const unsigned char* kt = &ktile[buf][0];
    const int64_t tok0 = t_begin + (int64_t)tile * kTileTokens;
    const bool full = tok0 + kTileTokens <= t_end;

    if (PASS2) {
      // importance contribution: column sums of exp2(x - lse2) over the rows
      float* dst = &imp_lds[wave * kMaxChunkTokens + tile * kTileTokens + lc];
      pipelined_tile(kt, [&](int tb, const f32x4(&acc)[4]) {
        float part[4];
#pragma unroll
        for (int rb = 0; rb < 4; ++rb) {
          float p = 0.f;
#pragma unroll
          for (int i = 0; i < 4; ++i)
            p += __builtin_amdgcn_exp2f(__builtin_fmaf(acc[rb][i], a.c2, -row_l2[rb][i]));
          part[rb] = p;
        }
        const float sum = sum_lane_groups((part[0] + part[1]) + (part[2] + part[3]));
        if (lg == 0) dst[tb * 16] = sum;
      });
      continue;
    }

    // pass 1, fast path (full tile, running maxima seeded by an earlier
    // tile): add exp2(x - m) with m unchanged.  A row whose sum passes 2^100
    // (a logit far above its earlier maximum) sends the whole tile to the
    // slow path, from the sums saved before it; below that, fp32 keeps full
    // relative precision, so leaving m behind costs nothing.
    bool redo = !(full && tile > 0);
    if (!redo) {
      float zp[4][4];
#pragma unroll
      for (int rb = 0; rb < 4; ++rb)
#pragma unroll
        for (int i = 0; i < 4; ++i) zp[rb][i] = st_z[rb][i];
      pipelined_tile(kt, [&](int, const f32x4(&acc)[4]) {
#pragma unroll
        for (int rb = 0; rb < 4; ++rb)
#pragma unroll
          for (int i = 0; i < 4; ++i)
            st_z[rb][i] += __builtin_amdgcn_exp2f(__builtin_fmaf(acc[rb][i], a.c2, -st_m[rb][i]));
      });
      bool over = false;
#pragma unroll
      for (int rb = 0; rb < 4; ++rb)
#pragma unroll
        for (int i = 0; i < 4; ++i) over |= !(st_z[rb][i] <= 0x1p100f);
      if (__any(over)) {
        redo = true;
#pragma unroll
        for (int rb = 0; rb < 4; ++rb)
#pragma unroll
          for (int i = 0; i < 4; ++i) st_z[rb][i] = zp[rb][i];
      }
    }
    if (redo) {
      // Slow path: first tile of the chunk, ragged tail, or a new large
      // maximum.  Online max / rescale per column block, padding masked.
#pragma unroll
      for (int tb = 0; tb < 4; ++tb) {
        f32x4 acc[4];
        column_block(kt, tb, acc);
        const bool valid = tok0 + tb * 16 + lc < t_end;
#pragma unroll
        for (int rb = 0; rb < 4; ++rb)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const float x = valid ? acc[rb][i] * a.c2 : -INFINITY;
            const float mn = fmaxf(st_m[rb][i], x);
            const float ms = (mn == -INFINITY) ? 0.f : mn;
            st_z[rb][i] = st_z[rb][i] * __builtin_amdgcn_exp2f(st_m[rb][i] - ms) +
                          __builtin_amdgcn_exp2f(x - ms);
            st_m[rb][i] = mn;
          }
      }
    }
  }
  __syncthreads();

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
  // Units per launch: about 64 MiB of K, rounded down to fill whole rounds
  // of two resident workgroups per CU where that is possible.
  const double esz = dtype == 1 ? 2.0 : 4.0;
  const double unit_k_bytes = (double)T * D * esz;
  const double budget = 64.0 * 1024 * 1024;
  int per = (int)(budget / unit_k_bytes);
  if (per < 1) per = 1;
  const int wg_per_unit = p->chunks * p->row_groups;
  const int round_units = 512 / wg_per_unit;
  if (round_units > 1 && per > round_units) per -= per % round_units;
  if (per > p->units) per = p->units;
  p->units_per_launch = per;
  const float sc = scale > 0.f ? scale : (float)(1.0 / sqrt((double)D));
  p->c2 = (float)((double)sc * 1.4426950408889634);
  auto al = [](size_t x) { return (x + 255) & ~(size_t)255; };
  size_t off = 0;
  p->off_partial = off; off = al(off + (size_t)p->units * p->chunks * p->R * sizeof(float2));
  p->off_imp_partial = off;
  if (p->row_groups > 1) off = al(off + (size_t)p->row_groups * p->units * (size_t)T * sizeof(float));
  p->total_bytes = off;
  return true;
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
