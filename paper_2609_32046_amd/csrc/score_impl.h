#pragma once
// Receiver-conditioned importance of sender positions as one persistent
// kernel (gfx950 / CDNA4): device code and launch templates, included by
// the per-dtype translation units score_*.hip.
//
// For one unit (sender s, layer l, KV head g) the query rows are the m tokens
// of every query head in the group: R = G*m rows of D values, and the logits
// are S = scale * Q K^T (R x T).  Importance is the column sum of the row
// softmax, I[t] = sum_r exp(S[r,t] - lse_r).  Because every row carries its
// own normaliser, no column sum can start before the whole row is known, so
// K is traversed twice, chunk by chunk (1024 to 4096 positions):
//
//   P1 (stats):   per row and chunk, the max and sum of exp2 in log2 units.
//   P2 (reduce):  fold the unit's chunk statistics in fixed chunk order into
//                 lse2 (log2 of the row normaliser), recompute the logits and
//                 add exp2(x - lse2) over the rows.
//
// Scheduling.  Every P1 and P2 item of every unit sits in one ordered list
// (WorkList in kernels.h); resident workgroups take items from a device
// queue (one atomic counter) until the list is exhausted.  A P2 item waits
// until all P1 items of its unit (and row group) are counted in, on a
// per-unit counter.  The list places P2 of unit u lag steps after its P1, so
// by the time a P2 item is taken its statistics are normally complete and
// the unit's K is still in the 256 MB Infinity Cache; the whole stage is one
// launch with no idle boundaries between unit groups.  Dependencies always
// precede their dependants in the list and are taken only by running
// workgroups, so the waits always end whatever the number of resident
// workgroups; each wait is still bounded (PersistArgs::spin_limit) and a
// timeout raises an error flag, poisons the item's output (NaN importance)
// and stops every later wait.
//
// The chunk statistics that P1 workgroups hand to P2 workgroups inside the
// launch are written with device-scope atomic stores and read with
// device-scope atomic loads; each writer waits for its stores to complete
// before the workgroup counts itself in with a relaxed atomic add, so no
// cache-wide release/acquire maintenance is needed.
//
// Score items run the contraction on bf16 (fp32 for fp32 inputs) MFMA with
// fp32 accumulation.  Each wavefront holds 16*RB query rows in registers
// (RB = 4 row blocks; 5 when a unit has 257 to 320 rows, so that four
// waves cover it instead of five of eight);
// K tiles of 64 or 128 positions are staged through an LDS ring (XOR-swizzled 16-byte
// chunks so B-fragment reads are bank-conflict free) and shared by every
// wave of the workgroup.  The contraction index is permuted consistently for
// Q and K: lane group j (lanes 16j..16j+15) holds a contiguous quarter of
// each row, so every fragment is one 16-byte load.  The scale is applied in
// fp32 to the accumulator (folded with log2 e), never to bf16 operands.
#include <math.h>

#include <algorithm>
#include <mutex>

#include "kernels.h"

namespace cb {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));


// K positions per LDS tile: 128 for bf16 workgroups of four or more waves
// (half the per-tile barrier, wait and address work per position, two
// 32 KiB ring stages), else kTileTokens.
template <int ESZ, int W>
struct TileTokens {
  static constexpr int value = (ESZ == 2 && W >= 4) ? 2 * kTileTokens : kTileTokens;
};

template <int ESZ, int D, int TT>
struct Geo {
  static constexpr int kRowBytes = D * ESZ;
  static constexpr int kChunks = kRowBytes / 16;          // 16-byte chunks per K row
  static constexpr int kSegs = kChunks / 4;               // chunks per lane group
  static constexpr int kSwz = kChunks >= 16 ? 15 : kChunks - 1;
  static constexpr int kTileBytes = TT * kRowBytes;
  static constexpr int kTileChunks = TT * kChunks;
  static constexpr int kBlocks = TT / 16;                 // 16-position column blocks per tile
};

// K-tile slot layout: thread `tid` of an NT-thread workgroup owns slots
// j*NT + tid, j < per, of a tile of rows of `chunks` 16-byte chunks stored
// swizzled (chunk c of row r at position c ^ (r & swz)).  When NT rows of
// chunks span a multiple of swz+1 whole rows, slot j of a thread is its slot
// 0 moved down j*NT/chunks rows: one per-lane offset serves every load of a
// tile.  Checked exhaustively at compile time where it is used.
struct SlotGeo {
  int row, off;
};
constexpr SlotGeo slot_geo(int slot, int chunks, int swz, int row_bytes) {
  const int r = slot / chunks;
  const int c = (slot % chunks) ^ (r & swz);
  return SlotGeo{r, r * row_bytes + c * 16};
}
constexpr bool slots_linear(int nt, int per, int chunks, int swz, int row_bytes) {
  if (nt % chunks != 0 || ((nt / chunks) & swz) != 0) return false;
  for (int tid = 0; tid < nt; ++tid)
    for (int j = 0; j < per; ++j) {
      const SlotGeo g0 = slot_geo(tid, chunks, swz, row_bytes);
      const SlotGeo gj = slot_geo(j * nt + tid, chunks, swz, row_bytes);
      if (gj.row != g0.row + j * (nt / chunks) || gj.off != g0.off + j * (nt / chunks) * row_bytes)
        return false;
    }
  return true;
}

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

// LDS ring depth: as many K tiles as fit the workgroup's share of the
// 160 KiB LDS at two waves per SIMD (8/W workgroups per CU), between 2 and 4,
// after the other LDS arrays.
template <int ESZ, int D, int W, bool POS, int RB = 4>
struct Stages {
  static constexpr int kTT = TileTokens<ESZ, W>::value;
  static constexpr int kTile = kTT * D * ESZ;
  static constexpr int kOther = W * ((POS ? 5 : 2) * kTT + 16 * RB) * 4;
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
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"   // m0 is set on purpose
__device__ __forceinline__ void load_lds16(const void* gptr, uint32_t lds_base) {
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off"
               :
               : "v"(gptr), "s"(lds_base)
               : "memory", "m0");
}
// The same load with a uniform 64-bit base in scalar registers and a 32-bit
// per-lane byte offset.
__device__ __forceinline__ void load_lds16_s(const void* sbase, uint32_t voff, uint32_t lds_base) {
  asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1"
               :
               : "v"(voff), "s"(sbase), "s"(lds_base)
               : "memory", "m0");
}
#pragma clang diagnostic pop

// A pointer every lane holds the same value of, moved to scalar registers.
__device__ __forceinline__ const unsigned char* uniform_ptr(const unsigned char* p) {
  const uint64_t v = reinterpret_cast<uintptr_t>(p);
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(v >> 32));
  return reinterpret_cast<const unsigned char*>(((uint64_t)hi << 32) | lo);
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

// Sum / max over the 16 lanes of a DPP row (lanes 16j..16j+15: the 16 token
// columns of one query row in the MFMA output), returned in every one of
// them.  Two quad permutes, a half-row mirror and a row mirror, each fused
// into the VALU op; the combination order is the same in every lane, so all
// 16 hold bitwise-equal results.
template <int CTRL>
__device__ __forceinline__ float dpp_f32(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL,
                                                               0xf, 0xf, false));
}
__device__ __forceinline__ float row16_sum(float v) {
  v += dpp_f32<0xB1>(v);    // quad_perm [1,0,3,2]
  v += dpp_f32<0x4E>(v);    // quad_perm [2,3,0,1]
  v += dpp_f32<0x141>(v);   // row_half_mirror
  v += dpp_f32<0x140>(v);   // row_mirror
  return v;
}
__device__ __forceinline__ float row16_max(float v) {
  v = fmaxf(v, dpp_f32<0xB1>(v));
  v = fmaxf(v, dpp_f32<0x4E>(v));
  v = fmaxf(v, dpp_f32<0x141>(v));
  v = fmaxf(v, dpp_f32<0x140>(v));
  return v;
}

// Maximum over the four lane groups (see sum_lane_groups).
__device__ __forceinline__ float max_lane_groups(float v) {
  const auto p = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v),
                                                  false, false);
  const float s = fmaxf(__uint_as_float(p[0]), __uint_as_float(p[1]));
  const auto q = __builtin_amdgcn_permlane32_swap(__float_as_uint(s), __float_as_uint(s),
                                                  false, false);
  return fmaxf(__uint_as_float(q[0]), __uint_as_float(q[1]));
}

// v plus its value in the paired lane group (lanes l and l^16), the same in
// both lanes.
__device__ __forceinline__ float sum_lane_pairs(float v) {
  const auto p = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v),
                                                  false, false);
  return __uint_as_float(p[0]) + __uint_as_float(p[1]);
}

// Position pooling inside a 16-lane DPP row (the 16 positions of a column
// block): row_shl:n gives lane c the value of lane c+n, row_shr:n that of
// lane c-n; lanes whose source falls outside the row read 0.  Values are
// the bit patterns of non-negative floats, whose unsigned order is their
// numeric order, so 0 is the identity of the maximum.
template <int CTRL>
__device__ __forceinline__ uint32_t dpp_z(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, CTRL, 0xf, 0xf, true);
}
template <int N> __device__ __forceinline__ uint32_t row_shl(uint32_t v) { return dpp_z<0x100 + N>(v); }
template <int N> __device__ __forceinline__ uint32_t row_shr(uint32_t v) { return dpp_z<0x110 + N>(v); }
__device__ __forceinline__ uint32_t umax(uint32_t a, uint32_t b) { return a > b ? a : b; }
// max over positions c-3..c (left part) and c..c+3 (right part) of a block
__device__ __forceinline__ uint32_t left4(uint32_t x) {
  const uint32_t l2 = umax(x, row_shr<1>(x));
  return umax(l2, row_shr<2>(l2));
}
__device__ __forceinline__ uint32_t right4(uint32_t x) {
  const uint32_t r2 = umax(x, row_shl<1>(x));
  return umax(r2, row_shl<2>(r2));
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


// ---- device-scope hand-over between workgroups ---------------------------

__device__ __forceinline__ uint32_t poll_u32(const uint32_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void count_in(uint32_t* p) {
  __hip_atomic_fetch_add(p, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void put_f32(float* p, float v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float get_f32(const float* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void put_f2(float2* p, float2 v) {
  __hip_atomic_store(reinterpret_cast<unsigned long long*>(p),
                     __builtin_bit_cast(unsigned long long, v), __ATOMIC_RELAXED,
                     __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float2 get_f2(const float2* p) {
  return __builtin_bit_cast(
      float2, __hip_atomic_load(reinterpret_cast<const unsigned long long*>(p),
                                __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
}
__device__ __forceinline__ int32_t get_i32(const int32_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Every wave waits for its own stores to complete, then the workgroup
// meets; after this one thread may publish the workgroup's results.
__device__ __forceinline__ void stores_done_barrier() {
  __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
  __syncthreads();
}

// Thread 0 waits until *p >= target; all threads get the outcome.  Gives up
// after `limit` polls (raising the error flag; a limit of 0 gives up at
// once) or as soon as another wait has raised it.
__device__ __forceinline__ bool wait_for(const uint32_t* p, uint32_t target, uint32_t* err,
                                         uint32_t limit, int* s_ok) {
  if (threadIdx.x == 0) {
    int ok = 1;
    uint32_t n = 0;
    while (n < limit && poll_u32(p) < target) {
      ++n;
      if ((n & 63u) == 0 && poll_u32(err) != 0u) {
        ok = 0;
        break;
      }
      __builtin_amdgcn_s_sleep(2);
    }
    if (ok && n >= limit) {
      __hip_atomic_fetch_or(err, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      ok = 0;
    }
    *s_ok = ok;
  }
  __syncthreads();
  return *s_ok != 0;
}

__device__ __forceinline__ int64_t take_item(uint32_t* sync) {
  return (int64_t)atomicAdd(reinterpret_cast<unsigned long long*>(sync), 1ull);
}

struct Item {
  int stage, unit, sub;
};

__device__ __forceinline__ Item decode(const WorkList& wl, int64_t item) {
  int i = 0;
  while (i + 1 < wl.nseg && item >= wl.seg_item[i + 1]) ++i;
  const int64_t rem = item - wl.seg_item[i];
  const int step = wl.seg_step[i] + (int)(rem / wl.seg_size[i]);
  int r = (int)(rem % wl.seg_size[i]);
  for (int s = 0; s < wl.nstages; ++s) {
    const int u = step - wl.lag[s];
    if (u >= 0 && u < wl.units) {
      if (r < wl.per_unit[s]) return Item{s, u, r};
      r -= wl.per_unit[s];
    }
  }
  return Item{-1, 0, 0};
}

// LDS of one workgroup, shared by every item type.
template <int ESZ, int D, int W, bool POS, int RB = 4>
struct Shared {
  static constexpr int kTT = TileTokens<ESZ, W>::value;
  using Gm = Geo<ESZ, D, kTT>;
  static constexpr int kStages = Stages<ESZ, D, W, POS, RB>::value;
  unsigned char ktile[kStages][Gm::kTileBytes] __attribute__((aligned(16)));
  float imp[2][W][kTT];          // P2 per-wave column sums of a tile (by tile parity)
  // Position variant: per-wave correction numerators of a tile, by tile
  // index mod 3 (a tile's last block is finalised during the next tile).
  float num[POS ? 3 : 1][W][POS ? kTT : 1];
  float lse[W * 16 * RB];        // P2 row normalisers
  int64_t next;                  // next item, taken by thread 0 during this one
  int ok;                        // outcome of the last dependency wait
};

// ---- score items: P1 and P2 of one (unit, row group, chunk) ---------------
// Query row rho of a unit (0 <= rho < Rp): whether it is a real row, and its
// index h*m + r among the unit's G*m query rows.  The importance path uses
// rho = h*m + r; the position variant rho = r*Gp + h (padding heads h >= G).
template <bool POS>
__device__ __forceinline__ bool real_row(const PersistArgs& a, int rho, int* qrow) {
  if (!POS) {
    *qrow = rho;
    return rho < a.R;
  }
  const int r = rho >> a.gshift, h = rho & (a.Gp - 1);
  *qrow = h * a.m + r;
  return r < a.m && h < a.G;
}

// PM (position variant): 0 reads the power mode and head grouping from the
// arguments; 1 fixes p = 2 and groups of four query heads at compile time,
// so the per-block pooling epilogue has no run-time branches.
template <int ESZ, int D, int W, int RB, bool PASS2, bool POS, int PM = 0>
__device__ __forceinline__ void score_item(const PersistArgs& a, int u, int sub,
                                           Shared<ESZ, D, W, POS, RB>& sh) {
  const int pow_mode = PM == 1 ? (int)kPowSquare : a.pow_mode;
  const int gshift = PM == 1 ? 2 : a.gshift;
  static_assert(RB == 4 || (RB == 5 && !POS), "five row blocks only for the importance path");
  constexpr int kRPW = 16 * RB;                  // query rows per wave
  constexpr int kGroupRows = kRPW * kMaxWaves;   // rows per row group
  constexpr int TT = TileTokens<ESZ, W>::value;   // positions per K tile
  using Gm = Geo<ESZ, D, TT>;
  constexpr int kBlocks = Gm::kBlocks;
  constexpr int kPer = Gm::kTileChunks / (W * 64);   // 16-byte loads per thread per tile
  constexpr int kStages = Stages<ESZ, D, W, POS, RB>::value;  // K tiles resident/in flight in LDS
  static_assert(Gm::kTileChunks % (W * 64) == 0, "tile must split evenly");
  auto& ktile = sh.ktile;
  float* lse_lds = sh.lse;

  const int chunk = sub % a.chunks;
  const int rg = sub / a.chunks;
  const int layer = (u / a.Hkv) % a.L;
  const int kvh = u % a.Hkv;
  uint32_t* done1 = a.sync + kSyncHeader;
  uint32_t* done2 = done1 + (size_t)a.units * a.row_groups;

  // The thread index passes through an empty asm so that the per-lane
  // addresses derived from it are recomputed for each item instead of being
  // hoisted out of the persistent loop, where they would outlive the register
  // budget and be spilled to scratch memory.
  int tid = threadIdx.x;
  asm volatile("" : "+v"(tid));
  const int wave = tid >> 6;
  const int lane = tid & 63;
  const int lg = lane >> 4;   // lane group: which quarter of the contraction / which 4 rows
  const int lc = lane & 15;   // lane column: token within a 16-token block / Q row

  const unsigned char* qb = static_cast<const unsigned char*>(a.q) +
                            (size_t)((layer * a.Hq + kvh * a.G) * a.m) * Gm::kRowBytes;
  const unsigned char* kb = static_cast<const unsigned char*>(a.k) +
                            (size_t)u * (size_t)a.T * Gm::kRowBytes;

  const int wrow0 = rg * kGroupRows + wave * kRPW;
  const bool wave_active = wrow0 < a.Rp;

  // ---- P2 prologue: wait for the row group's statistics, fold them --------
  // One thread per row (some take two with five row blocks per wave); chunks
  // are folded in ascending order, eight loads in flight, so every workgroup
  // of the unit derives bitwise-identical lse2.
  if (PASS2) {
    const bool ok = wait_for(done1 + (size_t)u * a.row_groups + rg, (uint32_t)a.chunks,
                             a.sync + kSyncError, a.spin_limit, &sh.ok);
    const int row_base = rg * kGroupRows;
    const int nrows = (a.Rp - row_base < W * kRPW) ? a.Rp - row_base : W * kRPW;
    for (int lr = tid; lr < nrows; lr += W * 64) {
      const int row = row_base + lr;
      const float2* p = a.partial + (size_t)u * a.chunks * a.Rp + row;
      float m = -INFINITY, z = 0.f;
      int c = 0;
      for (; c + 8 <= a.chunks; c += 8) {
        float2 v[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) v[j] = get_f2(p + (size_t)(c + j) * a.Rp);
#pragma unroll
        for (int j = 0; j < 8; ++j) lse_merge(m, z, v[j].x, v[j].y);
      }
      for (; c < a.chunks; ++c) {
        const float2 v = get_f2(p + (size_t)c * a.Rp);
        lse_merge(m, z, v.x, v.y);
      }
      const float l2 = ok ? m + __log2f(z) : __builtin_nanf("");
      lse_lds[lr] = l2;
      int qrow;
      if (chunk == 0 && a.row_lse && real_row<POS>(a, row, &qrow))
        a.row_lse[(size_t)u * a.R + qrow] = l2 * 0.69314718055994530942f;
    }
  }
  // ---- query rows of this wave, resident in registers -----------------------
  u32x4 qf[RB][Gm::kSegs];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    int qrow;
    const bool real = real_row<POS>(a, wrow0 + rb * 16 + lc, &qrow);
    const u32x4* src = reinterpret_cast<const u32x4*>(qb + (size_t)(real ? qrow : 0) *
                                                              Gm::kRowBytes) + lg * Gm::kSegs;
#pragma unroll
    for (int sg = 0; sg < Gm::kSegs; ++sg) qf[rb][sg] = real ? src[sg] : u32x4{0, 0, 0, 0};
  }

  // ---- per-lane row state -----------------------------------------------------
  // Rows held by this lane: wrow0 + rb*16 + 4*lg + i.
  float st_m[RB][4], st_z[RB][4];   // pass 1: reference max / sum (log2 units)
  bool per_lane_max = false;      // pass 1: a slow-path tile made the row maxima per lane
  float row_l2[RB][4];             // pass 2: lse2 of the row (+inf for padding rows)
#pragma unroll
  for (int rb = 0; rb < RB; ++rb)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      st_m[rb][i] = -INFINITY;
      st_z[rb][i] = 0.f;
      row_l2[rb][i] = INFINITY;
    }

  const int64_t t_begin = (int64_t)chunk * a.chunk_tokens;
  const int64_t t_end = (t_begin + a.chunk_tokens < a.T) ? t_begin + a.chunk_tokens : a.T;
  const int ntiles = (int)((t_end - t_begin + TT - 1) / TT);

  int64_t next = 0;

  // P2 output of one tile: the sum over waves (in wave order) of the
  // per-wave column sums, as device-scope stores (the unit's SEL item reads
  // them); NaN if the statistics never arrived.
  float* imp_out = (a.row_groups > 1)
                       ? a.imp_partial + ((size_t)rg * a.units + u) * (size_t)a.T
                       : a.importance + (size_t)u * (size_t)a.T;
  auto flush_tile = [&](int tile, int t) {
    const int64_t pos = t_begin + (int64_t)tile * TT + t;
    if (pos >= t_end) return;
    float s = 0.f;
#pragma unroll
    for (int w = 0; w < W; ++w) s += sh.imp[tile & 1][w][t];
    imp_out[pos] = sh.ok ? s : __builtin_nanf("");
  };

  // Position variant: the correction numerator of a tile, combined over the
  // waves that hold rows of this row group, in wave order.
  float* num_out = nullptr;
  int num_waves = 0;
  if (POS) {
    num_out = (a.row_groups > 1)
                  ? a.numer_partial + ((size_t)rg * a.units + u) * (size_t)a.T
                  : a.numer + (size_t)u * (size_t)a.T;
    const int rows = a.Rp - rg * kGroupRows;
    num_waves = (rows + kRPW - 1) / kRPW;
    if (num_waves > W) num_waves = W;
  }
  auto flush_num = [&](int tile) {
    for (int t = tid; t < TT; t += W * 64) {
      const int64_t pos = t_begin + (int64_t)tile * TT + t;
      if (pos >= t_end) continue;
      float s = 0.f;
      for (int w = 0; w < num_waves; ++w) {
        const float v = sh.num[POS ? tile % 3 : 0][w][POS ? t : 0];
        s = pow_mode == kPowMax ? fmaxf(s, v) : s + v;
      }
      num_out[pos] = sh.ok ? s : __builtin_nanf("");
    }
  };

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
  // Where every load of a tile shares the lane's offset, the full-tile loads
  // take a scalar base per load and one offset register (no per-load
  // 64-bit addresses to keep live across the tile loop).
  constexpr bool kLinear =
      slots_linear(W * 64, kPer, Gm::kChunks, Gm::kSwz, Gm::kRowBytes);
  constexpr int kJBytes = (W * 64 / Gm::kChunks) * Gm::kRowBytes;
  auto issue_tile = [&](int tile, int buf) {
    const int64_t tbase = t_begin + (int64_t)tile * TT;
    const unsigned char* src = kb + (size_t)tbase * Gm::kRowBytes;
    const uint32_t dst = lds_ring + buf * Gm::kTileBytes;
    if (kLinear && tbase + TT <= t_end) {
      const unsigned char* ssrc = uniform_ptr(src);
#pragma unroll
      for (int j = 0; j < kPer; ++j)
        load_lds16_s(ssrc + (size_t)j * kJBytes, (uint32_t)koff[0],
                     __builtin_amdgcn_readfirstlane(dst + j * (W * 64) * 16));
    } else if (tbase + TT <= t_end) {
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
  auto mfma_block = [&](const u32x4 (&kf)[Gm::kSegs], f32x4 (&acc)[RB]) {
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) acc[rb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int sg = 0; sg < Gm::kSegs; ++sg)
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) mfma_seg<ESZ>(qf[rb][sg], kf[sg], acc[rb]);
  };
  auto column_block = [&](const unsigned char* kt, int tb, f32x4 (&acc)[RB]) {
    u32x4 kf[Gm::kSegs];
    load_block(kt, tb, kf);
    mfma_block(kf, acc);
  };
  // Software pipeline over the four column blocks of a tile: the LDS reads
  // and MFMAs of block tb+1 are issued ahead of block tb's exp epilogue, and
  // the scheduler is asked to interleave them, so the matrix unit and the
  // VALU work at the same time within one wave.
  constexpr int kMfmaPerBlock = RB * Gm::kSegs * (ESZ == 4 ? 4 : 1);
  auto pipelined_tile = [&](const unsigned char* kt, auto&& epilogue) {
    u32x4 kf[2][Gm::kSegs];
    f32x4 acc[2][RB];
    load_block(kt, 0, kf[0]);
    mfma_block(kf[0], acc[0]);
#pragma unroll
    for (int tb = 0; tb < kBlocks; ++tb) {
      const int cur = tb & 1;
      if (tb < kBlocks - 1) {
        load_block(kt, tb + 1, kf[cur ^ 1]);
        mfma_block(kf[cur ^ 1], acc[cur ^ 1]);
      }
      epilogue(tb, acc[cur]);
      if (tb < kBlocks - 1) interleave_mfma_valu<kMfmaPerBlock, 3>();
    }
  };

  // ---- position variant: pooled per-token weights ---------------------------
  // The query rows are ordered rho = r*Gp + h, so lane (lg, lc) of row block
  // rb holds, summed over its four rows i, the weight of query token
  // (wrow0 + rb*16 + 4*lg) >> gshift over Gp = 4 heads, or over half of
  // Gp = 8 heads (the paired lane group holds the other half), at position
  // lc of the column block.  Pool_7 over positions runs across the 16 lanes
  // of a DPP row and into the neighbouring blocks: a block is finalised when
  // the next block is known, from its left4/right4 parts; the blocks beyond
  // the chunk's two ends are computed separately from K in global memory.
  uint32_t r4p[4] = {0u, 0u, 0u, 0u};   // right4 of the previous block
  uint32_t pc[4] = {0u, 0u, 0u, 0u};    // previous block pooled, except the next block's part
  auto head_sum = [&](float v) { return gshift == 3 ? sum_lane_pairs(v) : v; };
  // Numerator terms of a finalised block, summed over this wave's tokens
  // (or their maximum at p = inf), into the tile's LDS slot.
  auto store_numer = [&](int btile, int btb, const uint32_t(&fin)[4]) {
    float acc = 0.f;
    if (pow_mode == kPowSquare) {
#pragma unroll
      for (int rb = 0; rb < 4; ++rb) {
        const float t = __uint_as_float(fin[rb]) * a.sq_scale;
        acc = __builtin_fmaf(t, t, acc);
      }
    } else if (pow_mode == kPowGeneral) {
#pragma unroll
      for (int rb = 0; rb < 4; ++rb)
        acc += __builtin_amdgcn_exp2f(__builtin_fmaf(
            a.pow_p, __builtin_amdgcn_logf(__uint_as_float(fin[rb])), a.pow_kappa));
    } else {
#pragma unroll
      for (int rb = 0; rb < 4; ++rb) acc = fmaxf(acc, __uint_as_float(fin[rb]));
    }
    if (pow_mode == kPowMax) {
      acc = max_lane_groups(acc);
    } else {
      if (gshift == 3 && (lg & 1)) acc = 0.f;   // the paired lane group holds the same tokens
      acc = sum_lane_groups(acc);
    }
    if (lg == 0) sh.num[POS ? btile % 3 : 0][wave][POS ? btb * 16 + lc : 0] = acc;
  };
  // Pool a new block x: finalise the previous one, keep this one's parts.
  auto pool_block = [&](const uint32_t(&x)[4], int tile, int tb) {
    uint32_t fin[4];
#pragma unroll
    for (int rb = 0; rb < 4; ++rb) {
      const uint32_t l4 = left4(x[rb]), r4 = right4(x[rb]);
      fin[rb] = umax(pc[rb], row_shr<13>(l4));   // lanes 13..15 see this block's 0..2
      pc[rb] = umax(umax(l4, r4), row_shl<13>(r4p[rb]));   // lanes 0..2 see 13..15 before
      r4p[rb] = r4;
    }
    if (tb > 0) {
      store_numer(tile, tb - 1, fin);
    } else if (tile > 0) {
      store_numer(tile - 1, kBlocks - 1, fin);
    }
  };
  // Weights of the block of 16 positions from tstart, from K in global memory
  // (positions outside [0, T) weigh 0).
  auto halo_bits = [&](int64_t tstart, uint32_t(&x)[4]) {
    const int64_t row = tstart + lc;
    const bool okr = row >= 0 && row < a.T;
    const u32x4* src = reinterpret_cast<const u32x4*>(kb + (size_t)(okr ? row : 0) *
                                                              Gm::kRowBytes) + lg * Gm::kSegs;
    u32x4 kf[Gm::kSegs];
#pragma unroll
    for (int sg = 0; sg < Gm::kSegs; ++sg) kf[sg] = src[sg];
    f32x4 acc[RB];
    mfma_block(kf, acc);
#pragma unroll
    for (int rb = 0; rb < 4; ++rb) {
      float p = 0.f;
#pragma unroll
      for (int i = 0; i < 4; ++i)
        p += __builtin_amdgcn_exp2f(__builtin_fmaf(acc[rb][i], a.c2, -row_l2[rb][i]));
      x[rb] = okr ? __float_as_uint(head_sum(p)) : 0u;
    }
  };
  auto load_row_l2 = [&]() {
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        int qrow;
        row_l2[rb][i] = real_row<POS>(a, wrow0 + rb * 16 + 4 * lg + i, &qrow)
                            ? lse_lds[wave * kRPW + rb * 16 + 4 * lg + i]
                            : INFINITY;
      }
  };
  if (PASS2 && POS) {
    __syncthreads();   // every row's lse2 is in LDS
    load_row_l2();
    if (wave_active && t_begin > 0) {
      uint32_t hx[4];
      halo_bits(t_begin - 16, hx);
#pragma unroll
      for (int rb = 0; rb < 4; ++rb) r4p[rb] = right4(hx[rb]);
    }
  }

  // Everything issued so far (query rows, chunk statistics, the left halo)
  // must land before the ring's vmcnt bookkeeping starts.
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
    // The next item is taken while the last tile is computed; no ring load
    // is in flight any more, so its latency hides behind the tile.
    if (tile == ntiles - 1 && tid == 0) next = take_item(a.sync);
    if (PASS2 && !POS && tile == 0) load_row_l2();
    // P2: the previous tile's per-wave column sums are complete; they are
    // added in wave order and the tile's importance is stored.  Numerators
    // trail by one more tile (a tile's last block is finalised in the next).
    if (PASS2 && tile > 0)
      for (int t = tid; t < TT; t += W * 64) flush_tile(tile - 1, t);
    if (PASS2 && POS && tile > 1) flush_num(tile - 2);
    if (!wave_active) {
      if (PASS2 && lg == 0)
#pragma unroll
        for (int tb = 0; tb < kBlocks; ++tb) sh.imp[tile & 1][wave][tb * 16 + lc] = 0.f;
      continue;
    }
    const unsigned char* kt = &ktile[buf][0];
    const int64_t tok0 = t_begin + (int64_t)tile * TT;
    const bool full = tok0 + TT <= t_end;

    if (PASS2) {
      // importance contribution: column sums of exp2(x - lse2) over the rows
      float* dst = &sh.imp[tile & 1][wave][lc];
      pipelined_tile(kt, [&](int tb, const f32x4(&acc)[RB]) {
        float part[RB];
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) {
          float p = 0.f;
#pragma unroll
          for (int i = 0; i < 4; ++i)
            p += __builtin_amdgcn_exp2f(__builtin_fmaf(acc[rb][i], a.c2, -row_l2[rb][i]));
          part[rb] = p;
        }
        float psum = (part[0] + part[1]) + (part[2] + part[3]);
#pragma unroll
        for (int rb = 4; rb < RB; ++rb) psum += part[rb];
        const float sum = sum_lane_groups(psum);
        if (lg == 0) dst[tb * 16] = sum;
        if constexpr (POS) {
          const bool okp = tok0 + tb * 16 + lc < a.T;
          uint32_t x[4];
#pragma unroll
          for (int rb = 0; rb < 4; ++rb) x[rb] = okp ? __float_as_uint(head_sum(part[rb])) : 0u;
          pool_block(x, tile, tb);
        }
      });
      continue;
    }

    // P1.  Each row's reference maximum m is the maximum over the first 16
    // positions of the chunk, the same in the 16 lanes that hold the row; the
    // fast path then adds exp2(x - m) with m fixed.  A row whose sum passes
    // 2^100 (a logit far above m) sends the whole tile to the slow path, from
    // the sums saved before it; below that, fp32 keeps full relative
    // precision, so a fixed m costs nothing.
    if (tile == 0) {
      f32x4 acc[RB];
      column_block(kt, 0, acc);
      const bool valid = tok0 + lc < t_end;
#pragma unroll
      for (int rb = 0; rb < RB; ++rb)
#pragma unroll
        for (int i = 0; i < 4; ++i)
          st_m[rb][i] = row16_max(valid ? acc[rb][i] * a.c2 : -INFINITY);
    }
    bool redo = false;
    {
      float zp[RB][4];
#pragma unroll
      for (int rb = 0; rb < RB; ++rb)
#pragma unroll
        for (int i = 0; i < 4; ++i) zp[rb][i] = st_z[rb][i];
      if (full) {
        pipelined_tile(kt, [&](int, const f32x4(&acc)[RB]) {
#pragma unroll
          for (int rb = 0; rb < RB; ++rb)
#pragma unroll
            for (int i = 0; i < 4; ++i)
              st_z[rb][i] += __builtin_amdgcn_exp2f(__builtin_fmaf(acc[rb][i], a.c2, -st_m[rb][i]));
        });
      } else {
        // Ragged tail: positions past the chunk end are masked out.
        pipelined_tile(kt, [&](int tb, const f32x4(&acc)[RB]) {
          const bool valid = tok0 + tb * 16 + lc < t_end;
#pragma unroll
          for (int rb = 0; rb < RB; ++rb)
#pragma unroll
            for (int i = 0; i < 4; ++i)
              st_z[rb][i] += __builtin_amdgcn_exp2f(
                  valid ? __builtin_fmaf(acc[rb][i], a.c2, -st_m[rb][i]) : -INFINITY);
        });
      }
      bool over = false;
#pragma unroll
      for (int rb = 0; rb < RB; ++rb)
#pragma unroll
        for (int i = 0; i < 4; ++i) over |= !(st_z[rb][i] <= 0x1p100f);
      if (__any(over)) {
        redo = true;
        per_lane_max = true;
#pragma unroll
        for (int rb = 0; rb < RB; ++rb)
#pragma unroll
          for (int i = 0; i < 4; ++i) st_z[rb][i] = zp[rb][i];
      }
    }
    if (redo) {
      // Slow path: a new large maximum.  Online max / rescale per column
      // block and lane, padding masked; from here on the lanes of a row hold
      // different maxima.
#pragma unroll
      for (int tb = 0; tb < kBlocks; ++tb) {
        f32x4 acc[RB];
        column_block(kt, tb, acc);
        const bool valid = tok0 + tb * 16 + lc < t_end;
#pragma unroll
        for (int rb = 0; rb < RB; ++rb)
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
  if (PASS2 && POS && wave_active) {
    // the chunk's last block: its right neighbour is the next chunk's first
    uint32_t hx[4] = {0u, 0u, 0u, 0u};
    if (t_end < a.T) halo_bits(t_end, hx);
    uint32_t fin[4];
#pragma unroll
    for (int rb = 0; rb < 4; ++rb) fin[rb] = umax(pc[rb], row_shr<13>(left4(hx[rb])));
    store_numer(ntiles - 1, kBlocks - 1, fin);
  }
  __syncthreads();

  if (PASS2) {
    for (int t = tid; t < TT; t += W * 64) flush_tile(ntiles - 1, t);
    if (POS) {
      if (ntiles > 1) flush_num(ntiles - 2);
      flush_num(ntiles - 1);
    }
    stores_done_barrier();
    if (tid == 0) {
      count_in(done2 + u);
      sh.next = next;
    }
    return;
  }

  // ---- P1: fold the 16 lane columns, publish per-chunk row statistics ------
  // With one maximum per row the sums simply add (DPP); after a slow-path
  // tile the (max, sum) pairs are merged with rescaling.
#pragma unroll
  for (int rb = 0; rb < RB; ++rb)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float m = st_m[rb][i], z = st_z[rb][i];
      if (!per_lane_max) {
        z = row16_sum(z);
      } else {
#pragma unroll
        for (int off = 1; off < 16; off <<= 1) {
          const float mo = __shfl_xor(m, off);
          const float zo = __shfl_xor(z, off);
          lse_merge(m, z, mo, zo);
        }
      }
      const int row = wrow0 + rb * 16 + 4 * lg + i;
      if (lc == 0 && row < a.Rp)
        put_f2(a.partial + ((size_t)u * a.chunks + chunk) * a.Rp + row, make_float2(m, z));
    }
  stores_done_barrier();
  if (tid == 0) {
    count_in(done1 + (size_t)u * a.row_groups + rg);
    sh.next = next;
  }
}

template <int ESZ, int D, int W, bool POS, int RB, int PM = 0>
// bf16: two waves per SIMD (<= 256 registers per lane) so one wave's MFMAs
// overlap another's exp/VALU epilogue.
__global__ __launch_bounds__(W * 64, ESZ == 2 ? 2 : 1) void persistent_kernel(PersistArgs a) {
  __shared__ Shared<ESZ, D, W, POS, RB> sh;
  if (threadIdx.x == 0) sh.next = take_item(a.sync);
  __syncthreads();
  int64_t item = sh.next;
  while (item < a.wl.items) {
    const Item it = decode(a.wl, item);
    switch (it.stage) {
      case kStageP1: score_item<ESZ, D, W, RB, false, POS, PM>(a, it.unit, it.sub, sh); break;
      case kStageP2: score_item<ESZ, D, W, RB, true, POS, PM>(a, it.unit, it.sub, sh); break;
      default:   // not reached: every item index below wl.items decodes
        if (threadIdx.x == 0) sh.next = take_item(a.sync);
        break;
    }
    __syncthreads();
    item = sh.next;
  }
}

// out[u][t] = sum (or maximum) over row groups, in order.
__global__ void rowgroup_sum(const float* __restrict__ part, float* __restrict__ out,
                             int row_groups, int64_t per_group, int64_t n, int take_max) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  float s = 0.f;
  for (int r = 0; r < row_groups; ++r)
    s = take_max ? fmaxf(s, part[r * per_group + i]) : s + part[r * per_group + i];
  out[i] = s;
}

__global__ void zero_words(uint32_t* __restrict__ p, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    p[i] = 0u;
}

// Resident workgroups per CU of one kernel instantiation, cached per device.
std::mutex g_occ_mu;
int g_occ[64][2][2][4][2][2][2];
int g_cus[64];

template <int ESZ, int D, int W, bool POS, int RB = 4, int PM = 0>
hipError_t launch_w(const ScorePlan& p, PersistArgs& a, hipStream_t s) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= 64) return hipErrorInvalidDevice;
  const int wi = W == 1 ? 0 : W == 2 ? 1 : W == 4 ? 2 : 3;
  int per_cu = 0, cus = 0;
  {
    std::lock_guard<std::mutex> lock(g_occ_mu);
    int& occ = g_occ[dev][ESZ == 2][D == 128][wi][POS][RB == 5][PM];
    if (occ == 0) {
      e = hipOccupancyMaxActiveBlocksPerMultiprocessor(
          &occ, reinterpret_cast<const void*>(&persistent_kernel<ESZ, D, W, POS, RB, PM>), W * 64, 0);
      if (e != hipSuccess) return e;
      if (occ < 1) occ = 1;
    }
    if (g_cus[dev] == 0) {
      e = hipDeviceGetAttribute(&g_cus[dev], hipDeviceAttributeMultiprocessorCount, dev);
      if (e != hipSuccess) return e;
    }
    per_cu = occ;
    cus = g_cus[dev];
  }
  const int resident = per_cu * cus;
  int per_unit[kMaxStages];
  // Item size: the largest that gives the resident workgroups more P1 items
  // than there are workgroups.  With exactly one each, every P1 item runs in
  // the first round and every P2 item in the second, with nothing to overlap
  // the second pass's re-reads of K (8 layers x 8 KV heads x 65536
  // positions: 476 us at 2048 positions against 512 us at 4096).
  a.chunk_tokens = kMinChunkTokens;
  for (int c = kMaxChunkTokens; c > kMinChunkTokens; c /= 2)
    if ((int64_t)p.units * p.row_groups * ((p.T + c - 1) / c) > resident) {
      a.chunk_tokens = c;
      break;
    }
  a.chunks = (int)((p.T + a.chunk_tokens - 1) / a.chunk_tokens);
  per_unit[kStageP1] = a.chunks * p.row_groups;
  per_unit[kStageP2] = a.chunks * p.row_groups;
  make_work_list(p.units, kMaxStages, per_unit, resident, &a.wl);
  const int64_t grid = a.wl.items < resident ? a.wl.items : resident;
  zero_words<<<(unsigned)((p.sync_words + 255) / 256 < 1024 ? (p.sync_words + 255) / 256 : 1024),
               256, 0, s>>>(a.sync, (int64_t)p.sync_words);
  persistent_kernel<ESZ, D, W, POS, RB, PM><<<(unsigned)grid, W * 64, 0, s>>>(a);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (p.row_groups > 1) {
    const int64_t n = (int64_t)p.units * p.T;
    rowgroup_sum<<<(unsigned)((n + 255) / 256), 256, 0, s>>>(a.imp_partial, a.importance,
                                                            p.row_groups, n, n, 0);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (POS) {
      rowgroup_sum<<<(unsigned)((n + 255) / 256), 256, 0, s>>>(
          a.numer_partial, a.numer, p.row_groups, n, n, a.pow_mode == kPowMax);
      e = hipGetLastError();
    }
  }
  return e;
}

template <int ESZ, int D, bool POS>
hipError_t launch_d(const ScorePlan& p, PersistArgs& a, hipStream_t s) {
  if constexpr (!POS) {
    if (p.rb == 5) return launch_w<ESZ, D, 4, POS, 5>(p, a, s);
  } else if (a.pow_mode == kPowSquare && a.gshift == 2) {
    // the paper's default score (p = 2) with four query heads per KV head
    switch (p.waves) {
      case 1: return launch_w<ESZ, D, 1, true, 4, 1>(p, a, s);
      case 2: return launch_w<ESZ, D, 2, true, 4, 1>(p, a, s);
      case 4: return launch_w<ESZ, D, 4, true, 4, 1>(p, a, s);
      default: return launch_w<ESZ, D, 8, true, 4, 1>(p, a, s);
    }
  }
  switch (p.waves) {
    case 1: return launch_w<ESZ, D, 1, POS>(p, a, s);
    case 2: return launch_w<ESZ, D, 2, POS>(p, a, s);
    case 4: return launch_w<ESZ, D, 4, POS>(p, a, s);
    default: return launch_w<ESZ, D, 8, POS>(p, a, s);
  }
}

}  // namespace

// Launch of the persistent score kernel for one element size and head
// dimension; each combination is instantiated in a translation unit of its
// own (score_<dtype>_d<D>.hip, and score_pos_<dtype>_d<D>.hip for the
// position variant) so that they compile in parallel.
template <int ESZ, int D>
hipError_t launch_score_d(const ScorePlan& p, PersistArgs& a, hipStream_t s) {
  return launch_d<ESZ, D, false>(p, a, s);
}
template <int ESZ, int D>
hipError_t launch_position_d(const ScorePlan& p, PersistArgs& a, hipStream_t s) {
  return launch_d<ESZ, D, true>(p, a, s);
}

}  // namespace cb
