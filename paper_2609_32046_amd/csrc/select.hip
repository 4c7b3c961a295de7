// Per-unit top-k with the (score descending, index ascending) rule, output in
// source order (gfx950).
//
// One workgroup of 1024 threads per unit.  Scores are mapped to uint32 keys
// whose unsigned order is the float order (-0 -> +0, NaN -> 0, the lowest).
// An MSB-first radix select over four 8-bit digits finds the keep-th largest
// key theta and how many keys equal to theta must be taken (`need`); each
// digit pass builds per-wave histograms in LDS (flat score distributions put
// most keys in one bin, so a single shared histogram would serialise).  A
// final ordered pass flags every key above theta plus the first `need` keys
// equal to theta, and a block-wide exclusive scan turns the flags into output
// positions, which are therefore ascending in index.  Integer work only, so
// the result is exact and deterministic.
//
// Keys live in LDS when T <= kLdsKeys; longer rows are re-read from global
// memory (L2) on every pass.
#include "kernels.h"

namespace cb {
namespace {

constexpr int kThreads = 1024;
constexpr int kWaves = kThreads / 64;
constexpr int kLdsKeys = 32768;   // 128 KiB of keys

__device__ __forceinline__ uint32_t order_key(float f) {
  uint32_t b = __float_as_uint(f);
  if ((b & 0x7f800000u) == 0x7f800000u && (b & 0x007fffffu)) return 0u;   // NaN
  if (b == 0x80000000u) b = 0u;                                            // -0 == +0
  return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}

// Exclusive scan of one value per thread over the block; returns the prefix
// and writes the total to *total.  `scratch` holds kWaves + 1 entries.
__device__ __forceinline__ uint32_t block_exclusive_scan(uint32_t v, uint32_t* scratch,
                                                          uint32_t* total) {
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

template <bool IN_LDS>
__global__ __launch_bounds__(kThreads) void select_kernel(const float* __restrict__ importance,
                                                          int64_t T64, int64_t keep64,
                                                          int32_t* __restrict__ idx) {
  extern __shared__ uint32_t keys_lds[];
  __shared__ uint32_t hist[kWaves][256];
  __shared__ uint32_t scan_scratch[kWaves + 1];
  __shared__ uint32_t s_prefix, s_need;

  const int T = (int)T64;
  const int keep = (int)keep64;
  const int u = blockIdx.x;
  const float* row = importance + (size_t)u * T;
  const int tid = threadIdx.x, wave = tid >> 6;

  auto key_at = [&](int t) -> uint32_t { return IN_LDS ? keys_lds[t] : order_key(row[t]); };

  if (IN_LDS)
    for (int t = tid; t < T; t += kThreads) keys_lds[t] = order_key(row[t]);

  uint32_t prefix = 0, need = (uint32_t)keep;
  for (int pass = 0; pass < 4; ++pass) {
    const int shift = 24 - 8 * pass;
    const uint32_t hi_mask = pass == 0 ? 0u : (0xffffffffu << (shift + 8));
    for (int i = tid; i < kWaves * 256; i += kThreads) (&hist[0][0])[i] = 0;
    __syncthreads();
    for (int t = tid; t < T; t += kThreads) {
      const uint32_t key = key_at(t);
      if ((key & hi_mask) == prefix) atomicAdd(&hist[wave][(key >> shift) & 255u], 1u);
    }
    __syncthreads();
    if (tid < 256) {
      uint32_t s = 0;
      for (int w = 0; w < kWaves; ++w) s += hist[w][tid];
      hist[0][tid] = s;
    }
    __syncthreads();
    if (wave == 0) {
      // The digit d with (count of digits > d) < need <= (count of digits >= d).
      // Lane j owns digits 4j..4j+3; a suffix scan over lanes counts the
      // digits above each lane.  Exactly one (lane, digit) satisfies the test.
      const int lane = tid;
      uint32_t c[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) c[q] = hist[0][4 * lane + q];
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
          s_prefix = prefix | ((uint32_t)(4 * lane + q) << shift);
          s_need = need - above;
        }
        above += c[q];
      }
    }
    __syncthreads();
    prefix = s_prefix;
    need = s_need;
    __syncthreads();
  }
  const uint32_t theta = prefix;

  // Ordered flag pass: thread tid owns the contiguous span [lo, hi).
  const int per = (T + kThreads - 1) / kThreads;
  const int lo = tid * per < T ? tid * per : T;
  const int hi = lo + per < T ? lo + per : T;
  uint32_t gt = 0, eq = 0;
  for (int t = lo; t < hi; ++t) {
    const uint32_t key = key_at(t);
    gt += key > theta;
    eq += key == theta;
  }
  uint32_t gt_total, eq_total;
  const uint32_t gt_before = block_exclusive_scan(gt, scan_scratch, &gt_total);
  const uint32_t eq_before = block_exclusive_scan(eq, scan_scratch, &eq_total);
  (void)gt_total;
  (void)eq_total;
  uint32_t eq_seen = eq_before;
  uint32_t pos = gt_before + (eq_before < need ? eq_before : need);
  int32_t* out = idx + (size_t)u * keep;
  for (int t = lo; t < hi; ++t) {
    const uint32_t key = key_at(t);
    bool take = key > theta;
    if (key == theta) {
      take = eq_seen < need;
      ++eq_seen;
    }
    if (take && pos < (uint32_t)keep) out[pos++] = t;
  }
}

}  // namespace

hipError_t launch_select(const float* importance, int64_t units, int64_t T, int64_t keep,
                         int32_t* idx, hipStream_t s) {
  if (T <= kLdsKeys) {
    // Up to 128 KiB of dynamic LDS (of gfx950's 160 KiB per workgroup).
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&select_kernel<true>),
                              hipFuncAttributeMaxDynamicSharedMemorySize,
                              (int)(kLdsKeys * sizeof(uint32_t)));
    select_kernel<true><<<(unsigned)units, kThreads, (size_t)T * sizeof(uint32_t), s>>>(
        importance, T, keep, idx);
  } else {
    select_kernel<false><<<(unsigned)units, kThreads, 0, s>>>(importance, T, keep, idx);
  }
  return hipGetLastError();
}

}  // namespace cb
