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
  static constexpr int kWords = kWaves * 256 + kWaves + 1 + 2;
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

// Histogram counting with one LDS atomic per run of equal digits in a
// thread's (position-ordered) keys instead of one per key: near-uniform
// scores put almost every key of a row into the same one or two bins, where
// per-key atomics from all 64 lanes of a wave would serialise on one address.
struct DigitRuns {
  uint32_t digit = 0xffffffffu, count = 0;
  __device__ __forceinline__ void add(uint32_t* h, uint32_t d) {
    if (d != digit) {
      if (count) atomicAdd(&h[digit], count);
      digit = d;
      count = 0;
    }
    ++count;
  }
  __device__ __forceinline__ void flush(uint32_t* h) {
    if (count) atomicAdd(&h[digit], count);
  }
};

// Radix-select driver shared by both key sources below.  `digit_pass`
// adds this thread's keys that match `prefix` on the digits above `shift`
// into hist[wave][digit]; `count` and `emit` walk this thread's contiguous
// span of positions for the ordered output.
template <int NT, typename DigitPass, typename Count, typename Emit>
__device__ __forceinline__ void radix_select(int keep, uint32_t* work, DigitPass&& digit_pass,
                                             Count&& count, Emit&& emit) {
  constexpr int kWaves = NT / 64;
  uint32_t* hist = work;                          // [kWaves][256]
  uint32_t* scan_scratch = work + kWaves * 256;   // kWaves + 1
  uint32_t* s_vars = scan_scratch + kWaves + 1;   // prefix, need
  const int tid = threadIdx.x, wave = tid >> 6;

  uint32_t prefix = 0, need = (uint32_t)keep;
  for (int pass = 0; pass < 4; ++pass) {
    const int shift = 24 - 8 * pass;
    const uint32_t hi_mask = pass == 0 ? 0u : (0xffffffffu << (shift + 8));
    for (int i = tid; i < kWaves * 256; i += NT) hist[i] = 0;
    __syncthreads();
    digit_pass(hist + wave * 256, prefix, hi_mask, shift);
    __syncthreads();
    for (int d = tid; d < 256; d += NT) {
      uint32_t s = 0;
      for (int w = 0; w < kWaves; ++w) s += hist[w * 256 + d];
      hist[d] = s;
    }
    __syncthreads();
    if (wave == 0) {
      // The digit d with (count of digits > d) < need <= (count of digits >= d).
      // Lane j owns digits 4j..4j+3; a suffix scan over lanes counts the
      // digits above each lane.  Exactly one (lane, digit) satisfies the test.
      const int lane = tid;
      uint32_t c[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) c[q] = hist[4 * lane + q];
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
          s_vars[0] = prefix | ((uint32_t)(4 * lane + q) << shift);
          s_vars[1] = need - above;
        }
        above += c[q];
      }
    }
    __syncthreads();
    prefix = s_vars[0];
    need = s_vars[1];
    __syncthreads();
  }
  const uint32_t theta = prefix;

  // Ordered output: every key above theta, plus the first `need` keys equal
  // to theta in position order.  Block scans give each thread's first slot.
  uint32_t gt = 0, eq = 0;
  count(theta, gt, eq);
  uint32_t gt_total, eq_total;
  const uint32_t gt_before = block_exclusive_scan<NT>(gt, scan_scratch, &gt_total);
  const uint32_t eq_before = block_exclusive_scan<NT>(eq, scan_scratch, &eq_total);
  (void)gt_total;
  (void)eq_total;
  emit(theta, need, eq_before, gt_before + (eq_before < need ? eq_before : need));
}

// Select `keep` of the T scores in `row` into out[0..keep), ascending.  All
// NT threads of the workgroup call it; `work` holds SelectLds<NT>::kWords
// words of LDS.  Thread i owns the contiguous positions [i*per, (i+1)*per),
// per = ceil(T / NT).  With per <= KPT its keys are loaded once into
// registers (one pass over the scores, all loads in flight); otherwise every
// pass re-reads the scores from global memory (L2), eight loads at a time.
template <int NT, int KPT>
__device__ __forceinline__ void select_unit(const float* __restrict__ row, int T, int keep,
                                            int32_t* __restrict__ out, uint32_t* work) {
  const int tid = threadIdx.x;
  const int per = (T + NT - 1) / NT;
  const int lo = tid * per < T ? tid * per : T;
  const int hi = lo + per < T ? lo + per : T;
  const int n = hi - lo;

  // Loads first, unconditionally (addresses clamped into the row), so that
  // they are all in flight together; conversion and masking afterwards.
  auto at = [&](int j) { return row + (lo + j < T ? lo + j : T - 1); };
  if (per <= KPT) {
    uint32_t key[KPT];
#pragma unroll
    for (int j = 0; j < KPT; ++j) key[j] = __float_as_uint(*at(j));
#pragma unroll
    for (int j = 0; j < KPT; ++j) key[j] = j < n ? order_key(__uint_as_float(key[j])) : 0u;
    radix_select<NT>(
        keep, work,
        [&](uint32_t* h, uint32_t prefix, uint32_t hi_mask, int shift) {
          DigitRuns runs;
#pragma unroll
          for (int j = 0; j < KPT; ++j)
            if (j < n && (key[j] & hi_mask) == prefix) runs.add(h, (key[j] >> shift) & 255u);
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
#pragma unroll
          for (int j = 0; j < KPT; ++j) {
            if (j >= n) continue;
            bool take = key[j] > theta;
            if (key[j] == theta) {
              take = eq_seen < need;
              ++eq_seen;
            }
            if (take && pos < (uint32_t)keep) out[pos++] = lo + j;
          }
        });
    return;
  }

  constexpr int B = 8;
  radix_select<NT>(
      keep, work,
      [&](uint32_t* h, uint32_t prefix, uint32_t hi_mask, int shift) {
        for (int j0 = 0; j0 < n; j0 += B) {
          uint32_t kb[B];
#pragma unroll
          for (int j = 0; j < B; ++j) kb[j] = __float_as_uint(*at(j0 + j));
#pragma unroll
          for (int j = 0; j < B; ++j) kb[j] = j0 + j < n ? order_key(__uint_as_float(kb[j])) : 0u;
          DigitRuns runs;
#pragma unroll
          for (int j = 0; j < B; ++j)
            if (j0 + j < n && (kb[j] & hi_mask) == prefix) runs.add(h, (kb[j] >> shift) & 255u);
          runs.flush(h);
        }
      },
      [&](uint32_t theta, uint32_t& gt, uint32_t& eq) {
        for (int j0 = 0; j0 < n; j0 += B) {
          uint32_t kb[B];
#pragma unroll
          for (int j = 0; j < B; ++j) kb[j] = __float_as_uint(*at(j0 + j));
#pragma unroll
          for (int j = 0; j < B; ++j) kb[j] = j0 + j < n ? order_key(__uint_as_float(kb[j])) : 0u;
#pragma unroll
          for (int j = 0; j < B; ++j) {
            gt += j0 + j < n && kb[j] > theta;
            eq += j0 + j < n && kb[j] == theta;
          }
        }
      },
      [&](uint32_t theta, uint32_t need, uint32_t eq_seen, uint32_t pos) {
        for (int j0 = 0; j0 < n; j0 += B) {
          uint32_t kb[B];
#pragma unroll
          for (int j = 0; j < B; ++j) kb[j] = __float_as_uint(*at(j0 + j));
#pragma unroll
          for (int j = 0; j < B; ++j) kb[j] = j0 + j < n ? order_key(__uint_as_float(kb[j])) : 0u;
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
