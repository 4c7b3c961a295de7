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
  // two histogram buffers [kWaves][256], scan scratch, two (prefix, need),
  // the count of keys equal to the threshold, the exchange outcome of a
  // split row
  static constexpr int kWords = 2 * kWaves * 256 + kWaves + 1 + 6;
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

// Threshold of the radix select, shared by every key source below:
// `digit_pass` adds this thread's keys that match `prefix` on the digits
// above `shift` into hist[wave][digit].  On return *theta is the keep-th
// largest key and *need the number of keys equal to it that the selection
// takes; all NT threads hold the same values.  The first of the two
// histogram buffers (work[0, NT/64*256)) is free for the caller afterwards.
// With kCleared the caller has already zeroed the first histogram buffer
// (select_clear_first_hist) and passed a barrier since.  *n_theta (nullable)
// receives the number of keys equal to theta.
struct NoMerge {
  __device__ __forceinline__ void operator()(int, uint32_t (&)[4]) const {}
};

// `merge` (wave 0, all lanes) may replace the workgroup's counts of the
// digits 4*lane .. 4*lane+3 of a pass by those of the whole row, when the
// row is split over several workgroups.
template <int NT, bool kCleared = false, typename DigitPass, typename Merge = NoMerge>
__device__ __forceinline__ void radix_threshold(int keep, uint32_t* work, DigitPass&& digit_pass,
                                                uint32_t* theta, uint32_t* need_out,
                                                uint32_t* n_theta = nullptr,
                                                Merge&& merge = Merge{}) {
  constexpr int kWaves = NT / 64;
  uint32_t* hists = work;                             // [2][kWaves][256]
  uint32_t* scan_scratch = work + 2 * kWaves * 256;   // kWaves + 1
  uint32_t* s_vars = scan_scratch + kWaves + 1;       // [2] x (prefix, need), n_theta
  const int tid = threadIdx.x, wave = tid >> 6;

  // Pass p counts into buffer p & 1 and clears the other one for pass p+1;
  // that buffer was last read (by wave 0) before the previous pass's final
  // barrier.  Two barriers per pass: histograms complete, digit chosen.
  if (!kCleared) {
    for (int i = tid; i < kWaves * 256; i += NT) hists[i] = 0;
    __syncthreads();
  }
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
      merge(pass, c);
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
          s_vars[4] = c[q];   // after the last pass: the keys equal to theta
        }
        above += c[q];
      }
    }
    __syncthreads();
    prefix = s_vars[2 * (pass & 1)];
    need = s_vars[2 * (pass & 1) + 1];
  }
  *theta = prefix;
  *need_out = need;
  if (n_theta) *n_theta = s_vars[4];
}

// Radix select over keys that each thread holds as one contiguous span of
// positions: the threshold above, then `count` and `emit` walk this thread's
// span for the ordered output.
template <int NT, typename DigitPass, typename Count, typename Emit>
__device__ __forceinline__ void radix_select(int keep, uint32_t* work, DigitPass&& digit_pass,
                                             Count&& count, Emit&& emit) {
  constexpr int kWaves = NT / 64;
  uint32_t* scan_scratch = work + 2 * kWaves * 256;   // kWaves + 1
  uint32_t theta, need;
  radix_threshold<NT>(keep, work, digit_pass, &theta, &need);

  // Ordered output: every key above theta, plus the first `need` keys equal
  // to theta in position order.  Block scans give each thread's first slot.
  uint32_t gt = 0, eq = 0;
  count(theta, gt, eq);
  uint32_t total;
  const uint32_t gt_before = block_exclusive_scan<NT>(gt, scan_scratch, &total);
  const uint32_t eq_before = block_exclusive_scan<NT>(eq, scan_scratch, &total);
  emit(theta, need, eq_before, gt_before + (eq_before < need ? eq_before : need));
}

// Words of LDS that stage a chunk of T scores: one pad word after every 32,
// so that threads reading their own contiguous spans (a stride of `per`
// words between lanes) spread over the banks.
__host__ __device__ constexpr int64_t select_stage_words(int64_t T) { return T + (T >> 5) + 1; }
__device__ __forceinline__ int stage_slot(int p) { return p + (p >> 5); }
// Scores per LDS chunk in the ordered passes of long rows.
constexpr int kLongChunk = 16384;

// Select `keep` of the T scores in `row` into out[0..keep), ascending, for
// rows too long to hold in registers.  All NT threads of the workgroup call
// it; `work` holds SelectLds<NT>::kWords words of LDS.  Thread i owns the
// contiguous positions [i*per, (i+1)*per), per = ceil(T / NT).  Every pass
// re-reads the scores from global memory (L2): the digit passes read the row
// coalesced; the ordered passes walk each thread's span, either eight keys at
// a time from L2 (`stage` unused) or, with STAGE_LONG (`stage` holds
// select_stage_words(kLongChunk) words), from chunks of kLongChunk scores
// staged through LDS with coalesced loads.
template <int NT, bool STAGE_LONG = false>
__device__ __forceinline__ void select_unit(const float* __restrict__ row, int T, int keep,
                                            int32_t* __restrict__ out, uint32_t* work,
                                            uint32_t* stage) {
  const int tid = threadIdx.x;
  const int per = (T + NT - 1) / NT;
  const int lo = tid * per < T ? tid * per : T;
  const int hi = lo + per < T ? lo + per : T;
  const int n = hi - lo;

  auto at = [&](int j) { return row + (lo + j < T ? lo + j : T - 1); };

  // The digit passes read the row coalesced, in 16-byte loads
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

typedef uint32_t v4u32 __attribute__((ext_vector_type(4)));

// Number of set bits of m at lanes below this one.
__device__ __forceinline__ uint32_t lanes_below(uint64_t m) {
  return __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
}

// Rows of up to 4*KV*NT scores held in registers as 16-byte vectors, read
// once, coalesced, straight from global memory: thread i owns the vectors
// j*NT + i (j < KV), that is positions 4*(j*NT + i) .. 4*(j*NT + i) + 3.
// Position order is therefore (j, wave, lane, element).
//
// The first histogram buffer is cleared before the loads are issued, so the
// first digit pass starts on the keys that have arrived while the rest are
// in flight.  After the threshold, each wave counts per j the keys it takes
// with ballots, one wave scans those counts in (j, wave) order, and every
// taken key is stored at its output slot: the prefix of its (j, wave) plus
// the taken keys of the lanes below it (mbcnt) and of its own earlier
// elements.  When every key equal to theta is taken (the usual case: a
// unique threshold) a key is taken iff key >= theta, one flag; otherwise
// the first `need` keys equal to theta in position order are taken, which
// needs the count of keys above theta and of keys equal to it separately.
//
// A row may be split over `parts` workgroups (SelectPart): each holds its
// part (positions pos0 .. pos0 + T - 1 of the row; every part but the last
// is full, so padding only ever follows the row's last position), and the
// digit counts of every pass are summed over the parts through global
// memory.  Before the output each part adds the keys above and equal to
// theta of the parts before it, which those counts already hold: a key is
// above theta iff in some pass it matched the prefix so far and had a larger
// digit, and equal iff it matched the last pass's digit.
struct SelectPart {
  int parts, part;        // parts == 1: the whole row, no exchange
  int pos0;               // row position of this part's first score
  uint32_t* counters;     // [kSelCounters] per unit, zero at launch: arrivals per exchange
  uint32_t* hist;         // [4][parts][256] per unit: digit counts of each pass and part
  uint32_t* err;          // raised by a wait that gives up
  uint32_t spin_limit;    // polls before a wait gives up
};
constexpr int kSelCounters = 8;

// Device-scope hand-over: relaxed agent-scope atomics (coherent across the
// XCDs' L2s); a writer's stores complete before it counts itself in.
__device__ __forceinline__ uint32_t sel_poll(const uint32_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void sel_put2(uint32_t* p, uint32_t a, uint32_t b) {
  __hip_atomic_store(reinterpret_cast<uint64_t*>(p), (uint64_t)a | ((uint64_t)b << 32),
                     __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint64_t sel_get2(const uint32_t* p) {
  return __hip_atomic_load(reinterpret_cast<const uint64_t*>(p), __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
}
// Adds words [4*lane, 4*lane+4) (stride 256 words per part) of parts
// [p0, p1) into c, four parts' loads in flight at a time.
__device__ __forceinline__ void sel_sum_parts(const uint32_t* base, int p0, int p1, int lane,
                                              uint32_t (&c)[4]) {
  constexpr int kBatch = 4;
  for (int b0 = p0; b0 < p1; b0 += kBatch) {
    uint64_t v[kBatch][2];
#pragma unroll
    for (int b = 0; b < kBatch; ++b)
      if (b0 + b < p1) {
        v[b][0] = sel_get2(base + (size_t)(b0 + b) * 256 + 4 * lane);
        v[b][1] = sel_get2(base + (size_t)(b0 + b) * 256 + 4 * lane + 2);
      }
#pragma unroll
    for (int b = 0; b < kBatch; ++b)
      if (b0 + b < p1) {
        c[0] += (uint32_t)v[b][0];
        c[1] += (uint32_t)(v[b][0] >> 32);
        c[2] += (uint32_t)v[b][1];
        c[3] += (uint32_t)(v[b][1] >> 32);
      }
  }
}
// Wave 0: count this part in at exchange x and wait for all parts.  False if
// the wait gave up (after spin_limit polls, or when another wait already
// raised the error word).
__device__ __forceinline__ bool sel_arrive_wait(const SelectPart& sp, int x) {
  __builtin_amdgcn_s_waitcnt(0);   // this wave's stores of the exchange are complete
  int ok = 1;
  if ((threadIdx.x & 63) == 0) {
    __hip_atomic_fetch_add(sp.counters + x, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    uint32_t n = 0;
    while (sel_poll(sp.counters + x) < (uint32_t)sp.parts) {
      if (n >= sp.spin_limit || ((n & 63u) == 0 && sel_poll(sp.err) != 0u)) {
        __hip_atomic_fetch_or(sp.err, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        ok = 0;
        break;
      }
      ++n;
      __builtin_amdgcn_s_sleep(2);
    }
  }
  return __shfl(ok, 0) != 0;
}

template <int NT, int KV, bool SPLIT = false>
__device__ __forceinline__ void select_unit_vec(const float* __restrict__ row, int T, int keep,
                                                int32_t* __restrict__ out, uint32_t* work,
                                                const SelectPart* sp = nullptr) {
  constexpr int kWaves = NT / 64;
  constexpr int E = KV * kWaves;            // (j, wave) count entries
  static_assert(2 * E + 2 <= kWaves * 256, "count tables exceed the free histogram buffer");
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int first = 4 * tid;                // position of (j = 0, element 0) in the part
  // Exchange outcome (split rows): 1 while every wait has ended in time.
  uint32_t* s_ok = work + 2 * kWaves * 256 + kWaves + 1 + 5;
  if (SPLIT && tid == 0) *s_ok = 1u;

  for (int i = tid; i < kWaves * 256; i += NT) work[i] = 0;
  __syncthreads();

  // Buffer loads: one per-lane offset and a scalar offset per j, so that no
  // 64-bit address per load is held in registers; loads past the row's
  // 4*T bytes return 0.
  const __amdgpu_buffer_rsrc_t rsrc =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(row), 0, 4 * T, 0x00020000);
  uint32_t key[KV][4];
  if ((T & 3) == 0 && (reinterpret_cast<uintptr_t>(row) & 15) == 0) {
#pragma unroll
    for (int j = 0; j < KV; ++j) {
      const v4u32 x = __builtin_amdgcn_raw_buffer_load_b128(rsrc, 16 * tid, 16 * j * NT, 0);
      key[j][0] = x[0];
      key[j][1] = x[1];
      key[j][2] = x[2];
      key[j][3] = x[3];
    }
  } else {
#pragma unroll
    for (int j = 0; j < KV; ++j)
#pragma unroll
      for (int e = 0; e < 4; ++e)
        key[j][e] = __builtin_amdgcn_raw_buffer_load_b32(rsrc, 16 * tid, 16 * j * NT + 4 * e, 0);
  }
  // Positions at or past T get key 0, the lowest key (that of NaN), and stay
  // in every count: they come after every real position, and keep <= T, so
  // the keep-th key in (key descending, position ascending) order is a real
  // one; theta and need are those of the real keys, and no padding key is
  // ever taken.  This spares a validity mask per key in every pass.
#pragma unroll
  for (int j = 0; j < KV; ++j)
#pragma unroll
    for (int e = 0; e < 4; ++e)
      key[j][e] = first + 4 * j * NT + e < T ? order_key(__uint_as_float(key[j][e])) : 0u;

  // Split rows: wave 0 publishes this part's counts of a pass, waits for
  // every part's, and sums them in part order.
  auto merge = [&](int pass, uint32_t (&c)[4]) {
    if constexpr (SPLIT) {
      uint32_t* h = sp->hist + (size_t)pass * sp->parts * 256;
      sel_put2(h + sp->part * 256 + 4 * lane, c[0], c[1]);
      sel_put2(h + sp->part * 256 + 4 * lane + 2, c[2], c[3]);
      if (!sel_arrive_wait(*sp, pass)) {
        if (lane == 0) *s_ok = 0u;
        return;   // the part's own counts: a consistent but unused threshold
      }
#pragma unroll
      for (int q = 0; q < 4; ++q) c[q] = 0u;
      sel_sum_parts(h, 0, sp->parts, lane, c);
    }
  };
  uint32_t theta, need, n_theta;
  radix_threshold<NT, true>(
      keep, work,
      [&](uint32_t* h, uint32_t prefix, uint32_t hi_mask, int shift) {
        // After the first passes only keys in the chosen bins still count,
        // usually few: a wave with none of them skips the key at the cost of
        // one compare.
        DigitRuns runs;
#pragma unroll
        for (int j = 0; j < KV; ++j)
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const bool m = (key[j][e] & hi_mask) == prefix;
            if (__ballot(m)) runs.add(h, (key[j][e] >> shift) & 255u, m);
          }
        runs.flush(h);
      },
      &theta, &need, &n_theta, merge);
  // Every key equal to theta is taken (then n_theta == need), or only the
  // first `need` of them.  Uniform across the workgroup.
  const bool all_ties = n_theta == need;

  // Counts per (j, wave), in the histogram buffer the threshold left free:
  // taken keys (all_ties), else keys above theta and keys equal to it.
  uint32_t* cgt = work;
  uint32_t* ceq = work + E;
#pragma unroll
  for (int j = 0; j < KV; ++j) {
    uint32_t ng = 0, ne = 0;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      if (all_ties) {
        ng += (uint32_t)__popcll(__ballot(key[j][e] >= theta));
      } else {
        ng += (uint32_t)__popcll(__ballot(key[j][e] > theta));
        ne += (uint32_t)__popcll(__ballot(key[j][e] == theta));
      }
    }
    if (lane == 0) {
      cgt[j * kWaves + wave] = ng;
      ceq[j * kWaves + wave] = ne;
    }
  }
  __syncthreads();
  if (wave == 0) {
    // Exclusive scan of both count tables in (j, wave) order: lane l holds
    // entries [l*PL, (l+1)*PL).
    constexpr int PL = (E + 63) / 64;
    uint32_t g[PL], q[PL], sg = 0, sq = 0;
#pragma unroll
    for (int i = 0; i < PL; ++i) {
      const int x = lane * PL + i;
      g[i] = x < E ? cgt[x] : 0u;
      q[i] = x < E ? ceq[x] : 0u;
      sg += g[i];
      sq += q[i];
    }
    uint32_t ig = sg, iq = sq;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const uint32_t og = __shfl_up(ig, off), oq = __shfl_up(iq, off);
      if (lane >= off) {
        ig += og;
        iq += oq;
      }
    }
    uint32_t rg = ig - sg, rq = iq - sq;
    if constexpr (SPLIT) {
      // The keys of the parts before this one come first in the row: their
      // counts above and equal to theta, from every pass's published digit
      // counts (all parts have published every pass once the last wait
      // ended).  Lane l holds digits 4l .. 4l+3.
      if (*s_ok != 0u) {
        uint32_t bg = 0, bq = 0;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          const uint32_t dk = (theta >> (24 - 8 * k)) & 255u;
          uint32_t c[4] = {0u, 0u, 0u, 0u};
          sel_sum_parts(sp->hist + (size_t)k * sp->parts * 256, 0, sp->part, lane, c);
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const uint32_t d = 4u * lane + q;
            bg += d > dk ? c[q] : 0u;
            if (k == 3) bq += d == dk ? c[q] : 0u;
          }
        }
#pragma unroll
        for (int off = 32; off >= 1; off >>= 1) {
          bg += __shfl_xor(bg, off);
          bq += __shfl_xor(bq, off);
        }
        if (all_ties) {   // the tables count taken keys, above and equal alike
          rg += bg + bq;
        } else {
          rg += bg;
          rq += bq;
        }
      }
    }
#pragma unroll
    for (int i = 0; i < PL; ++i) {
      const int x = lane * PL + i;
      if (x < E) {
        cgt[x] = rg;
        ceq[x] = rq;
      }
      rg += g[i];
      rq += q[i];
    }
  }
  __syncthreads();
  if (SPLIT && *s_ok == 0u) {
    // A wait gave up: this part's share of the unit's slots holds -1.
    const int lo = (int)((int64_t)keep * sp->part / sp->parts);
    const int hi = (int)((int64_t)keep * (sp->part + 1) / sp->parts);
    for (int i = lo + tid; i < hi; i += NT) out[i] = -1;
    return;
  }

  // Output.  The flags are recomputed here rather than kept from the count
  // loop: the empty asm hides that they are the same, so the compiler does
  // not hold every ballot of that loop in scalar registers; likewise the
  // positions come from an opaque copy of `first`.
  int at = first + (SPLIT ? sp->pos0 : 0);
  asm volatile("" : "+v"(theta), "+v"(need), "+v"(at));
  // (split rows: positions at or past the part's end hold padding keys, never
  // taken unless a wait gave up; they are not written then either)
  const int at_end = T + (SPLIT ? sp->pos0 : 0);
  if (all_ties) {
#pragma unroll
    for (int j = 0; j < KV; ++j) {
      bool t[4];
      uint32_t slot = cgt[j * kWaves + wave];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        t[e] = key[j][e] >= theta;
        slot += lanes_below(__ballot(t[e]));
      }
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const bool real = !SPLIT || at + 4 * j * NT + e < at_end;
        if (t[e] && slot < (uint32_t)keep && real) out[slot] = at + 4 * j * NT + e;
        slot += t[e];
      }
    }
  } else {
    // A key's slot is (keys above theta before it) + min(keys equal to theta
    // before it, need).
#pragma unroll
    for (int j = 0; j < KV; ++j) {
      bool g[4], q[4];
      uint32_t gb = cgt[j * kWaves + wave], eb = ceq[j * kWaves + wave];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        g[e] = key[j][e] > theta;
        q[e] = key[j][e] == theta;
        gb += lanes_below(__ballot(g[e]));
        eb += lanes_below(__ballot(q[e]));
      }
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const uint32_t slot = gb + (eb < need ? eb : need);
        const bool real = !SPLIT || at + 4 * j * NT + e < at_end;
        if ((g[e] || (q[e] && eb < need)) && slot < (uint32_t)keep && real)
          out[slot] = at + 4 * j * NT + e;
        gb += g[e];
        eb += q[e];
      }
    }
  }
}
}  // namespace cb
