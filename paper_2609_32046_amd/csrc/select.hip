// Per-unit top-k kernels (gfx950) running the radix select of
// select_impl.h, one workgroup per unit.
//
// Rows of up to 65536 scores are read once into registers, four scores per
// 16-byte vector and KV vectors per thread (select_unit_vec), in the
// workgroup size measured fastest for each length on MI355X: 512 threads
// with KV = 1 or 2 up to 4096 scores, 1024 with KV = 2 up to 8192, 512 with
// KV = 8 up to 16384 (four workgroups fit a compute unit), 1024 with KV = 8
// or 16 up to 65536.  Longer rows re-read the
// scores from L2 on every digit pass; when there are fewer units than
// compute units they run in 1024-thread workgroups (the extra threads per
// unit are otherwise idle hardware) whose ordered passes read the row
// through LDS in chunks, else in 512-thread ones that read each thread's
// span from L2.
#include <atomic>

#include "kernels.h"
#include "select_impl.h"

namespace cb {
namespace {

template <int NT, bool STAGE_LONG>
__global__ __launch_bounds__(NT) void select_kernel(const float* __restrict__ importance,
                                                    int64_t T64, int64_t keep64,
                                                    int32_t* __restrict__ idx,
                                                    const uint32_t* __restrict__ err) {
  __shared__ __align__(16) uint32_t work[SelectLds<NT>::kWords];
  extern __shared__ uint32_t stage[];
  const int T = (int)T64;
  const int keep = (int)keep64;
  const int u = blockIdx.x;
  if (err && *err != 0u) {   // the scores are not valid: no selection
    for (int i = threadIdx.x; i < keep; i += NT) idx[(size_t)u * keep + i] = -1;
    return;
  }
  select_unit<NT, STAGE_LONG>(importance + (size_t)u * T, T, keep, idx + (size_t)u * keep, work, stage);
}

template <int NT, int KV>
__global__ __launch_bounds__(NT) void select_vec_kernel(const float* __restrict__ importance,
                                                        int64_t T64, int64_t keep64,
                                                        int32_t* __restrict__ idx,
                                                        const uint32_t* __restrict__ err) {
  __shared__ __align__(16) uint32_t work[SelectLds<NT>::kWords];
  const int T = (int)T64;
  const int keep = (int)keep64;
  const int u = blockIdx.x;
  if (err && *err != 0u) {   // the scores are not valid: no selection
    for (int i = threadIdx.x; i < keep; i += NT) idx[(size_t)u * keep + i] = -1;
    return;
  }
  select_unit_vec<NT, KV>(importance + (size_t)u * T, T, keep, idx + (size_t)u * keep, work);
}

// One part of a split row per workgroup: unit blockIdx.x / parts, part
// blockIdx.x % parts.
struct SplitArgs {
  const float* importance;
  int64_t T, keep;
  int32_t* idx;
  uint32_t* counters;
  uint32_t* data;
  uint32_t* err;
  uint32_t spin_limit;
  int parts, part_len;
  int64_t data_words;   // per unit
};

template <int KV>
__global__ __launch_bounds__(1024) void select_split_kernel(SplitArgs a) {
  __shared__ __align__(16) uint32_t work[SelectLds<1024>::kWords];
  const int T = (int)a.T;
  const int keep = (int)a.keep;
  const int u = blockIdx.x / a.parts;
  const int part = blockIdx.x % a.parts;
  int32_t* out = a.idx + (size_t)u * keep;
  if (__hip_atomic_load(a.err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0u) {
    // the scores are not valid, or another part's wait gave up
    const int lo = (int)((int64_t)keep * part / a.parts);
    const int hi = (int)((int64_t)keep * (part + 1) / a.parts);
    for (int i = lo + (int)threadIdx.x; i < hi; i += 1024) out[i] = -1;
    return;
  }
  const int pos0 = part * a.part_len;
  const int len = T - pos0 < a.part_len ? T - pos0 : a.part_len;
  uint32_t* d = a.data + (size_t)u * a.data_words;
  const SelectPart sp{a.parts, part, pos0, a.counters + (size_t)u * kSelCounters, d, a.err,
                      a.spin_limit};
  select_unit_vec<1024, KV, true>(a.importance + (size_t)u * T + pos0, len, keep, out, work, &sp);
}

// p 16-byte aligned: 16-byte stores, then the n % 4 tail.
__global__ void fill_minus_one(int32_t* __restrict__ p, int64_t n) {
  const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  const int64_t n4 = n >> 2;
  int4* p4 = reinterpret_cast<int4*>(p);
  for (int64_t i = gid; i < n4; i += stride) p4[i] = make_int4(-1, -1, -1, -1);
  for (int64_t i = 4 * n4 + gid; i < n; i += stride) p[i] = -1;
}

__global__ void clear_words(uint32_t* __restrict__ p, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    p[i] = 0u;
}

// Compute units of the current device, queried once per device.
int compute_units() {
  static std::atomic<int> cache[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  int n = cache[dev].load(std::memory_order_relaxed);
  if (n == 0) {
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        n <= 0)
      n = 256;
    cache[dev].store(n, std::memory_order_relaxed);
  }
  return n;
}

// Workgroups of select_split_kernel<kv> resident at once on the current
// device, queried once per device and kv.
int64_t split_capacity(int kv) {
  static std::atomic<int> cache[64][3];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 0;
  const int ki = kv == 4 ? 0 : kv == 8 ? 1 : 2;
  int occ = cache[dev][ki].load(std::memory_order_relaxed);
  if (occ == 0) {
    const void* fn = kv == 4 ? reinterpret_cast<const void*>(&select_split_kernel<4>)
                   : kv == 8 ? reinterpret_cast<const void*>(&select_split_kernel<8>)
                             : reinterpret_cast<const void*>(&select_split_kernel<16>);
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&occ, fn, 1024, 0) != hipSuccess || occ < 0)
      occ = 0;
    cache[dev][ki].store(occ > 0 ? occ : -1, std::memory_order_relaxed);
  }
  return occ > 0 ? (int64_t)occ * compute_units() : 0;
}

}  // namespace

static_assert(kSelCounters == kSplitCounterWords, "split counters per unit");

bool select_split_plan(int64_t units, int64_t T, SelectSplit* sp) {
  *sp = SelectSplit{1, 0, 0, 0};
  if (units < 1 || T <= 4 * 8 * 512) return false;
  const int64_t pmax = kSplitGroups / units;
  if (pmax < 2) return false;
  for (int kv = 4; kv <= 16; kv *= 2) {
    const int64_t len = 4LL * kv * 1024;
    const int64_t parts = (T + len - 1) / len;
    if (parts > pmax) continue;
    if (parts < 2) return false;
    sp->parts = (int)parts;
    sp->kv = kv;
    sp->part_len = (int)len;
    sp->data_words_per_unit = (size_t)4 * parts * 256;
    return true;
  }
  return false;
}

bool select_split_fits(const SelectSplit& sp, int64_t units) {
  return sp.parts > 1 && units * sp.parts <= split_capacity(sp.kv);
}

hipError_t launch_select_split(const float* importance, int64_t units, int64_t T, int64_t keep,
                               int32_t* idx, const SelectSplit& sp, uint32_t* counters,
                               uint32_t* data, uint32_t* err, uint32_t spin_limit,
                               hipStream_t s) {
  const SplitArgs a{importance, T, keep, idx, counters, data, err, spin_limit,
                    sp.parts, sp.part_len, (int64_t)sp.data_words_per_unit};
  // Every slot starts at -1: once a wait gives up, the parts' rankings need
  // not agree, and a slot no part writes must still hold -1.
  const int64_t n = units * keep;
  const int64_t fw = (n / 4 + 255) / 256;
  const int64_t fb = fw < 1 ? 1 : fw < 1024 ? fw : 1024;
  fill_minus_one<<<(unsigned)fb, 256, 0, s>>>(idx, n);
  const unsigned g = (unsigned)(units * sp.parts);
  if (sp.kv == 4)
    select_split_kernel<4><<<g, 1024, 0, s>>>(a);
  else if (sp.kv == 8)
    select_split_kernel<8><<<g, 1024, 0, s>>>(a);
  else
    select_split_kernel<16><<<g, 1024, 0, s>>>(a);
  return hipGetLastError();
}

hipError_t launch_clear_words(uint32_t* p, int64_t n, hipStream_t s) {
  const int64_t blocks = (n + 255) / 256 < 1024 ? (n + 255) / 256 : 1024;
  clear_words<<<(unsigned)(blocks > 0 ? blocks : 1), 256, 0, s>>>(p, n);
  return hipGetLastError();
}

hipError_t launch_select(const float* importance, int64_t units, int64_t T, int64_t keep,
                         int32_t* idx, const uint32_t* err, hipStream_t s) {
  const unsigned g = (unsigned)units;
  if (T <= 4 * 1 * 512) {
    select_vec_kernel<512, 1><<<g, 512, 0, s>>>(importance, T, keep, idx, err);
  } else if (T <= 4 * 2 * 512) {
    select_vec_kernel<512, 2><<<g, 512, 0, s>>>(importance, T, keep, idx, err);
  } else if (T <= 4 * 2 * 1024) {
    select_vec_kernel<1024, 2><<<g, 1024, 0, s>>>(importance, T, keep, idx, err);
  } else if (T <= 4 * 8 * 512) {
    select_vec_kernel<512, 8><<<g, 512, 0, s>>>(importance, T, keep, idx, err);
  } else if (T <= 4 * 8 * 1024) {
    select_vec_kernel<1024, 8><<<g, 1024, 0, s>>>(importance, T, keep, idx, err);
  } else if (T <= 4 * 16 * 1024) {
    select_vec_kernel<1024, 16><<<g, 1024, 0, s>>>(importance, T, keep, idx, err);
  } else if (units < compute_units()) {
    // T > 65536: ceil(T / 1024) > 64 keys per thread; the ordered passes
    // stage chunks of the row in LDS.
    const size_t lds = (size_t)select_stage_words(kLongChunk) * 4;
    select_kernel<1024, true><<<g, 1024, lds, s>>>(importance, T, keep, idx, err);
  } else {
    select_kernel<512, false><<<g, 512, 0, s>>>(importance, T, keep, idx, err);
  }
  return hipGetLastError();
}

}  // namespace cb
