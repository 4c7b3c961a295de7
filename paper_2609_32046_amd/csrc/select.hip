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

}  // namespace

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
