// Per-unit top-k kernels (gfx950) running the radix select of
// select_impl.h, one workgroup per unit.
//
// select_kernel: 1024 threads, keys held in registers for T <= 32768.  The
// fastest form when it has the GPU to itself (cb_select).
//
// select_light_kernel: 256 threads and about 4 KiB of LDS, keys in registers
// for T <= 8192.  Small enough to be resident next to two score workgroups
// on a CU, so that in cb_pipeline the selection of one unit group runs while
// later groups are being scored.
//
// Longer rows re-read the scores from L2 on every digit pass.
#include "kernels.h"
#include "select_impl.h"

namespace cb {
namespace {

constexpr int kThreads = 1024;
constexpr int kKeysPerThread = 32;

__global__ __launch_bounds__(kThreads) void select_kernel(const float* __restrict__ importance,
                                                          int64_t T64, int64_t keep64,
                                                          int32_t* __restrict__ idx) {
  __shared__ uint32_t work[SelectLds<kThreads>::kWords];
  const int T = (int)T64;
  const int keep = (int)keep64;
  const int u = blockIdx.x;
  select_unit<kThreads, kKeysPerThread>(importance + (size_t)u * T, T, keep,
                                        idx + (size_t)u * keep, work);
}

constexpr int kLightThreads = 256;

__global__ __launch_bounds__(kLightThreads) void select_light_kernel(
    const float* __restrict__ importance, int64_t T64, int64_t keep64,
    int32_t* __restrict__ idx) {
  __shared__ uint32_t work[SelectLds<kLightThreads>::kWords];
  const int T = (int)T64;
  const int keep = (int)keep64;
  const int u = blockIdx.x;
  select_unit<kLightThreads, kKeysPerThread>(importance + (size_t)u * T, T, keep,
                                             idx + (size_t)u * keep, work);
}

}  // namespace

hipError_t launch_select_light(const float* importance, int64_t units, int64_t T, int64_t keep,
                               int32_t* idx, hipStream_t s) {
  select_light_kernel<<<(unsigned)units, kLightThreads, 0, s>>>(importance, T, keep, idx);
  return hipGetLastError();
}

hipError_t launch_select(const float* importance, int64_t units, int64_t T, int64_t keep,
                         int32_t* idx, hipStream_t s) {
  select_kernel<<<(unsigned)units, kThreads, 0, s>>>(importance, T, keep, idx);
  return hipGetLastError();
}

}  // namespace cb
