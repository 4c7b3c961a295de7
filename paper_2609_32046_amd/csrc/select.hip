// Per-unit top-k kernels (gfx950) running the radix select of
// select_impl.h, one workgroup per unit.
//
// Rows of up to 512*32 scores run in 512-thread workgroups: the row is
// staged once through LDS (dynamic shared memory, select_stage_words(T)
// words) and held in registers, KPT = 16 or 32 keys per thread, whichever is
// the smaller that covers the row.  Longer rows re-read the scores from L2
// on every digit pass; when there are fewer units than compute units they
// run in 1024-thread workgroups (the extra threads per unit are otherwise
// idle hardware) whose ordered passes read the row through LDS in chunks,
// else in 512-thread ones that read each thread's span from L2.
#include <atomic>

#include "kernels.h"
#include "select_impl.h"

namespace cb {
namespace {

template <int NT, int KPT, bool STAGE_LONG>
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
  select_unit<NT, KPT, STAGE_LONG>(importance + (size_t)u * T, T, keep, idx + (size_t)u * keep, work, stage);
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
  const int64_t per = (T + 511) / 512;
  if (per <= 16) {
    const size_t lds = (size_t)select_stage_words(T) * 4;
    select_kernel<512, 16, false><<<(unsigned)units, 512, lds, s>>>(importance, T, keep, idx, err);
  } else if (per <= 32) {
    const size_t lds = (size_t)select_stage_words(T) * 4;
    select_kernel<512, 32, false><<<(unsigned)units, 512, lds, s>>>(importance, T, keep, idx, err);
  } else if (units < compute_units()) {
    // T > 16384: ceil(T / 1024) > 16 keys per thread, so the L2 path runs;
    // its ordered passes stage chunks of the row in LDS.
    const size_t lds = (size_t)select_stage_words(kLongChunk) * 4;
    select_kernel<1024, 16, true><<<(unsigned)units, 1024, lds, s>>>(importance, T, keep, idx, err);
  } else {
    // per > 32: the L2 path, no staging buffer.
    select_kernel<512, 32, false><<<(unsigned)units, 512, 0, s>>>(importance, T, keep, idx, err);
  }
  return hipGetLastError();
}

}  // namespace cb
