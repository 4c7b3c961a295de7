// Internal interface of the position-level selector kernels (position.hip).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace cb {

// After the position variant of the score kernel: Q, C and S per sender and
// position.
struct PositionFinish {
  const float* importance;   // [U][T]
  const float* numer;        // [U][T], the score kernel's numerator terms
  double* qpre;              // [S][T] workspace
  double* corr64;            // [S][T] workspace
  float* score;              // [S][T]
  float* qscore;             // [S][T] or null
  float* corr;               // [S][T] or null
  int64_t T;
  int S, LH, m, G, Hq;
  int pow_mode;
  double p, alpha, num_scale;
};
hipError_t launch_position_finish(const PositionFinish& f, hipStream_t s);

// Span rule per sender: rem = budget - forced positions (>= 0); writes
// out_count = min(budget, T) positions per sender.  keys: [S][ceil(T/width)].
hipError_t launch_spans(const float* score, int64_t S, int64_t T, int width, int64_t n_latent,
                        int64_t rem, int64_t out_count, uint64_t* keys, int32_t* idx,
                        hipStream_t s);

// out[s*count + j][:] = rows[s][idx[s*count + j]][:]; row_bytes % 4 == 0.
hipError_t launch_gather_rows(const void* rows, int64_t S, int64_t T, int64_t row_bytes,
                              const int32_t* idx, int64_t count, void* out, hipStream_t s);

}  // namespace cb
