// Position-level variant of the persistent score kernel (second pass also
// accumulates the correction numerator), for fp32 inputs with head_dim 128.
#include "score_impl.h"

namespace cb {
template hipError_t launch_position_d<4, 128>(const ScorePlan&, PersistArgs&, hipStream_t);
}  // namespace cb
