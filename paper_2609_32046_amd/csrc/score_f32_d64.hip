// Persistent score kernel instantiated for f32 inputs with head_dim 64.
#include "score_impl.h"

namespace cb {
template hipError_t launch_score_d<4, 64>(const ScorePlan&, PersistArgs&, hipStream_t);
}  // namespace cb
