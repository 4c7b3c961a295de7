// Persistent score kernel instantiated for bf16 inputs with head_dim 128.
#include "score_impl.h"

namespace cb {
template hipError_t launch_score_d<2, 128>(const ScorePlan&, PersistArgs&, hipStream_t);
}  // namespace cb
