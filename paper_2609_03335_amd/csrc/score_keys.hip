// Ranking keys of Eq. 12 (Sec. 3.5) for batches of candidate plans on
// gfx950: the scoring kernel of score_kernel.h in its key mode.
#include "score_kernel.h"

namespace wfp {

hipError_t launch_score_keys(const ScoreParams& sp, const int8_t* dev, const uint16_t* prio,
                             const uint8_t* flags, int64_t n_plans, wf_plan_key* keys,
                             const SearchArgs* search, hipStream_t stream) {
  return launch_all<true>(sp, dev, prio, flags, n_plans, keys, nullptr, search, stream);
}

}  // namespace wfp
