// assign_smallk_f16.hip -- the small-K Lloyd step in one pass (assignment
// plus one-hot MFMA cluster sums) and the update's sums, for f16 points.
#include "assign_smallk.h"

namespace fkm {

hipError_t launch_sums_f16(const void* X, const Workspace& w, int64_t B, int64_t N, int64_t D,
                         int64_t K, int mode, int32_t* idx, float* min_dist, hipStream_t s) {
  return launch_sums_dt<DT_F16>(X, w, B, N, D, K, mode, idx, min_dist, s);
}

}  // namespace fkm
