// assign_pipe_f16.hip -- the pipelined resident-X assignment for f16 points.
#include "assign_pipe.h"

namespace fkm {

hipError_t launch_pipe_f16(const void* X, const Workspace& w, int64_t B, int64_t N, int64_t D,
                          int32_t* idx, float* min_dist, hipStream_t s) {
  return launch_pipe_dt<DT_F16>(X, w, B, N, D, idx, min_dist, s);
}

}  // namespace fkm
