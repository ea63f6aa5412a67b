// knn_f16.hip -- KNN search for f16 rows.
#include "knn.h"

namespace fkm {

hipError_t launch_knn_f16(const void* Q, const void* R, int64_t B, int64_t M, int64_t N,
                         int64_t Din, int64_t D, int k, void* chat, float* cinit, int64_t Np,
                         int32_t* nbr_idx, float* nbr_dist, hipStream_t s) {
  return launch_knn_dt<DT_F16>(Q, R, B, M, N, Din, D, k, chat, cinit, Np, nbr_idx, nbr_dist, s);
}

}  // namespace fkm
