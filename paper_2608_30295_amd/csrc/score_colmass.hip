// Column-mass pass of the score kernels (pass 2 of the selection): the
// group-mean attention mass of every key column, or with a chunk size that
// divides the 64-column tile its chunk maxima (BlockMax) directly.
#include "score.h"

namespace catekv {

hipError_t launch_score_colmass(int dtype, int rows_pad, dim3 grid, hipStream_t s, const ScoreArgs& a) {
  return dtype == CATEKV_BF16 ? launch_score_mt<uint16_t, kColMass, 0, false>(rows_pad, grid, s, a)
                              : launch_score_mt<float, kColMass, 0, false>(rows_pad, grid, s, a);
}

}  // namespace catekv
