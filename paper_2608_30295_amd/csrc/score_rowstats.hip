// Row-statistics pass of the score kernels (pass 1): per query row, the
// maximum and the sum of exp(s - max) over one column block.
#include "score.h"

namespace catekv {

hipError_t launch_score_rowstats(int dtype, int G, bool causal, int rows_pad, dim3 grid, hipStream_t s,
                                 const ScoreArgs& a) {
  const bool bf = dtype == CATEKV_BF16;
  if (!causal) {
    // the group size only places Q rows here: one build per dtype
    return bf ? launch_score_mt<uint16_t, kRowStats, 0, false>(rows_pad, grid, s, a)
              : launch_score_mt<float, kRowStats, 0, false>(rows_pad, grid, s, a);
  }
#define CATEKV_SC(GG) \
  if (G == GG) return bf ? launch_score_mt<uint16_t, kRowStats, GG, true>(rows_pad, grid, s, a) \
                         : launch_score_mt<float, kRowStats, GG, true>(rows_pad, grid, s, a);
  CATEKV_SC(1) CATEKV_SC(2) CATEKV_SC(4) CATEKV_SC(8)
#undef CATEKV_SC
  return hipErrorInvalidValue;
}

}  // namespace catekv
