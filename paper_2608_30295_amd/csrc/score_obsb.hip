// Bracketing pass of CV scoring: the observation-matrix pass with A's values
// classified against the sampled bracket instead of stored.
#include "score.h"

namespace catekv {

hipError_t launch_score_obs_bracket(int dtype, int G, bool causal, int rows_pad, dim3 grid, hipStream_t s,
                                    const ScoreArgs& a) {
  const bool bf = dtype == CATEKV_BF16;
#define CATEKV_SC(GG) \
  if (G == GG) { \
    if (causal) return bf ? launch_score_mt<uint16_t, kObsBracket, GG, true>(rows_pad, grid, s, a) \
                          : launch_score_mt<float, kObsBracket, GG, true>(rows_pad, grid, s, a); \
    return bf ? launch_score_mt<uint16_t, kObsBracket, GG, false>(rows_pad, grid, s, a) \
              : launch_score_mt<float, kObsBracket, GG, false>(rows_pad, grid, s, a); \
  }
  CATEKV_SC(1) CATEKV_SC(2) CATEKV_SC(4) CATEKV_SC(8)
#undef CATEKV_SC
  return hipErrorInvalidValue;
}

}  // namespace catekv
