// Attention-logit kernels without the stage-2 sketch for Full, Fast and 2-D
// keys (the kernel template is in isoq_scores.h, the dispatch in
// isoq_scores_pick.h).
#include "isoq_scores_pick.h"

namespace isoq {

ScoreKernel score_kernel_for(int variant, int d, int bits, bool f16, int group)
{
    switch (variant) {
    case VAR_FULL: return pick_d<VAR_FULL>(d, bits, f16, group);
    case VAR_FAST: return pick_d<VAR_FAST>(d, bits, f16, group);
    case VAR_PLANAR2D: return pick_d<VAR_PLANAR2D>(d, bits, f16, group);
    case VAR_BLOCK8: return score_kernel_for_block8(d, bits, f16, group);
    }
    return {nullptr, 0};
}

}  // namespace isoq
