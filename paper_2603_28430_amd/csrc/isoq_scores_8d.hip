// Attention-logit kernels for keys quantized with 8-D grouped blocks (the
// kernel template is in isoq_scores.h, the dispatch in isoq_scores_pick.h).
#include "isoq_scores_pick.h"

namespace isoq {

ScoreKernel score_kernel_for_block8(int d, int bits, bool f16, int group)
{
    return pick_d<VAR_BLOCK8>(d, bits, f16, group);
}

}  // namespace isoq
