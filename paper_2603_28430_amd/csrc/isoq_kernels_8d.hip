// Stage-1 kernels with 8-D grouped blocks (one 8x8 orthogonal matrix per 8
// coordinates) at the tuned widths; the template is in isoq_kernels.h, and
// this translation unit builds in parallel with the other variants'.
#include "isoq_kernels.h"

namespace isoq {

const void *kernel_for_block8(int d, int bits, bool f16, bool generic_sets, int mode)
{
    return pick_d<VAR_BLOCK8>(d, bits, f16, generic_sets, mode);
}

}  // namespace isoq
