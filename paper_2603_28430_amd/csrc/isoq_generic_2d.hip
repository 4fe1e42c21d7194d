// Stage-1 kernels of the 2-D planar case for widths outside {64, 128, 256, 512} (the
// template is in isoq_generic.h; one file per variant so they build in parallel).
#include "isoq_generic.h"

namespace isoq {

const void *generic_kernel_2d(int slots, int bits, bool f16, int mode, bool pairs)
{
    return gen_pick<VAR_PLANAR2D>(slots, bits, f16, mode, pairs);
}

}  // namespace isoq
