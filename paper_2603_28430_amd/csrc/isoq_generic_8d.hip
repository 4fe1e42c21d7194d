// Stage-1 kernels with 8-D grouped blocks for widths outside {64, 128, 256, 512}
// (8-coordinate slots; the template is in isoq_generic.h).
#include "isoq_generic.h"

namespace isoq {

const void *generic_kernel_8d(int slots, int bits, bool f16, int mode, bool pairs)
{
    return gen_pick<VAR_BLOCK8>(slots, bits, f16, mode, pairs);
}

}  // namespace isoq
