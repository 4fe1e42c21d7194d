// Stage-1 kernels of IsoQuant-Fast for widths outside {64, 128, 256, 512} (the
// template is in isoq_generic.h; one file per variant so they build in parallel).
#include "isoq_generic.h"

namespace isoq {

const void *generic_kernel_fast(int slots, int bits, bool f16, int mode, bool pairs)
{
    return gen_pick<VAR_FAST>(slots, bits, f16, mode, pairs);
}

}  // namespace isoq
