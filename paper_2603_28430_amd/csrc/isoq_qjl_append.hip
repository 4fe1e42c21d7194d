// Quantize-on-append with the stage-2 sketch: key rows of new tokens into
// the slots of a paged cache (the kernel is in isoq_qjl.h).
#include "isoq_qjl.h"

namespace isoq {

const void *qjl_append_kernel_for(int variant, int d, int bits, bool f16, int m, int waves)
{
    return qjl_pick<MODE_APPEND_QJL>(variant, d, bits, f16, m, waves);
}

}  // namespace isoq
