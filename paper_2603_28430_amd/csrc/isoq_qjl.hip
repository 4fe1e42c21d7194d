// Quantize with the stage-2 sketch, rows in and rows out (the kernel is in
// isoq_qjl.h); also the dispatch of both sketch kernels.
#include "isoq_qjl.h"

namespace isoq {

const void *qjl_append_kernel_for(int variant, int d, int bits, bool f16, int m, int waves);

const void *qjl_kernel_for(int variant, int d, int bits, bool f16, int m, bool append, int waves)
{
    if (append)
        return qjl_append_kernel_for(variant, d, bits, f16, m, waves);
    return qjl_pick<MODE_QJL>(variant, d, bits, f16, m, waves);
}

}  // namespace isoq
