// Stage-1 packed-row kernels for fp16 rows of width d = 16 k up to 504
// outside the tuned four, and the K/V append at d = 96, 160 and 192 (the
// template is in isoq_packed.h).
#include "isoq_packed.h"

namespace isoq {

const void *packed_kernel_full(int bits, int mode, int chunks, int cache_lp)
{
    return packed_pick<VAR_FULL>(bits, mode, chunks, cache_lp);
}
const void *packed_kernel_fast(int bits, int mode, int chunks, int cache_lp)
{
    return packed_pick<VAR_FAST>(bits, mode, chunks, cache_lp);
}
const void *packed_kernel_2d(int bits, int mode, int chunks, int cache_lp)
{
    return packed_pick<VAR_PLANAR2D>(bits, mode, chunks, cache_lp);
}

}  // namespace isoq
