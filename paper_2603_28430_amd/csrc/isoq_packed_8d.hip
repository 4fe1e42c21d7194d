// Packed-row stage-1 kernels (fp16 rows of width d = 16 k up to 504 outside
// the tuned four, and the K/V append at the head widths) with 8-D grouped
// blocks: each 8-coordinate chunk of a lane is one block (the template is in
// isoq_packed.h).
#include "isoq_packed.h"

namespace isoq {

const void *packed_kernel_8d(int bits, int mode, int chunks, int cache_lp)
{
    return packed_pick<VAR_BLOCK8>(bits, mode, chunks, cache_lp);
}

}  // namespace isoq
