// Packed-row kernels with the stage-2 sketch (the template is in
// isoq_packed.h): fp16 rows at d = 80, 96, 160 and 192, m = 64 or 128 sign
// bits, quantize into rows or append into the slots of a paged cache.
#include "isoq_packed.h"

namespace isoq {
namespace {

template <int VAR, int D, int BITS>
const void *packed_qjl_pick_m(int m, bool append)
{
    switch (m * 2 + (append ? 1 : 0)) {
    case 128: return reinterpret_cast<const void *>(&packed_qjl_kernel<VAR, D, BITS, MODE_QJL, 64>);
    case 129: return reinterpret_cast<const void *>(&packed_qjl_kernel<VAR, D, BITS, MODE_APPEND_QJL, 64>);
    case 256: return reinterpret_cast<const void *>(&packed_qjl_kernel<VAR, D, BITS, MODE_QJL, 128>);
    case 257: return reinterpret_cast<const void *>(&packed_qjl_kernel<VAR, D, BITS, MODE_APPEND_QJL, 128>);
    }
    return nullptr;
}

template <int VAR, int D>
const void *packed_qjl_pick_bits(int bits, int m, bool append)
{
    switch (bits) {
    case 2: return packed_qjl_pick_m<VAR, D, 2>(m, append);
    case 3: return packed_qjl_pick_m<VAR, D, 3>(m, append);
    case 4: return packed_qjl_pick_m<VAR, D, 4>(m, append);
    }
    return nullptr;
}

template <int VAR>
const void *packed_qjl_pick_d(int d, int bits, int m, bool append)
{
    switch (d) {
    case 80: return packed_qjl_pick_bits<VAR, 80>(bits, m, append);
    case 96: return packed_qjl_pick_bits<VAR, 96>(bits, m, append);
    case 160: return packed_qjl_pick_bits<VAR, 160>(bits, m, append);
    case 192: return packed_qjl_pick_bits<VAR, 192>(bits, m, append);
    }
    return nullptr;
}

}  // namespace

const void *packed_qjl_kernel_for(int variant, int d, int bits, int m, bool append)
{
    switch (variant) {
    case VAR_FULL: return packed_qjl_pick_d<VAR_FULL>(d, bits, m, append);
    case VAR_FAST: return packed_qjl_pick_d<VAR_FAST>(d, bits, m, append);
    case VAR_PLANAR2D: return packed_qjl_pick_d<VAR_PLANAR2D>(d, bits, m, append);
    }
    return nullptr;
}

}  // namespace isoq
