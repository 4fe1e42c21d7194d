// Quantize with the stage-2 residual sketch (Sec. 8): the stage-1 encoder of
// isoq_stage1.h in MODE_QJL, which also writes sign(S (x - x_hat)) as m bits
// and ||x - x_hat|| per row.  The projection is the path's one dense
// contraction, P = E S'^T over a wave's tile of rows, on MFMA (fp16 inputs,
// fp32 accumulation); S' = S T^{-1} per rotation set is staged in LDS once
// per block.
#include <hip/hip_runtime.h>

#include "isoq_stage1.h"

namespace isoq {
namespace {

template <int VAR, int D, int BITS, bool F16, int QM>
__global__ __launch_bounds__(kBlockThreads) void qjl_kernel(const KArgs a)
{
    using S = Stage1<VAR, D, BITS, F16, MODE_QJL, false, QM>;
    __shared__ float lds_levels[16];
    __shared__ __align__(16) float lds_params[S::LPV * S::PL];
    __shared__ __align__(16) LutEntry lds_lut[S::kUseLut ? kLutMaxCells : 1];
    __shared__ __align__(16) _Float16 lds_frag[QM * D];
    __shared__ __align__(16) _Float16 lds_e[(kBlockThreads / 64) * S::kTileRows * S::kEStride];
    S::run(a, lds_levels, lds_params, lds_lut, lds_frag, lds_e);
}

template <int VAR, int D, int BITS, bool F16>
const void *pick_m(int m)
{
    if constexpr (D == 128) {
        if (m == 64)
            return reinterpret_cast<const void *>(&qjl_kernel<VAR, D, BITS, F16, 64>);
        if (m == 128)
            return reinterpret_cast<const void *>(&qjl_kernel<VAR, D, BITS, F16, 128>);
    } else {
        if (m == 64)
            return reinterpret_cast<const void *>(&qjl_kernel<VAR, D, BITS, F16, 64>);
    }
    return nullptr;
}

template <int VAR, int D>
const void *pick_bits(int bits, bool f16, int m)
{
    switch (bits) {
    case 2: return f16 ? pick_m<VAR, D, 2, true>(m) : pick_m<VAR, D, 2, false>(m);
    case 3: return f16 ? pick_m<VAR, D, 3, true>(m) : pick_m<VAR, D, 3, false>(m);
    case 4: return f16 ? pick_m<VAR, D, 4, true>(m) : pick_m<VAR, D, 4, false>(m);
    }
    return nullptr;
}

template <int VAR>
const void *pick_d(int d, int bits, bool f16, int m)
{
    switch (d) {
    case 128: return pick_bits<VAR, 128>(bits, f16, m);
    case 256: return pick_bits<VAR, 256>(bits, f16, m);
    }
    return nullptr;
}

}  // namespace

const void *qjl_kernel_for(int variant, int d, int bits, bool f16, int m)
{
    switch (variant) {
    case VAR_FULL: return pick_d<VAR_FULL>(d, bits, f16, m);
    case VAR_FAST: return pick_d<VAR_FAST>(d, bits, f16, m);
    case VAR_PLANAR2D: return pick_d<VAR_PLANAR2D>(d, bits, f16, m);
    }
    return nullptr;
}

}  // namespace isoq
