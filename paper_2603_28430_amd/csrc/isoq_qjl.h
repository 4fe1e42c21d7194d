// Quantize with the stage-2 residual sketch (Sec. 8): the stage-1 encoder of
// isoq_stage1.h in MODE_QJL (rows in, rows out) or MODE_APPEND_QJL (token
// rows into the slots of a paged cache), which also writes
// sign(S (x - x_hat)) as m bits and ||x - x_hat|| per row.  The projection is the path's one dense
// contraction, P = E S'^T over a wave's tile of rows, on MFMA (fp16 inputs,
// fp32 accumulation); S' = S T^{-1} per rotation set is staged in LDS once
// per block.
#pragma once

#include <hip/hip_runtime.h>

#include <type_traits>

#include "isoq_stage1.h"

namespace isoq {
namespace {

template <int VAR, int D, int BITS, bool F16, int QM, int MODE>
__global__ __launch_bounds__(kBlockThreads) void qjl_kernel(const KArgs a)
{
    using S = Stage1<VAR, D, BITS, F16, MODE, false, QM>;
    __shared__ float lds_levels[16];
    __shared__ __align__(16) float lds_params[S::LPV * S::PL];
    __shared__ __align__(16) LutEntry lds_lut[S::kUseLut ? kLutMaxCells : 1];
    __shared__ __align__(16) _Float16 lds_frag[QM * D];
    __shared__ __align__(16) _Float16 lds_e[(kBlockThreads / 64) * S::kTileRows * S::kEStride];
    S::run(a, lds_levels, lds_params, lds_lut, lds_frag, lds_e);
}

template <int VAR, int D, int BITS, bool F16, int MODE>
const void *qjl_pick_m(int m)
{
    if constexpr (D <= 128) {
        if (m == 64)
            return reinterpret_cast<const void *>(&qjl_kernel<VAR, D, BITS, F16, 64, MODE>);
        if (m == 128)
            return reinterpret_cast<const void *>(&qjl_kernel<VAR, D, BITS, F16, 128, MODE>);
    } else {
        if (m == 64)
            return reinterpret_cast<const void *>(&qjl_kernel<VAR, D, BITS, F16, 64, MODE>);
    }
    return nullptr;
}

template <int VAR, int D, int MODE>
const void *qjl_pick_bits(int bits, bool f16, int m)
{
    switch (bits) {
    case 2: return f16 ? qjl_pick_m<VAR, D, 2, true, MODE>(m) : qjl_pick_m<VAR, D, 2, false, MODE>(m);
    case 3: return f16 ? qjl_pick_m<VAR, D, 3, true, MODE>(m) : qjl_pick_m<VAR, D, 3, false, MODE>(m);
    case 4: return f16 ? qjl_pick_m<VAR, D, 4, true, MODE>(m) : qjl_pick_m<VAR, D, 4, false, MODE>(m);
    }
    return nullptr;
}

template <int MODE>
const void *qjl_pick(int variant, int d, int bits, bool f16, int m)
{
    auto by_d = [&](auto var) -> const void * {
        constexpr int V = decltype(var)::value;
        switch (d) {
        case 64: return qjl_pick_bits<V, 64, MODE>(bits, f16, m);
        case 128: return qjl_pick_bits<V, 128, MODE>(bits, f16, m);
        case 256: return qjl_pick_bits<V, 256, MODE>(bits, f16, m);
        }
        return nullptr;
    };
    switch (variant) {
    case VAR_FULL: return by_d(std::integral_constant<int, VAR_FULL>{});
    case VAR_FAST: return by_d(std::integral_constant<int, VAR_FAST>{});
    case VAR_PLANAR2D: return by_d(std::integral_constant<int, VAR_PLANAR2D>{});
    }
    return nullptr;
}

}  // namespace
}  // namespace isoq
