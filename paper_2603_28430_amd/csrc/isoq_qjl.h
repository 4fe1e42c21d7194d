// Quantize with the stage-2 residual sketch (Sec. 8): the stage-1 encoder of
// isoq_stage1m.h (fp16 rows) or isoq_stage1.h (fp32 rows) in MODE_QJL (rows
// in, rows out) or MODE_APPEND_QJL (token rows into the slots of a paged
// cache), which also writes sign(S (x - x_hat)) as m bits and ||x - x_hat||
// per row.  The projection is the path's one dense contraction, P = E S'^T over a wave's tile of rows, on MFMA (fp16 inputs,
// fp32 accumulation); S' = S T^{-1} per rotation set is staged in LDS once
// per block.  Blocks have 8 waves, or 4 for quantize with several sets
// (WAVES, chosen by qjl_waves): at d = 128, m = 128 the staged projection
// (32 KB) and the waves' error tiles let three 4-wave blocks (12 waves) or
// two 8-wave blocks (16 waves) share a CU's LDS.
#pragma once

#include <hip/hip_runtime.h>

#include <type_traits>

#include "isoq_stage1.h"
#include "isoq_stage1m.h"

namespace isoq {
namespace {

// fp16 rows take the matrix-core encoder where quantize and append do (the
// quad layout of isoq_stage1m.h, so the records stay identical to theirs);
// fp32 rows and the 2-D case the VALU encoder.
template <int VAR, int D, int BITS, bool F16, int QM, int MODE, int WAVES>
__global__ __launch_bounds__(WAVES * 64) void qjl_kernel(const KArgs a)
{
    using S = Stage1<VAR, D, BITS, F16, MODE, false, QM, WAVES>;
    __shared__ __align__(16) LutEntry lds_lut[S::kUseLut ? kLutMaxCells : 1];
    __shared__ __align__(16) _Float16 lds_frag[QM * D];
    if constexpr (F16 && quad_layout(VAR, D, BITS)) {
        using M = Stage1M<VAR, D, BITS, MODE, QM, WAVES>;
        static_assert(M::kTileRows == S::kTileRows, "the two layouts tile rows alike");
        __shared__ __align__(16) u32x4 lds_par[M::kLdsWords];
        __shared__ __align__(16) _Float16 lds_e[WAVES * M::kTileRows * M::kEStride];
        __shared__ int64_t lds_crow[MODE == MODE_APPEND_QJL ? WAVES * M::kTileRows : 1];
        M::run(a, lds_lut, lds_par, lds_frag, lds_e, lds_crow);
    } else {
        __shared__ float lds_levels[16];
        __shared__ __align__(16) float lds_params[S::LPV * S::PL];
        __shared__ __align__(16) _Float16 lds_e[WAVES * S::kTileRows * S::kEStride];
        S::run(a, lds_levels, lds_params, lds_lut, lds_frag, lds_e);
    }
}

// Instantiated (m, waves): m = 64, and m = 128 at d <= 128, with 8 waves; with
// 4 waves as well for quantize into rows (several sets).  At d = 512 (m = 64)
// the staged projection takes 64 KB of LDS, so a CU holds one block.
template <int VAR, int D, int BITS, bool F16, int MODE>
const void *qjl_pick_m(int m, int waves)
{
    if (m == 64 && waves == 8)
        return reinterpret_cast<const void *>(&qjl_kernel<VAR, D, BITS, F16, 64, MODE, 8>);
    if constexpr (MODE == MODE_QJL) {
        if (m == 64 && waves == 4)
            return reinterpret_cast<const void *>(&qjl_kernel<VAR, D, BITS, F16, 64, MODE, 4>);
    }
    if constexpr (D <= 128) {
        if (m == 128 && waves == 8)
            return reinterpret_cast<const void *>(&qjl_kernel<VAR, D, BITS, F16, 128, MODE, 8>);
        if constexpr (MODE == MODE_QJL) {
            if (m == 128 && waves == 4)
                return reinterpret_cast<const void *>(&qjl_kernel<VAR, D, BITS, F16, 128, MODE, 4>);
        }
    }
    return nullptr;
}

template <int VAR, int D, int MODE>
const void *qjl_pick_bits(int bits, bool f16, int m, int waves)
{
    switch (bits) {
    case 2: return f16 ? qjl_pick_m<VAR, D, 2, true, MODE>(m, waves) : qjl_pick_m<VAR, D, 2, false, MODE>(m, waves);
    case 3: return f16 ? qjl_pick_m<VAR, D, 3, true, MODE>(m, waves) : qjl_pick_m<VAR, D, 3, false, MODE>(m, waves);
    case 4: return f16 ? qjl_pick_m<VAR, D, 4, true, MODE>(m, waves) : qjl_pick_m<VAR, D, 4, false, MODE>(m, waves);
    }
    return nullptr;
}

template <int MODE>
const void *qjl_pick(int variant, int d, int bits, bool f16, int m, int waves)
{
    auto by_d = [&](auto var) -> const void * {
        constexpr int V = decltype(var)::value;
        switch (d) {
        case 64: return qjl_pick_bits<V, 64, MODE>(bits, f16, m, waves);
        case 128: return qjl_pick_bits<V, 128, MODE>(bits, f16, m, waves);
        case 256: return qjl_pick_bits<V, 256, MODE>(bits, f16, m, waves);
        case 512: return qjl_pick_bits<V, 512, MODE>(bits, f16, m, waves);
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
