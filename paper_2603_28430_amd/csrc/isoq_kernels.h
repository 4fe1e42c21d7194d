// The stage-1 kernel entry points (round trip, quantize, dequantize, append)
// and the compile-time dispatch over width, bits, row type and mode, shared by
// the translation units that instantiate them for the rotation variants
// (isoq_kernels.hip: Full, Fast, 2-D; isoq_kernels_8d.hip: 8-D blocks).
#pragma once

#include <hip/hip_runtime.h>

#include "isoq_stage1.h"

namespace isoq {
namespace {

template <int VAR, int D, int BITS, bool F16, int MODE, bool GENERIC_SETS>
__global__ __launch_bounds__(kBlockThreads) void stage1_kernel(const KArgs a)
{
    using S = Stage1<VAR, D, BITS, F16, MODE, GENERIC_SETS>;
    __shared__ float lds_levels[16];
    __shared__ __align__(16) float lds_params[GENERIC_SETS ? 4 : S::LPV * S::PL];
    __shared__ __align__(16) LutEntry lds_lut[S::kUseLut && MODE != MODE_DEQUANTIZE ? kLutMaxCells : 1];
    S::run(a, lds_levels, lds_params, lds_lut);
}

// K and V in one launch: blockIdx.z = 0 encodes the keys, 1 the values;
// blockIdx.x is the head, whose parameter set the block stages once, and
// blockIdx.y the range of tokens.
template <int VAR, int D, int BITS, bool F16>
__global__ __launch_bounds__(kBlockThreads) void append_kernel(const KArgs k, const KArgs v)
{
    using S = Stage1<VAR, D, BITS, F16, MODE_APPEND, false>;
    __shared__ float lds_levels[16];
    __shared__ __align__(16) float lds_params[S::LPV * S::PL];
    __shared__ __align__(16) LutEntry lds_lut[S::kUseLut ? kLutMaxCells : 1];
    S::run(blockIdx.z == 0 ? k : v, lds_levels, lds_params, lds_lut);
}

template <int VAR, int D, int BITS, bool F16, bool GEN>
const void *pick_mode(int mode)
{
    switch (mode) {
    case MODE_APPEND: return GEN ? nullptr : reinterpret_cast<const void *>(&append_kernel<VAR, D, BITS, F16>);
    case MODE_ROUNDTRIP: return reinterpret_cast<const void *>(&stage1_kernel<VAR, D, BITS, F16, MODE_ROUNDTRIP, GEN>);
    case MODE_QUANTIZE: return reinterpret_cast<const void *>(&stage1_kernel<VAR, D, BITS, F16, MODE_QUANTIZE, GEN>);
    case MODE_DEQUANTIZE: return reinterpret_cast<const void *>(&stage1_kernel<VAR, D, BITS, F16, MODE_DEQUANTIZE, GEN>);
    }
    return nullptr;
}

template <int VAR, int D, int BITS>
const void *pick_dtype(bool f16, bool gen, int mode)
{
    if (f16)
        return gen ? pick_mode<VAR, D, BITS, true, true>(mode) : pick_mode<VAR, D, BITS, true, false>(mode);
    return gen ? pick_mode<VAR, D, BITS, false, true>(mode) : pick_mode<VAR, D, BITS, false, false>(mode);
}

template <int VAR, int D>
const void *pick_bits(int bits, bool f16, bool gen, int mode)
{
    switch (bits) {
    case 2: return pick_dtype<VAR, D, 2>(f16, gen, mode);
    case 3: return pick_dtype<VAR, D, 3>(f16, gen, mode);
    case 4: return pick_dtype<VAR, D, 4>(f16, gen, mode);
    }
    return nullptr;
}

template <int VAR>
const void *pick_d(int d, int bits, bool f16, bool gen, int mode)
{
    switch (d) {
    case 64: return pick_bits<VAR, 64>(bits, f16, gen, mode);
    case 128: return pick_bits<VAR, 128>(bits, f16, gen, mode);
    case 256: return pick_bits<VAR, 256>(bits, f16, gen, mode);
    case 512: return pick_bits<VAR, 512>(bits, f16, gen, mode);
    }
    return nullptr;
}

}  // namespace
}  // namespace isoq
