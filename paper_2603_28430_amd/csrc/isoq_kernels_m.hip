// Stage-1 encoders with the forward rotation on the matrix cores (the quad
// layout of isoq_stage1m.h): round trip, quantize and the K/V append for fp16
// rows at d = 64, 128 and 256: Full, Fast, 8-D blocks, and 2-D at 2 and 3
// bits.
#include <hip/hip_runtime.h>

#include "isoq_stage1m.h"

namespace isoq {
namespace {

template <int VAR, int D, int BITS, int MODE, bool STREAMS>
__device__ __forceinline__ void stage1m_body(const KArgs &a)
{
    using S = Stage1M<VAR, D, BITS, MODE, 0, 4, STREAMS>;
    __shared__ __align__(16) LutEntry lds_lut[S::kUseLut ? kLutMaxCells : 1];
    __shared__ __align__(16) u32x4 lds_par[S::kLdsWords];
    S::run(a, lds_lut, lds_par);
}

template <int VAR, int D, int BITS, int MODE, bool STREAMS>
__global__ __launch_bounds__(kBlockThreads) void stage1m_kernel(const KArgs a)
{
    stage1m_body<VAR, D, BITS, MODE, STREAMS>(a);
}

// Round trips built for more waves per SIMD than the compiler would size
// their registers for (0: no hint), where that fits without spilling and
// measured faster: Full at d = 256, 3 and 4 bits, 106-112 VGPRs (four waves)
// -> 96 at five, 4-5% and 2-3% faster; Fast at d = 256, 4 bits, 84 (five) ->
// 75 at six, 1.5% faster.  (Hints that fit at other widths and bit widths
// measured equal or slower; the 8-D round trips spill at five.)
template <int VAR, int D, int BITS>
constexpr int roundtrip_waves()
{
    if (VAR == VAR_FULL && D == 256 && BITS >= 3)
        return 5;
    if (VAR == VAR_FAST && D == 256 && BITS == 4)
        return 6;
    return 0;
}

template <int VAR, int D, int BITS, int MODE, bool STREAMS, int W>
__global__ __launch_bounds__(kBlockThreads) __attribute__((amdgpu_waves_per_eu(W))) void stage1m_kernel_w(
    const KArgs a)
{
    stage1m_body<VAR, D, BITS, MODE, STREAMS>(a);
}

template <int VAR, int D, int BITS>
__global__ __launch_bounds__(kBlockThreads) void append_m_kernel(const KArgs k, const KArgs v)
{
    using S = Stage1M<VAR, D, BITS, MODE_APPEND>;
    __shared__ __align__(16) LutEntry lds_lut[S::kUseLut ? kLutMaxCells : 1];
    __shared__ __align__(16) u32x4 lds_par[S::kLdsWords];
    S::run(blockIdx.z == 0 ? k : v, lds_lut, lds_par);
}

template <int VAR, int D, int BITS>
const void *m_mode(int mode)
{
    switch (mode) {
    case MODE_ROUNDTRIP:
        if constexpr (constexpr int W = roundtrip_waves<VAR, D, BITS>(); W > 0)
            return reinterpret_cast<const void *>(&stage1m_kernel_w<VAR, D, BITS, MODE_ROUNDTRIP, false, W>);
        else
            return reinterpret_cast<const void *>(&stage1m_kernel<VAR, D, BITS, MODE_ROUNDTRIP, false>);
    case MODE_QUANTIZE: return reinterpret_cast<const void *>(&stage1m_kernel<VAR, D, BITS, MODE_QUANTIZE, false>);
    case MODE_STREAMS_ROUNDTRIP:
        return reinterpret_cast<const void *>(&stage1m_kernel<VAR, D, BITS, MODE_ROUNDTRIP, true>);
    case MODE_STREAMS_QUANTIZE:
        return reinterpret_cast<const void *>(&stage1m_kernel<VAR, D, BITS, MODE_QUANTIZE, true>);
    case MODE_APPEND: return reinterpret_cast<const void *>(&append_m_kernel<VAR, D, BITS>);
    }
    return nullptr;
}

template <int VAR, int D>
const void *m_bits(int bits, int mode)
{
    switch (bits) {
    case 2: return m_mode<VAR, D, 2>(mode);
    case 3: return m_mode<VAR, D, 3>(mode);
    case 4:
        if constexpr (quad_layout(VAR, D, 4))
            return m_mode<VAR, D, 4>(mode);
        return nullptr;
    }
    return nullptr;
}

template <int VAR>
const void *m_d(int d, int bits, int mode)
{
    switch (d) {
    case 64: return m_bits<VAR, 64>(bits, mode);
    case 128: return m_bits<VAR, 128>(bits, mode);
    case 256: return m_bits<VAR, 256>(bits, mode);
    }
    return nullptr;
}

}  // namespace

const void *kernel_m_for(int variant, int d, int bits, int mode)
{
    switch (variant) {
    case VAR_FULL: return m_d<VAR_FULL>(d, bits, mode);
    case VAR_FAST: return m_d<VAR_FAST>(d, bits, mode);
    case VAR_PLANAR2D: return m_d<VAR_PLANAR2D>(d, bits, mode);
    case VAR_BLOCK8: return m_d<VAR_BLOCK8>(d, bits, mode);
    }
    return nullptr;
}

}  // namespace isoq
