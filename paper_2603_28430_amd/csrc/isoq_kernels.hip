// IsoQuant stage-1 kernels for gfx950 (MI355X).
//
// One template covers the three entry points of Algorithm 1:
//   MODE_ROUNDTRIP   x -> x_hat fused (norm, rotation, quantizer, inverse)
//   MODE_QUANTIZE    x -> packed indices + rho
//   MODE_DEQUANTIZE  packed indices + rho -> x_hat
//   MODE_APPEND      quantize (token, head) rows into the slots of a paged
//                    K/V cache: blockIdx.x is the head, blockIdx.y the token
//                    range, blockIdx.z selects K or V
//
// Mapping.  A lane owns 8 coordinates of one row: two 4-coordinate slots,
// each a quaternion block (Full/Fast, Sec. 5.2-5.3) or two planar pairs
// (Sec. 5.4), so the rotation never leaves the lane.  fp16 rows: slots 2s and
// 2s + 1, 16 bytes (one global_load_dwordx4); fp32 rows: slots s and
// s + d/8 in the round trip, quantize and dequantize (two 16-byte accesses
// that each cover a dense span across the wave), adjacent slots in append.
// A row spans d/8 lanes (8, 16, 32 or 64) and a wave holds 512/d rows; the
// squared norm is reduced with DPP row operations inside each 16-lane row and
// with permlane swaps across rows.  Every lane keeps the parameters of its own blocks in
// VGPRs for the whole kernel; the codebook sits in kernel-argument SGPRs.
//
// Blocks are not persistent: each owns a tile of consecutive row groups,
// issues all of the tile's loads together, then computes and stores group by
// group (see Stage1::tile).  The path is bound by HBM bandwidth, so the
// arithmetic is plain fp32 VALU work and uses no MFMA.
//
// Quantizer (shared b-bit codebook, symmetric): the rotated value y of the
// unnormalised row is compared with rho' t_k (rho' = max(rho, 1e-12)), which
// equals comparing y / rho' with t_k; the magnitude index m counts the
// positive thresholds below |y|, the sign decision is y > 0 (the middle
// threshold t_{K/2-1} = 0), and the selected level is pre-multiplied by rho so
// that the inverse rotation directly yields rho * rec (Algorithm 1, last step).
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

const void *kernel_for(int variant, int d, int bits, bool f16, bool generic_sets, int mode)
{
    switch (variant) {
    case VAR_FULL: return pick_d<VAR_FULL>(d, bits, f16, generic_sets, mode);
    case VAR_FAST: return pick_d<VAR_FAST>(d, bits, f16, generic_sets, mode);
    case VAR_PLANAR2D: return pick_d<VAR_PLANAR2D>(d, bits, f16, generic_sets, mode);
    }
    return nullptr;
}

}  // namespace isoq
