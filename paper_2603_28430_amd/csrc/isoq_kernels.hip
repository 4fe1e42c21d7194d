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
#include "isoq_kernels.h"

namespace isoq {

const void *kernel_for(int variant, int d, int bits, bool f16, bool generic_sets, int mode)
{
    switch (variant) {
    case VAR_FULL: return pick_d<VAR_FULL>(d, bits, f16, generic_sets, mode);
    case VAR_FAST: return pick_d<VAR_FAST>(d, bits, f16, generic_sets, mode);
    case VAR_PLANAR2D: return pick_d<VAR_PLANAR2D>(d, bits, f16, generic_sets, mode);
    case VAR_BLOCK8: return kernel_for_block8(d, bits, f16, generic_sets, mode);
    }
    return nullptr;
}

}  // namespace isoq
