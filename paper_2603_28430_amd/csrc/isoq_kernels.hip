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
// Mapping.  A lane owns 8 consecutive coordinates of one row: 16 bytes of
// fp16 (one global_load_dwordx4) or 32 bytes of fp32 (two).  Those 8
// coordinates are two quaternion blocks (Full/Fast, Sec. 5.2-5.3) or four
// planar pairs (Sec. 5.4), so the rotation never leaves the lane.  A row spans
// d/8 lanes (16, 32 or 64) and a wave holds 512/d rows; the squared norm is
// reduced with DPP row operations inside each 16-lane row and with permlane
// swaps across rows.  Every lane keeps the parameters of its own blocks in
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

#include "isoq_device.h"
#include "isoq_internal.h"

namespace isoq {
namespace {

// ---- packed index records --------------------------------------------------
// Lane `sub` of a row owns coordinates 8 sub .. 8 sub + 7, i.e. bits
// [8 sub * BITS, 8 (sub + 1) * BITS) of the row's record: a 16-bit half-word
// (2 bits), a 32-bit word (4 bits), or 24 bits at byte 3 sub (3 bits), which
// the four lanes of a DPP quad merge into three aligned words.
template <int BITS>
__device__ __forceinline__ void store_bits(uint8_t *rec, int sub, uint32_t p, bool ok)
{
    if constexpr (BITS == 2) {
        if (ok)
            reinterpret_cast<uint16_t *>(rec)[sub] = (uint16_t)p;
    } else if constexpr (BITS == 4) {
        if (ok)
            reinterpret_cast<uint32_t *>(rec)[sub] = p;
    } else {
        // lane k of a quad holds bits [24 k, 24 k + 24) of 96; lanes 0..2
        // write word k = p_k >> 8 k | p_(k+1) << (24 - 8 k)
        const uint32_t nb = dpp_u<DPP_QUAD_1233>(p);  // bits of the next lane in the quad
        const int k = sub & 3;
        if (ok && k < 3)
            reinterpret_cast<uint32_t *>(rec)[3 * (sub >> 2) + k] = (p >> (8 * k)) | (nb << (24 - 8 * k));
    }
}

template <int BITS>
__device__ __forceinline__ uint32_t load_bits(const uint8_t *rec, int sub)
{
    if constexpr (BITS == 2) {
        return reinterpret_cast<const uint16_t *>(rec)[sub];
    } else if constexpr (BITS == 4) {
        return reinterpret_cast<const uint32_t *>(rec)[sub];
    } else {
        const uint32_t *q = reinterpret_cast<const uint32_t *>(rec + 12 * (sub >> 2));
        const uint32_t w0 = q[0], w1 = q[1], w2 = q[2];
        const int k = sub & 3;  // 24 k = 32 lo_word + shift
        const uint32_t lo = k < 2 ? w0 : (k == 2 ? w1 : w2);
        const uint32_t hi = k < 2 ? w1 : (k == 2 ? w2 : 0u);
        const int sh = (24 * k) & 31;
        return (uint32_t)((((uint64_t)hi << 32) | lo) >> sh) & 0xFFFFFFu;
    }
}

// Append the lane's bit of each mask to p, first mask first (p = 2 p + bit):
// v_addc_co_u32 with the mask as carry-in does the shift and the insert in one
// instruction.  The masks are written by VALU compares; a VALU read of an SGPR
// as carry-in needs wait states after such a write, which the compiler cannot
// insert inside an asm statement, so the block starts with s_nop 4.
__device__ __forceinline__ uint32_t push_bits8(uint32_t p, const uint64_t m[8])
{
    asm("s_nop 4\n\t"
        "v_addc_co_u32_e64 %0, vcc, %0, %0, %1\n\t"
        "v_addc_co_u32_e64 %0, vcc, %0, %0, %2\n\t"
        "v_addc_co_u32_e64 %0, vcc, %0, %0, %3\n\t"
        "v_addc_co_u32_e64 %0, vcc, %0, %0, %4\n\t"
        "v_addc_co_u32_e64 %0, vcc, %0, %0, %5\n\t"
        "v_addc_co_u32_e64 %0, vcc, %0, %0, %6\n\t"
        "v_addc_co_u32_e64 %0, vcc, %0, %0, %7\n\t"
        "v_addc_co_u32_e64 %0, vcc, %0, %0, %8"
        : "+v"(p)
        : "s"(m[0]), "s"(m[1]), "s"(m[2]), "s"(m[3]), "s"(m[4]), "s"(m[5]), "s"(m[6]), "s"(m[7])
        : "vcc");
    return p;
}

__device__ __forceinline__ uint32_t push_bits12(uint32_t p, const uint64_t m[12])
{
    asm("s_nop 4\n\t"
        "v_addc_co_u32_e64 %0, vcc, %0, %0, %1\n\t"
        "v_addc_co_u32_e64 %0, vcc, %0, %0, %2\n\t"
        "v_addc_co_u32_e64 %0, vcc, %0, %0, %3\n\t"
        "v_addc_co_u32_e64 %0, vcc, %0, %0, %4\n\t"
        "v_addc_co_u32_e64 %0, vcc, %0, %0, %5\n\t"
        "v_addc_co_u32_e64 %0, vcc, %0, %0, %6\n\t"
        "v_addc_co_u32_e64 %0, vcc, %0, %0, %7\n\t"
        "v_addc_co_u32_e64 %0, vcc, %0, %0, %8\n\t"
        "v_addc_co_u32_e64 %0, vcc, %0, %0, %9\n\t"
        "v_addc_co_u32_e64 %0, vcc, %0, %0, %10\n\t"
        "v_addc_co_u32_e64 %0, vcc, %0, %0, %11\n\t"
        "v_addc_co_u32_e64 %0, vcc, %0, %0, %12"
        : "+v"(p)
        : "s"(m[0]), "s"(m[1]), "s"(m[2]), "s"(m[3]), "s"(m[4]), "s"(m[5]), "s"(m[6]), "s"(m[7]),
          "s"(m[8]), "s"(m[9]), "s"(m[10]), "s"(m[11])
        : "vcc");
    return p;
}

// ---- the kernel ---------------------------------------------------------------
// Work split.  A row group is the 512/d rows one wave holds.  Block b (four
// waves) owns the kTileGroups * 4 consecutive groups starting at
// b * kTileGroups * 4; wave w takes groups base + 4u + w, u < kTileGroups, so
// that each load or store instruction of the block touches one contiguous
// span.  Blocks are not persistent: the dispatcher streams them through the
// chip in address order, which keeps HBM pages and channels evenly busy.
// When there is one parameter set, or rows_per_set is a multiple of the rows
// of a block, all rows of a block share a set and the block stages that set's
// parameters once through LDS (GENERIC_SETS = false).  Otherwise each lane
// finds the set of its row for every group and reads its parameters from
// global memory.  Parameters are staged before the tile's loads are issued:
// measured on MI355X, this order beats issuing the data loads first.
template <int VAR, int D, int BITS, bool F16, int MODE, bool GENERIC_SETS>
struct Stage1 {
    static constexpr int LPV = D / kCoordsPerLane;      // lanes per row
    static constexpr int VPW = 64 / LPV;                // rows per wave
    static constexpr int H = 1 << (BITS - 1);           // positive levels
    static constexpr int PL = VAR == VAR_FULL ? 32 : 8; // parameter floats per lane
    static constexpr int64_t ROWB = (int64_t)D * (F16 ? 2 : 4);  // bytes per row
    static constexpr int64_t RECB = (int64_t)D * BITS / 8;       // bytes per index record
    static constexpr int LANEB = F16 ? 16 : 32;         // row bytes per lane
    static constexpr bool kUseLut = BITS == 4;           // magnitude lookup table
    static constexpr bool kEncode = MODE == MODE_QUANTIZE || MODE == MODE_APPEND;  // records out

    struct In {
        Raw<F16> raw;
        uint32_t bits;
        float rho;
    };

    // Row addressing.  The row of a lane is grow + lr: grow, the first row of
    // the group, is wave-uniform, and lr < VPW is the lane's row slot, so
    // addresses are a scalar base plus a loop-invariant lane offset.  In the
    // last (tail) tile, lanes past the end take the last row: they recompute
    // it and store the same bits to the same place, which keeps the loop free
    // of divergent branches.
    template <bool TAIL>
    __device__ static __forceinline__ int lane_row(const KArgs &a, int64_t grow, int slot)
    {
        if constexpr (TAIL)
            return (int)(min(grow + slot, a.n - 1) - grow);
        return slot;
    }

    __device__ static __forceinline__ void fetch(const KArgs &a, int64_t grow, int lr, int sub, In &in)
    {
        if constexpr (MODE == MODE_DEQUANTIZE) {
            in.bits = load_bits<BITS>(a.rec_in + grow * RECB + (uint32_t)(lr * RECB), sub);
            in.rho = (a.norms_in + grow)[lr];
        } else if constexpr (MODE == MODE_APPEND) {
            // token grow + lr, head blockIdx.x of rows [n_tokens][n_heads][d]
            const int64_t tstride = (int64_t)a.n_heads * ROWB;
            load_row_chunk<F16>(static_cast<const char *>(a.x) + grow * tstride + (int64_t)blockIdx.x * ROWB +
                                    (uint32_t)(lr * (uint32_t)tstride + sub * LANEB),
                                in.raw);
        } else {
            load_row_chunk<F16>(static_cast<const char *>(a.x) + grow * ROWB + (uint32_t)(lr * ROWB + sub * LANEB),
                                in.raw);
        }
    }

    __device__ static __forceinline__ void compute(const KArgs &a, const float *P, const float *lev,
                                                   const float *thr, const float *lds_levels,
                                                   const LutEntry *lut, const In &in, int64_t grow,
                                                   int lr, int sub)
    {
        float yq[8];
        if constexpr (MODE == MODE_DEQUANTIZE) {
#pragma unroll
            for (int j = 0; j < 8; j++) {
                const uint32_t idx = (in.bits >> (BITS * j)) & (2 * H - 1);
                yq[j] = lds_levels[idx] * in.rho;
            }
        } else {
            float x[8];
            unpack<F16>(in.raw, x);
            const float rho = __builtin_amdgcn_sqrtf(row_sum<LPV>(sum_squares<F16>(in.raw, x)));
            const float rho_e = fmaxf(rho, kEps);
            float y[8], m[8];
            rotate_forward<VAR>(P, x, y);
#pragma unroll
            for (int j = 0; j < 8; j++)
                m[j] = fabsf(y[j]);
            if constexpr (kUseLut) {
                // 4 bits: cell of the normalised magnitude, one compare against
                // the cell's threshold (quantize and round trip use the same t)
                const float s = a.lut_inv_h * __builtin_amdgcn_rcpf(rho_e);
                const float last = (float)(a.lut_cells - 1);
                uint32_t p = 0;
#pragma unroll
                for (int j = 0; j < 8; j++) {
                    const float t = m[j] * s;
                    const LutEntry e = lut[(uint32_t)fminf(t, last)];
                    const bool above = t > e.t;
                    if constexpr (MODE == MODE_ROUNDTRIP) {
                        const float L = above ? e.hi : e.lo;
                        yq[j] = (y[j] > 0.f ? L : -L) * rho;
                    } else {
                        const uint32_t q = e.m + (above ? 1u : 0u);
                        p |= (q ^ (y[j] > 0.f ? (uint32_t)H : (uint32_t)(H - 1))) << (BITS * j);
                    }
                }
                if constexpr (kEncode)
                    emit(a, grow, lr, sub, p, rho);
            } else {
            float ths[H > 1 ? H - 1 : 1];
#pragma unroll
            for (int k = 0; k < H - 1; k++)
                ths[k] = thr[k] * rho_e;
            if constexpr (MODE == MODE_ROUNDTRIP) {
                float lvs[H];
#pragma unroll
                for (int k = 0; k < H; k++)
                    lvs[k] = lev[k] * rho;
                float L[8];
#pragma unroll
                for (int j = 0; j < 8; j++)
                    L[j] = lvs[0];
                // thresholds outer, coordinates inner: independent compares
                // fill the distance between each compare and its select
#pragma unroll
                for (int k = 0; k < H - 1; k++)
#pragma unroll
                    for (int j = 0; j < 8; j++)
                        L[j] = m[j] > ths[k] ? lvs[k + 1] : L[j];
#pragma unroll
                for (int j = 0; j < 8; j++)
                    yq[j] = y[j] > 0.f ? L[j] : -L[j];
            } else {
                // m = number of positive thresholds below |y|; the index is
                // H + m for y > 0 and H - 1 - m otherwise, i.e. m ^ H or
                // m ^ (H - 1)
                // For y > 0 the index is H + m, otherwise (H - 1) - m: its top
                // bit is the sign decision and every lower bit is the matching
                // bit of the magnitude index m, inverted when y <= 0.  The
                // lane masks of those bits are pushed into the record word
                // from its most significant end: coordinate 7's top bit first.
                // m: 3 bits, binary search (compare with the middle positive
                // threshold, then with the one it selects); 2 bits, one compare.
                uint64_t mk[8 * BITS];  // BITS masks per coordinate
#pragma unroll
                for (int j = 7; j >= 0; j--) {
                    uint64_t *o = mk + (7 - j) * BITS;
                    const uint64_t pos = __builtin_amdgcn_ballot_w64(y[j] > 0.f);
                    o[0] = pos;
                    if constexpr (H == 4) {
                        const bool hi = m[j] > ths[1];
                        const bool lo = m[j] > (hi ? ths[2] : ths[0]);
                        o[1] = ~(__builtin_amdgcn_ballot_w64(hi) ^ pos);
                        o[2] = ~(__builtin_amdgcn_ballot_w64(lo) ^ pos);
                    } else {
                        o[1] = ~(__builtin_amdgcn_ballot_w64(m[j] > ths[0]) ^ pos);
                    }
                }
                static_assert(BITS == 2 || BITS == 3, "2 or 3 bits on this branch");
                uint32_t p = 0;
                if constexpr (H == 4) {
                    p = push_bits12(p, mk);
                    p = push_bits12(p, mk + 12);
                } else {
                    p = push_bits8(p, mk);
                    p = push_bits8(p, mk + 8);
                }
                emit(a, grow, lr, sub, p, rho);
            }
            }
        }
        if constexpr (!kEncode) {
            float o[8];
            rotate_inverse<VAR>(P, yq, o);
            store_row_chunk<F16>(static_cast<char *>(a.y) + grow * ROWB + (uint32_t)(lr * ROWB + sub * LANEB), o);
        }
    }

    // Write one row's index record and norm: to row grow + lr (quantize), or
    // to the cache slot of token grow + lr for head blockIdx.x (append): slot
    // s is position s mod block_size of cache block s / block_size, and a
    // cache block holds [n_heads][block_size] records.  A skipped slot writes
    // nothing; the quad exchange inside store_bits runs on every lane either
    // way.
    __device__ static __forceinline__ void emit(const KArgs &a, int64_t grow, int lr, int sub,
                                                uint32_t p, float rho)
    {
        if constexpr (MODE == MODE_QUANTIZE) {
            store_bits<BITS>(a.rec_out + grow * RECB + (uint32_t)(lr * RECB), sub, p, true);
            if (sub == 0)
                (a.norms_out + grow)[lr] = rho;
        } else {
            const uint32_t h = blockIdx.x;
            const int64_t s = (a.slots + grow)[lr];
            const bool ok = s >= 0 && s < a.n_slots;
            const uint32_t su = ok ? (uint32_t)s : 0u;
            const uint32_t blk = fast_div(su, a.div_block);
            const int64_t crow = ((int64_t)blk * a.n_heads + h) * a.block_size + (su - blk * a.block_size);
            store_bits<BITS>(a.rec_out + crow * RECB, sub, p, ok);
            if (ok && sub == 0)
                a.norms_out[crow] = rho;
        }
    }

    // parameter set of `row` (GENERIC_SETS only)
    __device__ static __forceinline__ int set_of(const KArgs &a, int64_t row)
    {
        return (int)((row / a.rows_per_set) % a.n_sets);
    }

    __device__ static void run(const KArgs &a, float *lds_levels, float *lds_params, LutEntry *lds_lut)
    {
        const int lane = threadIdx.x & 63;
        const int sub = lane % LPV;
        const int slot = lane / LPV;
        const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
        const int64_t groups = (a.n + VPW - 1) / VPW;
        // append: blocks (head, token range) are dispatched head-fastest, so
        // the blocks in flight read all heads of the same tokens, one span
        const int64_t base = (int64_t)(MODE == MODE_APPEND ? blockIdx.y : blockIdx.x) * (kBlockThreads / 64) *
                             kTileGroups;

        // 1. block-wide tables: the codebook (dequantize) and the rotation
        //    parameters of the block's set, staged through LDS
        if constexpr (MODE == MODE_DEQUANTIZE) {
            if (threadIdx.x < 2 * H)
                lds_levels[threadIdx.x] = a.lev_all[threadIdx.x];
        }
        if constexpr (kUseLut && MODE != MODE_DEQUANTIZE) {
            const u32x4 *s4 = reinterpret_cast<const u32x4 *>(a.lut);
            u32x4 *d4 = reinterpret_cast<u32x4 *>(lds_lut);
            for (int i = threadIdx.x; i < a.lut_cells; i += kBlockThreads)
                d4[i] = s4[i];
        }
        float P[PL];
        if constexpr (!GENERIC_SETS) {
            // append: the block's head (every set is a head, or there is one)
            const int64_t set = a.n_sets <= 1           ? 0
                                : MODE == MODE_APPEND ? (int64_t)blockIdx.x
                                                      : (base * VPW / a.rows_per_set) % a.n_sets;
            const u32x4 *s4 = reinterpret_cast<const u32x4 *>(a.params + set * (LPV * PL));
            u32x4 *d4 = reinterpret_cast<u32x4 *>(lds_params);
            for (int i = threadIdx.x; i < LPV * PL / 4; i += kBlockThreads)
                d4[i] = s4[i];
        }
        if constexpr (MODE == MODE_DEQUANTIZE || !GENERIC_SETS || kUseLut)
            __syncthreads();
        if constexpr (!GENERIC_SETS)
            load_params<PL>(lds_params + sub * PL, P);
        if (base + w >= groups)
            return;

        float lev[H], thr[H > 1 ? H - 1 : 1];
#pragma unroll
        for (int k = 0; k < H; k++)
            lev[k] = a.lev_pos[k];
#pragma unroll
        for (int k = 0; k < H - 1; k++)
            thr[k] = a.thr_pos[k];

        const int64_t row0 = base * VPW;  // first row of the block
        if ((base + (kBlockThreads / 64) * kTileGroups) * VPW <= a.n)
            tile<false>(a, P, lev, thr, lds_levels, lds_lut, row0, groups, base, w, sub, slot);
        else
            tile<true>(a, P, lev, thr, lds_levels, lds_lut, row0, groups, base, w, sub, slot);
    }

    // The wave's kTileGroups groups: every load first (a group past the end
    // re-reads the last group and is neither computed nor stored), kept in
    // flight together by the scheduling barrier; then compute and store group
    // by group.
    template <bool TAIL>
    __device__ static __forceinline__ void tile(const KArgs &a, float *P, const float *lev,
                                                const float *thr, const float *lds_levels,
                                                const LutEntry *lut, int64_t row0, int64_t groups,
                                                int64_t base, int w, int sub, int slot)
    {
        In buf[kTileGroups];
#pragma unroll
        for (int u = 0; u < kTileGroups; u++) {
            const int gl = TAIL ? (int)(min(base + 4 * u + w, groups - 1) - base) : 4 * u + w;
            const int64_t grow = row0 + (int64_t)gl * VPW;
            fetch(a, grow, lane_row<TAIL>(a, grow, slot), sub, buf[u]);
        }
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int u = 0; u < kTileGroups; u++) {
            const int gl = 4 * u + w;
            if (TAIL && base + gl >= groups)
                break;
            const int64_t grow = row0 + (int64_t)gl * VPW;
            const int lr = lane_row<TAIL>(a, grow, slot);
            if constexpr (GENERIC_SETS)
                load_params<PL>(a.params + ((int64_t)set_of(a, grow + lr) * LPV + sub) * PL, P);
            compute(a, P, lev, thr, lds_levels, lut, buf[u], grow, lr, sub);
        }
    }
};

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
