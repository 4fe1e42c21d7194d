// The stage-1 kernel template shared by isoq_kernels.hip (round trip,
// quantize, dequantize, append) and isoq_qjl.h (quantize with the stage-2
// residual sketch, into rows or into cache slots): packed index records, the
// Stage1 work split and compute.
#pragma once

#include "isoq_device.h"
#include "isoq_internal.h"

namespace isoq {
namespace {

// ---- packed index records --------------------------------------------------
// Two lane layouts write the same record (coordinate j at bits [j b, j b + b)):
// a lane owning coordinates 8 sub .. 8 sub + 7 (store_bits / load_bits), or,
// for fp32 rows, a lane owning slots sub and sub + LPV, whose 4b-bit pieces lie
// in the first and the second half of the record (the _split variants).  In
// both, the lane's index word p holds coordinate j of its 8 at bits
// [j b, j b + b).
// Lane `sub` of a row owns coordinates 8 sub .. 8 sub + 7, i.e. bits
// [8 sub * BITS, 8 (sub + 1) * BITS) of the row's record: a 16-bit half-word
// (2 bits), a 32-bit word (4 bits), or 24 bits at byte 3 sub (3 bits), which
// the four lanes of a DPP quad merge into three aligned words.
template <int BITS, class Dst>
__device__ __forceinline__ void store_bits_to(const Dst &rec, int sub, uint32_t p, bool ok)
{
    if constexpr (BITS == 2) {
        if (ok)
            rec.template put<uint16_t>(2 * sub, (uint16_t)p);
    } else if constexpr (BITS == 4) {
        if (ok)
            rec.template put<uint32_t>(4 * sub, p);
    } else {
        // lane k of a quad holds bits [24 k, 24 k + 24) of 96; lanes 0..2
        // write word k = p_k >> 8 k | p_(k+1) << (24 - 8 k)
        const uint32_t nb = dpp_u<DPP_QUAD_1233>(p);  // bits of the next lane in the quad
        const int k = sub & 3;
        if (ok && k < 3)
            rec.template put<uint32_t>(4 * (3 * (sub >> 2) + k), (p >> (8 * k)) | (nb << (24 - 8 * k)));
    }
}

template <int BITS>
__device__ __forceinline__ void store_bits(uint8_t *rec, int sub, uint32_t p, bool ok)
{
    store_bits_to<BITS>(RecPtr{rec}, sub, p, ok);
}

template <int BITS, int LPV>
__device__ __forceinline__ void store_bits_split(uint8_t *rec, int sub, uint32_t p, bool ok)
{
    constexpr int PB = 4 * BITS;        // bits per piece
    constexpr int HALF = LPV * PB / 8;  // bytes per half record
    const uint32_t pa = p & ((1u << PB) - 1u), pb = p >> PB;
    if constexpr (BITS == 2) {
        if (ok) {
            rec[sub] = (uint8_t)pa;
            rec[HALF + sub] = (uint8_t)pb;
        }
    } else if constexpr (BITS == 4) {
        if (ok) {
            reinterpret_cast<uint16_t *>(rec)[sub] = (uint16_t)pa;
            reinterpret_cast<uint16_t *>(rec + HALF)[sub] = (uint16_t)pb;
        }
    } else {
        // 12-bit pieces: lanes 2q and 2q + 1 form the 24-bit unit q of a half,
        // and the even lanes of an octet merge its four units into three
        // words as store_bits merges a quad's (unit q + 1 is two lanes on;
        // the last unit of a row, which would read past it, writes nothing)
#pragma unroll
        for (int h = 0; h < 2; h++) {
            const uint32_t v = h ? pb : pa;
            const uint32_t u = v | ((uint32_t)__shfl_down((int)v, 1, 64) << 12);
            const uint32_t nu = (uint32_t)__shfl_down((int)u, 2, 64);
            const int q = sub >> 1, k = q & 3;
            if (ok && (sub & 1) == 0 && k < 3)
                reinterpret_cast<uint32_t *>(rec + h * HALF)[3 * (q >> 2) + k] = (u >> (8 * k)) | (nu << (24 - 8 * k));
        }
    }
}

template <int BITS, int LPV>
__device__ __forceinline__ uint32_t load_bits_split(const uint8_t *rec, int sub)
{
    constexpr int PB = 4 * BITS;
    constexpr int HALF = LPV * PB / 8;
    uint32_t pa, pb;
    if constexpr (BITS == 2) {
        pa = rec[sub];
        pb = rec[HALF + sub];
    } else if constexpr (BITS == 4) {
        pa = reinterpret_cast<const uint16_t *>(rec)[sub];
        pb = reinterpret_cast<const uint16_t *>(rec + HALF)[sub];
    } else {
        // the piece at bit 12 sub of a half: word k, and word k + 1 when the
        // piece straddles it (then that word still belongs to the half)
        const int o = 12 * sub, k = o >> 5, sh = o & 31;
        const int k1 = sh > 20 ? k + 1 : k;
        const uint32_t *wa = reinterpret_cast<const uint32_t *>(rec);
        const uint32_t *wb = reinterpret_cast<const uint32_t *>(rec + HALF);
        pa = (uint32_t)((((uint64_t)wa[k1] << 32) | wa[k]) >> sh) & 0xFFFu;
        pb = (uint32_t)((((uint64_t)wb[k1] << 32) | wb[k]) >> sh) & 0xFFFu;
    }
    return pa | (pb << PB);
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

__device__ __forceinline__ uint32_t push_bits4(uint32_t p, const uint64_t m[4])
{
    asm("s_nop 4\n\t"
        "v_addc_co_u32_e64 %0, vcc, %0, %0, %1\n\t"
        "v_addc_co_u32_e64 %0, vcc, %0, %0, %2\n\t"
        "v_addc_co_u32_e64 %0, vcc, %0, %0, %3\n\t"
        "v_addc_co_u32_e64 %0, vcc, %0, %0, %4"
        : "+v"(p)
        : "s"(m[0]), "s"(m[1]), "s"(m[2]), "s"(m[3])
        : "vcc");
    return p;
}

__device__ __forceinline__ uint32_t push_bits6(uint32_t p, const uint64_t m[6])
{
    asm("s_nop 4\n\t"
        "v_addc_co_u32_e64 %0, vcc, %0, %0, %1\n\t"
        "v_addc_co_u32_e64 %0, vcc, %0, %0, %2\n\t"
        "v_addc_co_u32_e64 %0, vcc, %0, %0, %3\n\t"
        "v_addc_co_u32_e64 %0, vcc, %0, %0, %4\n\t"
        "v_addc_co_u32_e64 %0, vcc, %0, %0, %5\n\t"
        "v_addc_co_u32_e64 %0, vcc, %0, %0, %6"
        : "+v"(p)
        : "s"(m[0]), "s"(m[1]), "s"(m[2]), "s"(m[3]), "s"(m[4]), "s"(m[5])
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

// ---- the quantizer of a lane's 8 rotated coordinates --------------------------
// Shared by the tuned kernels and the packed-row kernels (isoq_packed.h).  y:
// rotated coordinates (in units of rho when rho is folded into the thresholds),
// m = |y|.

// 4 bits: the cell of each normalised magnitude m s in the lookup table, then
// one compare against the cell's threshold (quantize and round trip use the
// same t).  Returns the index word (ENCODE); yq gets the signed selected levels
// times lscale (LEVELS).
template <int BITS, bool LEVELS, bool ENCODE>
__device__ __forceinline__ uint32_t lut_quantize(const float y[8], const float m[8], float s, float last,
                                                 const LutEntry *lut, float lscale, float yq[8])
{
    constexpr int H = 1 << (BITS - 1);
    uint32_t p = 0;
#pragma unroll
    for (int j = 0; j < 8; j++) {
        const float t = m[j] * s;
        const LutEntry e = lut[(uint32_t)fminf(t, last)];
        const bool above = t > e.t;
        if constexpr (LEVELS) {
            const float L = above ? e.hi : e.lo;
            yq[j] = (y[j] > 0.f ? L : -L) * lscale;
        }
        if constexpr (ENCODE) {
            const uint32_t q = e.m + (above ? 1u : 0u);
            p |= (q ^ (y[j] > 0.f ? (uint32_t)H : (uint32_t)(H - 1))) << (BITS * j);
        }
    }
    return p;
}

// 2 and 3 bits: the signed selected levels from the scaled positive
// thresholds ths and levels lvs, thresholds outer and coordinates inner, so
// that independent compares fill the distance between each compare and its
// select.
template <int H>
__device__ __forceinline__ void chain_levels(const float y[8], const float m[8], const float *ths, const float *lvs,
                                             float yq[8])
{
    float L[8];
#pragma unroll
    for (int j = 0; j < 8; j++)
        L[j] = lvs[0];
#pragma unroll
    for (int k = 0; k < H - 1; k++)
#pragma unroll
        for (int j = 0; j < 8; j++)
            L[j] = m[j] > ths[k] ? lvs[k + 1] : L[j];
#pragma unroll
    for (int j = 0; j < 8; j++)
        yq[j] = y[j] > 0.f ? L[j] : -L[j];
}

// 2 and 3 bits: the index word of the 8 coordinates from lane masks.  With
// QJL, yq also gets the signed normalised levels (from lev) that the
// encoder's compares select.
template <int BITS, bool QJL>
__device__ __forceinline__ uint32_t ballot_encode(const float y[8], const float m[8], const float *ths,
                                                  const float *lev, float yq[8])
{
    constexpr int H = 1 << (BITS - 1);
    // For y > 0 the index is H + m, otherwise (H - 1) - m: its top
    // bit is the sign decision and every lower bit is the matching
    // bit of the magnitude index m, inverted when y <= 0.  The
    // lane masks of those bits are pushed into the record word
    // from its most significant end: coordinate 7's top bit first.
    // m: 3 bits, binary search (compare with the middle positive
    // threshold, then with the one it selects); 2 bits, one compare.
    // 4 coordinates per asm block (2 with the stage-2 sketch,
    // whose extra state would otherwise push the live masks past
    // the scalar register file)
    static_assert(BITS == 2 || BITS == 3, "2 or 3 bits on this branch");
    constexpr int CPB = QJL ? 2 : 4;   // coordinates per push block
    uint32_t p = 0;
#pragma unroll
    for (int j0 = 7; j0 >= 0; j0 -= CPB) {
        uint64_t mk[CPB * BITS];  // BITS masks per coordinate
#pragma unroll
        for (int c = 0; c < CPB; c++) {
            const int j = j0 - c;
            uint64_t *o = mk + c * BITS;
            const uint64_t pos = __builtin_amdgcn_ballot_w64(y[j] > 0.f);
            o[0] = pos;
            if constexpr (H == 4) {
                const bool hi = m[j] > ths[1];
                const bool lo = m[j] > (hi ? ths[2] : ths[0]);
                o[1] = ~(__builtin_amdgcn_ballot_w64(hi) ^ pos);
                o[2] = ~(__builtin_amdgcn_ballot_w64(lo) ^ pos);
                if constexpr (QJL) {
                    // normalised level of magnitude index 2 hi + lo
                    const float La = lo ? lev[1] : lev[0];
                    const float Lb = lo ? lev[3] : lev[2];
                    const float L = hi ? Lb : La;
                    yq[j] = y[j] > 0.f ? L : -L;
                }
            } else {
                const bool above = m[j] > ths[0];
                o[1] = ~(__builtin_amdgcn_ballot_w64(above) ^ pos);
                if constexpr (QJL) {
                    const float L = above ? lev[1] : lev[0];
                    yq[j] = y[j] > 0.f ? L : -L;
                }
            }
        }
        if constexpr (CPB * BITS == 12)
            p = push_bits12(p, mk);
        else if constexpr (CPB * BITS == 8)
            p = push_bits8(p, mk);
        else if constexpr (CPB * BITS == 6)
            p = push_bits6(p, mk);
        else
            p = push_bits4(p, mk);
    }
    return p;
}

// ---- stage-2 projection of a wave's error tile -------------------------------------
// Chunk-position swizzle of an unpadded error tile (rows of D halfs, 16-byte
// chunks): chunk c of tile row r is stored at c ^ err_swizzle(r).  With the
// matrix-core encoder's writes (lanes 4b + i: chunk b of row 4q + i) and the
// projection's reads (lane l: row l mod 16, chunk 4 ks + l / 16), every 8 lanes
// of a 16-byte access then touch 8 different 16-byte bank groups of the 32
// banks; the padded layout (row stride D + 8 halfs) conflicted on the writes.
__device__ __forceinline__ int err_swizzle(int r) { return (2 * (r & 3)) ^ ((r >> 2) & 3); }

// P = E S'^T with E the tile's error rows (fp16, LDS, row stride ES halfs) and
// S' = S T^{-1} (fp16, LDS, fragment order), computed transposed, P^T = S' E^T,
// on v_mfma_f32_16x16x32_f16: for column tile nt lane l supplies row l % 16 of
// the tile's 16 rows of S' and column l % 16 of E^T (error row l % 16), both
// for k = 8 (l / 16) .. +7 of each 32-wide k step, and receives rows
// 4 (l / 16) .. +3 of column l % 16 of the 16 x 16 result.  The host orders
// S' so that row r of tile nt is sketch coordinate (m/4) (r / 4) + 4 nt + r % 4:
// lane l then holds, over the NT tiles, the m/4 consecutive coordinates
// (m/4) (l / 16) .. + m/4 - 1 of error row l % 16, so it turns its results into
// that part of the row's sign record by itself (bit b = coordinate
// (m/4) (l / 16) + b; a compare and a carry-in add per bit), with no exchange
// between lanes.  The sign bits of rho * P (rho > 0 unless the row is zero,
// whose e is zero) are the sketch.  A tile of more than 16 rows takes one such
// product per block of 16 rows.  dst_of(ar) is the sign row of tile row ar, or
// nullptr where nothing is written.  SWZ: the tile's rows are unpadded
// (ES = D) and chunk c of row r sits at chunk position c ^ err_swizzle(r).
template <int D, int QM, int TR, int ES, bool SWZ = false, typename DstOf>
__device__ __forceinline__ void qjl_project(const _Float16 *frag, const _Float16 *eq, DstOf dst_of)
{
    typedef _Float16 half8 __attribute__((ext_vector_type(8)));
    typedef float f32x4 __attribute__((ext_vector_type(4)));
    constexpr int KS = D / 32, NT = QM / 16;
    static_assert(NT == 4 || NT == 8, "m = 64 or 128: 16 or 32 sign bits per lane");
    constexpr int RB = (TR + 15) / 16;  // blocks of 16 tile rows (2 at d = 64)
    const int l = threadIdx.x & 63;
    const int r16 = l & 15, kq = l >> 4;
    // one block of 16 rows at a time (its fragments and accumulators only)
#pragma unroll 1
    for (int rb = 0; rb < RB; rb++) {
        // an offset the compiler cannot see through (it is zero), so that the
        // projection's fragments are read where they are used rather than
        // hoisted out of this loop and held in registers across it
        int fo = 0;
        asm volatile("" : "+s"(fo));
        half8 E[KS];
        const int ar = 16 * rb + r16;   // the tile row of this lane's column
#pragma unroll
        for (int ks = 0; ks < KS; ks++) {
            if (ar < TR) {
                const int pos = SWZ ? (4 * ks + kq) ^ err_swizzle(ar) : 4 * ks + kq;
                E[ks] = *reinterpret_cast<const half8 *>(eq + ar * ES + 8 * pos);
            } else {
#pragma unroll
                for (int i = 0; i < 8; i++)
                    E[ks][i] = (_Float16)0.f;
            }
        }
        // k-step outer, column tile inner: the NT accumulations are
        // independent, so consecutive MFMAs do not wait on each other
        f32x4 acc[NT];
#pragma unroll
        for (int nt = 0; nt < NT; nt++)
            acc[nt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < KS; ks++) {
#pragma unroll
            for (int nt = 0; nt < NT; nt++) {
                const half8 s = *reinterpret_cast<const half8 *>(frag + fo + ((nt * KS + ks) * 64 + l) * 8);
                acc[nt] = __builtin_amdgcn_mfma_f32_16x16x32_f16(s, E[ks], acc[nt], 0, 0, 0);
            }
            // at most one k-step's fragments in flight
            if constexpr (KS > 4)
                __builtin_amdgcn_sched_barrier(0);
        }
        // bit 4 nt + i is result register i of tile nt: pushed from the top
        // (tile NT - 1, register 3) down
        uint32_t p = 0;
#pragma unroll
        for (int nt = NT - 1; nt >= 0; nt--) {
            const uint64_t mk[4] = {__builtin_amdgcn_ballot_w64(acc[nt][3] > 0.f),
                                    __builtin_amdgcn_ballot_w64(acc[nt][2] > 0.f),
                                    __builtin_amdgcn_ballot_w64(acc[nt][1] > 0.f),
                                    __builtin_amdgcn_ballot_w64(acc[nt][0] > 0.f)};
            p = push_bits4(p, mk);
        }
        if (uint32_t *dst = dst_of(ar)) {
            if constexpr (NT == 8)
                dst[kq] = p;
            else
                reinterpret_cast<uint16_t *>(dst)[kq] = (uint16_t)p;
        }
    }
}

// ---- the kernel ---------------------------------------------------------------
// Work split.  A row group is the 512/d rows one wave holds.  Block b (WAVES
// waves, four except for some sketch kernels) owns the kTileGroups * WAVES
// consecutive groups starting at b * kTileGroups * WAVES; wave w takes groups
// base + WAVES u + w, u < kTileGroups, so
// that each load or store instruction of the block touches one contiguous
// span.  Blocks are not persistent: the dispatcher streams them through the
// chip in address order, which keeps HBM pages and channels evenly busy.
// When there is one parameter set, or rows_per_set is a multiple of the rows
// of a block, all rows of a block share a set and the block stages that set's
// parameters once through LDS (GENERIC_SETS = false).  Otherwise each lane
// finds the set of its row for every group and reads its parameters from
// global memory.  Parameters are staged before the tile's loads are issued:
// measured on MI355X, this order beats issuing the data loads first.
// QM: sketch size m of the stage-2 residual sketch (MODE_QJL and
// MODE_APPEND_QJL only).  WAVES: waves per block (BT = 64 WAVES threads).
template <int VAR, int D, int BITS, bool F16, int MODE, bool GENERIC_SETS, int QM = 0, int WAVES = 4>
struct Stage1 {
    static constexpr int BT = WAVES * 64;               // threads per block
    static constexpr int LPV = D / kCoordsPerLane;      // lanes per row
    static constexpr int VPW = 64 / LPV;                // rows per wave
    static constexpr int H = 1 << (BITS - 1);           // positive levels
    static constexpr int PL = kLanePL<VAR>;              // parameter floats per lane
    static constexpr int64_t ROWB = (int64_t)D * (F16 ? 2 : 4);  // bytes per row
    static constexpr int64_t RECB = (int64_t)D * BITS / 8;       // bytes per index record
    static constexpr int LANEB = F16 ? 16 : 32;         // row bytes per lane
    // fp32 round trip, quantize and dequantize: lane `sub` owns slots sub and
    // sub + LPV (coordinates 4 sub .. +3 and D/2 + 4 sub .. +3), so each
    // 16-byte access instruction of a wave covers one contiguous span (its
    // index pieces go to the two halves of the record); elsewhere, and for
    // 8-D blocks (whose 8 coordinates must stay together), it owns slots
    // 2 sub and 2 sub + 1
    static constexpr bool kSplit = !F16 && VAR != VAR_BLOCK8 &&
                                   (MODE == MODE_ROUNDTRIP || MODE == MODE_QUANTIZE || MODE == MODE_DEQUANTIZE);
    static constexpr int kLaneOff = kSplit ? 16 : LANEB;       // bytes to lane sub's first piece
    static constexpr int kStep = kSplit ? (int)(ROWB / 2) : 16;  // bytes to its second piece
    static constexpr bool kUseLut = BITS == 4;           // magnitude lookup table
    static constexpr bool kQjl = MODE == MODE_QJL || MODE == MODE_APPEND_QJL;
    static constexpr bool kAppend = MODE == MODE_APPEND || MODE == MODE_APPEND_QJL;  // rows go to cache slots
    static constexpr bool kEncode = MODE == MODE_QUANTIZE || MODE == MODE_APPEND || kQjl;  // records out
    static constexpr bool kLevels = MODE == MODE_ROUNDTRIP || kQjl;  // selected levels needed
    // stage-2 sketch: a wave's tile of rows, its fp16 error rows in LDS
    static constexpr int kTileRows = kTileGroups * VPW;   // 32 (d = 64), 16 (d = 128) or 8 (d = 256)
    static constexpr int kEStride = D + 8;                // halfs per LDS error row (padded)

    // Staged parameters in LDS.  With the 4-bit lookup table (whose reads
    // compete for LDS) chunk k (16 bytes) of lane sub goes to word k LPV + sub,
    // the lane's chunks in the order it uses them, so the lanes of a row read
    // consecutive words: a plain copy of the slot-major set puts every lane
    // of the row on the same four banks (Full's 128 bytes per lane: a 16-way
    // conflict), which cost the 4-bit kernels about 5%.  Without the table the
    // plain copy measured about 1% faster, so those kernels keep it.
    static constexpr bool kChunkMajor = kUseLut;

    __device__ static __forceinline__ void stage_params(const float *set, float *lds)
    {
        if constexpr (!kChunkMajor) {
            const u32x4 *s4 = reinterpret_cast<const u32x4 *>(set);
            u32x4 *d4 = reinterpret_cast<u32x4 *>(lds);
            for (int i = threadIdx.x; i < LPV * PL / 4; i += BT)
                d4[i] = s4[i];
            return;
        }
        constexpr int CPS = PL / 8;  // 16-byte chunks per slot
        const u32x4 *s4 = reinterpret_cast<const u32x4 *>(set);
        u32x4 *d4 = reinterpret_cast<u32x4 *>(lds);
        // LDS word j = k LPV + ln is written in order (no bank conflicts);
        // its chunk is gathered from the set (a few KB, cached)
        for (int j = threadIdx.x; j < LPV * PL / 4; j += BT) {
            const int k = j / LPV, ln = j - k * LPV;
            const int half = k / CPS, c = k - half * CPS;
            const int slot = kSplit ? half * LPV + ln : 2 * ln + half;
            d4[j] = s4[slot * CPS + c];
        }
    }

    __device__ static __forceinline__ void lds_lane_params(const float *lds, int sub, float P[PL])
    {
        if constexpr (!kChunkMajor) {
            lane_params(lds, sub, P);
            return;
        }
        const u32x4 *q = reinterpret_cast<const u32x4 *>(lds);
#pragma unroll
        for (int k = 0; k < PL / 4; k++) {
            const u32x4 w = q[k * LPV + sub];
            const uint32_t e0 = w[0], e1 = w[1], e2 = w[2], e3 = w[3];
            P[4 * k] = __uint_as_float(e0);
            P[4 * k + 1] = __uint_as_float(e1);
            P[4 * k + 2] = __uint_as_float(e2);
            P[4 * k + 3] = __uint_as_float(e3);
        }
    }

    // The lane's two slots' rotation parameters from a set's [2 LPV][PL / 2]
    // in global memory.
    __device__ static __forceinline__ void lane_params(const float *set, int sub, float P[PL])
    {
        if constexpr (kSplit) {
            load_params<PL / 2>(set + sub * (PL / 2), P);
            load_params<PL / 2>(set + (sub + LPV) * (PL / 2), P + PL / 2);
        } else {
            load_params<PL>(set + sub * PL, P);
        }
    }

    struct In {
        Raw<F16> raw;
        uint32_t bits;
        float rho;
        int64_t slot;  // append modes: the token's cache slot
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
            const uint8_t *rec = a.rec_in + grow * RECB + (uint32_t)(lr * RECB);
            if constexpr (kSplit)
                in.bits = load_bits_split<BITS, LPV>(rec, sub);
            else
                in.bits = load_bits<BITS>(rec, sub);
            in.rho = (a.norms_in + grow)[lr];
        } else if constexpr (kAppend) {
            // token grow + lr, head blockIdx.x of rows [n_tokens][n_heads][d];
            // its slot is loaded with the row, so that the write-out does not
            // wait for it
            in.slot = (a.slots + grow)[lr];
            const int64_t tstride = (int64_t)a.n_heads * ROWB;
            load_row_chunk<F16>(static_cast<const char *>(a.x) + grow * tstride + (int64_t)blockIdx.x * ROWB +
                                    (uint32_t)(lr * (uint32_t)tstride + sub * LANEB),
                                in.raw);
        } else {
            load_row_chunk<F16>(static_cast<const char *>(a.x) + grow * ROWB + (uint32_t)(lr * ROWB + sub * kLaneOff),
                                in.raw, kStep);
        }
    }

    // erow, eq: row of this lane in the wave's tile and the wave's LDS error
    // tile (MODE_QJL only).
    __device__ static __forceinline__ void compute(const KArgs &a, const float *P, const float *lev,
                                                   const float *thr, const float *lds_levels,
                                                   const LutEntry *lut, const In &in, int64_t grow,
                                                   int lr, int sub, int erow = 0, _Float16 *eq = nullptr)
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
            const float ss = kSplit ? row_sum<LPV>(slot_squares(x)) + row_sum<LPV>(slot_squares(x + 4))
                                    : row_sum<LPV>(sum_squares<F16>(in.raw, x));
            const float rho = __builtin_amdgcn_sqrtf(ss);
            const float rho_e = fmaxf(rho, kEps);
            float y[8], m[8];
            // selected levels are scaled by rho for the round trip (it then
            // yields rho * rec directly) and left normalised for the sketch
            const float lscale = kQjl ? 1.f : rho;
            rotate_forward<VAR>(P, x, y);
#pragma unroll
            for (int j = 0; j < 8; j++)
                m[j] = fabsf(y[j]);
            if constexpr (kUseLut) {
                const float s = a.lut_inv_h * __builtin_amdgcn_rcpf(rho_e);
                const uint32_t p =
                    lut_quantize<BITS, kLevels, kEncode>(y, m, s, (float)(a.lut_cells - 1), lut, lscale, yq);
                if constexpr (kEncode)
                    emit(a, grow, lr, sub, p, rho, in.slot);
            } else {
            float ths[H > 1 ? H - 1 : 1];
#pragma unroll
            for (int k = 0; k < H - 1; k++)
                ths[k] = thr[k] * rho_e;
            // with the sketch the levels come from the encoder's own
            // compares (below); the round trip runs the compare chain
            if constexpr (kLevels && !kQjl) {
                float lvs[H];
#pragma unroll
                for (int k = 0; k < H; k++)
                    lvs[k] = lev[k] * lscale;
                chain_levels<H>(y, m, ths, lvs, yq);
            }
            if constexpr (kEncode) {
                const uint32_t p = ballot_encode<BITS, kQjl>(y, m, ths, lev, yq);
                emit(a, grow, lr, sub, p, rho, in.slot);
            }
            }
            if constexpr (kQjl) {
                // stage 2: e = y / rho' - c[idx], the quantization error of the
                // normalised rotated row (zero for a zero row); gamma =
                // rho ||e|| = ||x - x_hat|| (T is orthogonal); e goes to the
                // wave's LDS tile as fp16 for the projection
                const float inv = rho > 0.f ? __builtin_amdgcn_rcpf(rho_e) : 0.f;
                float e[8], s2 = 0.f;
#pragma unroll
                for (int j = 0; j < 8; j++) {
                    e[j] = rho > 0.f ? fmaf(y[j], inv, -yq[j]) : 0.f;
                    s2 = fmaf(e[j], e[j], s2);
                }
                const float gamma = rho * __builtin_amdgcn_sqrtf(row_sum<LPV>(s2));
                if constexpr (kAppend) {
                    bool ok;
                    const int64_t r = cache_row_of(a, in.slot, ok);
                    if (ok && sub == 0)
                        a.qjl_gamma[r] = gamma;
                } else if (sub == 0) {
                    (a.qjl_gamma + grow)[lr] = gamma;
                }
                u32x4 h;
#pragma unroll
                for (int k = 0; k < 4; k++) {
                    uint32_t v;
                    asm("v_cvt_pk_f16_f32 %0, %1, %2" : "=v"(v) : "v"(e[2 * k]), "v"(e[2 * k + 1]));
                    h[k] = v;
                }
                *reinterpret_cast<u32x4 *>(eq + erow * kEStride + 8 * sub) = h;
            }
        }
        if constexpr (!kEncode) {
            float o[8];
            rotate_inverse<VAR>(P, yq, o);
            store_row_chunk<F16>(static_cast<char *>(a.y) + grow * ROWB + (uint32_t)(lr * ROWB + sub * kLaneOff), o,
                                 kStep);
        }
    }

    // Cache row of slot s for head blockIdx.x (append modes): slot s is
    // position s mod block_size of cache block s / block_size, and a cache
    // block holds [n_heads][block_size] records.  ok is false for a skipped
    // slot (s < 0 or past the cache; the row returned is then 0 and must not
    // be written).
    __device__ static __forceinline__ int64_t cache_row_of(const KArgs &a, int64_t s, bool &ok)
    {
        ok = s >= 0 && s < a.n_slots;
        const uint32_t su = ok ? (uint32_t)s : 0u;
        const uint32_t blk = fast_div(su, a.div_block);
        return ((int64_t)blk * a.n_heads + blockIdx.x) * a.block_size + (su - blk * a.block_size);
    }

    // The same for token grow + lr, its slot read from the slot mapping.
    __device__ static __forceinline__ int64_t cache_row(const KArgs &a, int64_t grow, int lr, bool &ok)
    {
        return cache_row_of(a, (a.slots + grow)[lr], ok);
    }

    // Write one row's index record and norm: to row grow + lr (quantize), or
    // to the cache row of the token's slot (append; `slot` was loaded with
    // the row).  A skipped slot writes nothing; the quad exchange inside
    // store_bits runs on every lane either way.
    __device__ static __forceinline__ void emit(const KArgs &a, int64_t grow, int lr, int sub,
                                                uint32_t p, float rho, int64_t slot)
    {
        if constexpr (!kAppend) {
            uint8_t *rec = a.rec_out + grow * RECB + (uint32_t)(lr * RECB);
            if constexpr (kSplit)
                store_bits_split<BITS, LPV>(rec, sub, p, true);
            else
                store_bits<BITS>(rec, sub, p, true);
            if (sub == 0)
                (a.norms_out + grow)[lr] = rho;
        } else {
            bool ok;
            int pos;
            const int64_t crow = cache_slot(a, slot, blockIdx.x, ok, pos);
            store_bits_to<BITS>(cache_rec<RECB>(a, crow, pos), sub, p, ok);
            if (ok && sub == 0)
                a.norms_out[crow] = rho;
        }
    }

    // parameter set of `row` (GENERIC_SETS only)
    __device__ static __forceinline__ int set_of(const KArgs &a, int64_t row)
    {
        return (int)((row / a.rows_per_set) % a.n_sets);
    }

    __device__ static void run(const KArgs &a, float *lds_levels, float *lds_params, LutEntry *lds_lut,
                               _Float16 *lds_frag = nullptr, _Float16 *lds_e = nullptr)
    {
        const int lane = threadIdx.x & 63;
        const int sub = lane % LPV;
        const int slot = lane / LPV;
        const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
        const int64_t groups = (a.n + VPW - 1) / VPW;
        // append: blocks (head, token range) are dispatched head-fastest, so
        // the blocks in flight read all heads of the same tokens, one span
        const int64_t base = (int64_t)(kAppend ? blockIdx.y : blockIdx.x) * WAVES * kTileGroups;

        // 1. block-wide tables: the codebook (dequantize) and the rotation
        //    parameters of the block's set, staged through LDS
        if constexpr (MODE == MODE_DEQUANTIZE) {
            if (threadIdx.x < 2 * H)
                lds_levels[threadIdx.x] = a.lev_all[threadIdx.x];
        }
        if constexpr (kUseLut && MODE != MODE_DEQUANTIZE) {
            const u32x4 *s4 = reinterpret_cast<const u32x4 *>(a.lut);
            u32x4 *d4 = reinterpret_cast<u32x4 *>(lds_lut);
            for (int i = threadIdx.x; i < a.lut_cells; i += BT)
                d4[i] = s4[i];
        }
        float P[PL];
        if constexpr (!GENERIC_SETS) {
            // append: the block's head (every set is a head, or there is one)
            const int64_t set = a.n_sets <= 1           ? 0
                                : kAppend             ? (int64_t)blockIdx.x
                                                      : (base * VPW / a.rows_per_set) % a.n_sets;
            stage_params(a.params + set * (LPV * PL), lds_params);
            if constexpr (kQjl) {
                // the set's projection S' = S T^{-1} in MFMA B-fragment order
                const u32x4 *f4 = reinterpret_cast<const u32x4 *>(a.qjl_frag + set * (int64_t)(QM * D));
                u32x4 *g4 = reinterpret_cast<u32x4 *>(lds_frag);
                for (int i = threadIdx.x; i < QM * D / 8; i += BT)
                    g4[i] = f4[i];
            }
        }
        if constexpr (MODE == MODE_DEQUANTIZE || !GENERIC_SETS || kUseLut)
            __syncthreads();
        if constexpr (!GENERIC_SETS)
            lds_lane_params(lds_params, sub, P);

        float lev[H], thr[H > 1 ? H - 1 : 1];
#pragma unroll
        for (int k = 0; k < H; k++)
            lev[k] = a.lev_pos[k];
#pragma unroll
        for (int k = 0; k < H - 1; k++)
            thr[k] = a.thr_pos[k];

        // With the stage-2 sketch a block may walk several tiles (stride
        // gridDim.x, or gridDim.y over one head's tokens when appending) so
        // that the staged projection serves them all; the host launches one
        // block per tile when the tiles' sets differ.  No barrier follows, so
        // each wave leaves on its own.
        _Float16 *eq = kQjl ? lds_e + w * kTileRows * kEStride : nullptr;
        const int64_t tstride = kQjl ? (int64_t)(kAppend ? gridDim.y : gridDim.x) : (int64_t)1 << 62;
        for (int64_t tb = (int64_t)(kAppend ? blockIdx.y : blockIdx.x);; tb += tstride) {
            const int64_t tbase = tb * WAVES * kTileGroups;
            if (tbase + w >= groups)
                return;
            const int64_t row0 = tbase * VPW;  // first row of the tile
            if ((tbase + WAVES * kTileGroups) * VPW <= a.n)
                tile<false>(a, P, lev, thr, lds_levels, lds_lut, row0, groups, tbase, w, sub, slot, eq);
            else
                tile<true>(a, P, lev, thr, lds_levels, lds_lut, row0, groups, tbase, w, sub, slot, eq);
            if constexpr (kQjl)
                sketch(a, lds_frag, eq, row0, groups, tbase, w);
            else
                return;
        }
    }

    // Stage-2 sketch of the wave's tile (qjl_project): tile row ar is row
    // slot ar mod VPW of group ar / VPW of the wave.
    __device__ static __forceinline__ void sketch(const KArgs &a, const _Float16 *frag, const _Float16 *eq,
                                                  int64_t row0, int64_t groups, int64_t base, int w)
    {
        qjl_project<D, QM, kTileRows, kEStride>(frag, eq, [&](int ar) -> uint32_t * {
            const int u = ar / VPW, sl = ar - u * VPW;
            const int64_t gl = WAVES * u + w;
            bool ok = ar < kTileRows && base + gl < groups;
            int64_t row = min(row0 + gl * VPW + sl, a.n - 1);
            if constexpr (kAppend) {
                // the token's cache row (a skipped slot writes nothing)
                bool in_cache;
                row = cache_row(a, row, 0, in_cache);
                ok = ok && in_cache;
            }
            return ok ? reinterpret_cast<uint32_t *>(a.qjl_signs + row * (QM / 8)) : nullptr;
        });
    }

    // The wave's kTileGroups groups: every load first (a group past the end
    // re-reads the last group and is neither computed nor stored), kept in
    // flight together by the scheduling barrier; then compute and store group
    // by group.
    template <bool TAIL>
    __device__ static __forceinline__ void tile(const KArgs &a, float *P, const float *lev,
                                                const float *thr, const float *lds_levels,
                                                const LutEntry *lut, int64_t row0, int64_t groups,
                                                int64_t base, int w, int sub, int slot, _Float16 *eq)
    {
        In buf[kTileGroups];
#pragma unroll
        for (int u = 0; u < kTileGroups; u++) {
            const int gl = TAIL ? (int)(min(base + WAVES * u + w, groups - 1) - base) : WAVES * u + w;
            const int64_t grow = row0 + (int64_t)gl * VPW;
            fetch(a, grow, lane_row<TAIL>(a, grow, slot), sub, buf[u]);
        }
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int u = 0; u < kTileGroups; u++) {
            const int gl = WAVES * u + w;
            if (TAIL && base + gl >= groups)
                break;
            const int64_t grow = row0 + (int64_t)gl * VPW;
            const int lr = lane_row<TAIL>(a, grow, slot);
            if constexpr (GENERIC_SETS)
                lane_params(a.params + (int64_t)set_of(a, grow + lr) * LPV * PL, sub, P);
            compute(a, P, lev, thr, lds_levels, lut, buf[u], grow, lr, sub, u * VPW + slot, eq);
        }
    }
};


}  // namespace
}  // namespace isoq
