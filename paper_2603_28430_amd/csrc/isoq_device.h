// Device helpers shared by the library's kernels (isoq_kernels.hip,
// isoq_scores.hip): vector types, cross-lane reductions, row chunk loads and
// stores, the block rotations of Sec. 5.2-5.4 on a lane's 8 coordinates, and
// division by run-time constants.
#pragma once

#include <hip/hip_runtime.h>

#include "isoq_internal.h"

namespace isoq {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));

constexpr float kEps = 1e-12f;

// DPP controls (data-parallel primitives on 16-lane rows)
constexpr int DPP_QUAD_1032 = 0xB1;   // quad_perm [1,0,3,2]
constexpr int DPP_QUAD_2301 = 0x4E;   // quad_perm [2,3,0,1]
constexpr int DPP_QUAD_1233 = 0xF9;   // quad_perm [1,2,3,3]
constexpr int DPP_ROW_MIRROR = 0x140;
constexpr int DPP_ROW_HALF_MIRROR = 0x141;

template <int CTRL>
__device__ __forceinline__ float dpp_f(float v)
{
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
}

template <int CTRL>
__device__ __forceinline__ uint32_t dpp_u(uint32_t v)
{
    return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, CTRL, 0xF, 0xF, false);
}

// The head a block with grid x index `x` works on, of n_heads.  The
// dispatcher deals blocks to the 8 XCDs in turn (block i to XCD i mod 8, with
// the grid's x index fastest), and each XCD has its own L2.  When a head's
// span of rows or records does not end on a 128-byte line (`shared`),
// adjacent heads share lines, which two XCDs would each fetch from HBM, so
// adjacent heads are kept on one XCD: with n_heads a multiple of 8, block x
// takes head (x mod 8) (n_heads / 8) + x / 8; otherwise head x.
__device__ __forceinline__ uint32_t xcd_head(uint32_t x, uint32_t n_heads, bool shared)
{
    return shared && n_heads % 8 == 0 ? (x % 8) * (n_heads / 8) + x / 8 : x;
}

__device__ __forceinline__ uint32_t fast_div(uint32_t n, const FastDiv &f)
{
    const uint32_t t = __umulhi(n, f.m);
    return (t + ((n - t) >> f.s1)) >> f.s2;
}

// Where an index record goes.  RecPtr: consecutive bytes.  CacheRec<P>: a
// record in a paged cache, pieces of P bytes (cache_piece): record byte k of
// position pos at byte ((k / P) bs + pos) P + k mod P of the head's block
// region.  Every store of n bytes is n-aligned inside the record and n <= P,
// so it never straddles two pieces.  at(k): the record from its byte k on.
struct RecPtr {
    uint8_t *rec;
    template <typename T>
    __device__ __forceinline__ void put(int k, T v) const
    {
        *reinterpret_cast<T *>(rec + k) = v;
    }
    __device__ __forceinline__ RecPtr at(int k) const { return RecPtr{rec + k}; }
};

template <int P>
struct CacheRec {
    uint8_t *region;   // the head's records of one cache block
    int pos, bs, off;
    template <typename T>
    __device__ __forceinline__ void put(int k, T v) const
    {
        const int b = off + k;
        *reinterpret_cast<T *>(region + ((int64_t)(b / P) * bs + pos) * P + (b % P)) = v;
    }
    __device__ __forceinline__ CacheRec at(int k) const { return CacheRec{region, pos, bs, off + k}; }
};

// CacheRec with the piece size known at run time: P = 1 << lp (16 or 8),
// or lp < 0 for records stored whole (P = rb, the record size).
struct CacheRecRt {
    uint8_t *region;
    int pos, bs, off, lp, rb;
    template <typename T>
    __device__ __forceinline__ void put(int k, T v) const
    {
        const int b = off + k;
        const int64_t o = lp < 0 ? (int64_t)pos * rb + b
                                 : ((((int64_t)(b >> lp)) * bs + pos) << lp) + (b & ((1 << lp) - 1));
        *reinterpret_cast<T *>(region + o) = v;
    }
    __device__ __forceinline__ CacheRecRt at(int k) const { return CacheRecRt{region, pos, bs, off + k, lp, rb}; }
};

// CacheRecRt with lp a constant.
template <int LP>
struct CacheRecK {
    uint8_t *region;
    int pos, bs, off, rb;
    template <typename T>
    __device__ __forceinline__ void put(int k, T v) const
    {
        const int b = off + k;
        int64_t o;
        if constexpr (LP < 0)
            o = (int64_t)pos * rb + b;
        else
            o = ((((int64_t)(b >> LP)) * bs + pos) << LP) + (b & ((1 << LP) - 1));
        *reinterpret_cast<T *>(region + o) = v;
    }
    __device__ __forceinline__ CacheRecK at(int k) const { return CacheRecK{region, pos, bs, off + k, rb}; }
};

// lp of CacheRecRt for records of R bytes (as cache_piece).
__device__ __forceinline__ int cache_piece_log2(int64_t R)
{
    return R % 16 == 0 ? 4 : R % 8 == 0 ? 3 : -1;
}

// Slot s of head `head` in a paged cache: slot s is position s mod
// block_size of cache block s / block_size, a block holding [n_heads]
// [block_size] records.  Returns the cache row (block n_heads + head)
// block_size + pos (norms are stored by it) and sets pos; ok is false for a
// skipped slot (s < 0 or past the cache: row 0 and position 0 are returned
// and must not be written).
__device__ __forceinline__ int64_t cache_slot(const KArgs &a, int64_t s, uint32_t head, bool &ok, int &pos)
{
    ok = s >= 0 && s < a.n_slots;
    const uint32_t su = ok ? (uint32_t)s : 0u;
    const uint32_t blk = fast_div(su, a.div_block);
    pos = (int)(su - blk * a.block_size);
    return ((int64_t)blk * a.n_heads + head) * a.block_size + pos;
}

// The record destination of cache row crow at position pos (records of R
// bytes at rec_out).
template <int64_t R>
__device__ __forceinline__ CacheRec<cache_piece(R)> cache_rec(const KArgs &a, int64_t crow, int pos)
{
    return CacheRec<cache_piece(R)>{a.rec_out + (crow - pos) * R, pos, (int)a.block_size, 0};
}

// Sum over the LPV lanes of a row; every lane of the row gets the same bits.
template <int LPV>
__device__ __forceinline__ float row_sum(float v)
{
    static_assert(LPV >= 4 && LPV <= 64 && (LPV & (LPV - 1)) == 0, "4 to 64 lanes, a power of two");
    v += dpp_f<DPP_QUAD_1032>(v);
    v += dpp_f<DPP_QUAD_2301>(v);
    // half mirror: lane i of an 8-lane half takes lane 7 - i (the other quad)
    if constexpr (LPV >= 8)
        v += dpp_f<DPP_ROW_HALF_MIRROR>(v);
    if constexpr (LPV >= 16)
        v += dpp_f<DPP_ROW_MIRROR>(v);
    // across 16-lane rows: v_permlane16_swap exchanges odd rows of its first
    // operand with even rows of its second, v_permlane32_swap the upper half
    // of the first with the lower half of the second; with both operands v,
    // the two results are (v of row r, v of row r ^ 1) (resp. r ^ 2) in the
    // same order on both rows, so every lane adds the same two values
    if constexpr (LPV >= 32) {
        const auto s = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
        v = __uint_as_float(s[0]) + __uint_as_float(s[1]);
    }
    if constexpr (LPV >= 64) {
        const auto s = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
        v = __uint_as_float(s[0]) + __uint_as_float(s[1]);
    }
    return v;
}

template <bool F16>
struct Raw {
    u32x4 w[F16 ? 1 : 2];
};

// A lane's 8 coordinates: one 16-byte piece (fp16), or two (fp32), the
// second `step` bytes after the first.
template <bool F16>
__device__ __forceinline__ void load_row_chunk(const char *p, Raw<F16> &r, int step = 16)
{
    r.w[0] = __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(p));
    if constexpr (!F16)
        r.w[1] = __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(p + step));
}

template <bool F16>
__device__ __forceinline__ void unpack(const Raw<F16> &r, float x[8])
{
    // Vector elements are copied to scalars before __builtin_bit_cast: applied
    // to an ext_vector element lvalue directly, it reads element 0 every time.
    if constexpr (F16) {
#pragma unroll
        for (int k = 0; k < 4; k++) {
            const uint32_t e = r.w[0][k];
            const f16x2 h = __builtin_bit_cast(f16x2, e);
            x[2 * k] = (float)h.x;
            x[2 * k + 1] = (float)h.y;
        }
    } else {
#pragma unroll
        for (int k = 0; k < 4; k++) {
            const uint32_t e0 = r.w[0][k], e1 = r.w[1][k];
            x[k] = __uint_as_float(e0);
            x[4 + k] = __uint_as_float(e1);
        }
    }
}

// Squared norm of one 4-coordinate slot (fp32 rows).
__device__ __forceinline__ float slot_squares(const float *x)
{
    float s = x[0] * x[0];
    s = fmaf(x[1], x[1], s);
    s = fmaf(x[2], x[2], s);
    return fmaf(x[3], x[3], s);
}

// A lane's part of the squared norm.  fp32 rows: the sum of its two slots'
// squared norms, so that a row's total is one balanced tree over its slots in
// order whether a lane owns adjacent slots (added here, then reduced across
// lanes) or slots half a row apart (each half reduced across lanes, then the
// halves added).
template <bool F16>
__device__ __forceinline__ float sum_squares(const Raw<F16> &r, const float x[8])
{
    if constexpr (F16) {
        float s = 0.f;
#pragma unroll
        for (int k = 0; k < 4; k++) {
            const uint32_t e = r.w[0][k];
            const f16x2 h = __builtin_bit_cast(f16x2, e);
            s = __builtin_amdgcn_fdot2(h, h, s, false);
        }
        return s;
    } else {
        return slot_squares(x) + slot_squares(x + 4);
    }
}

template <bool F16>
__device__ __forceinline__ void store_row_chunk(char *p, const float o[8], int step = 16)
{
    u32x4 *q = reinterpret_cast<u32x4 *>(p);
    if constexpr (F16) {
        // fp32 -> fp16 with one explicit v_cvt_pk_f16_f32 (round to nearest
        // even).  Left to itself the compiler folds the last FMA and the
        // conversion into a mixed-precision FMA (rounding once, straight to
        // fp16) in some kernels and not in others, which would let the fused
        // and the two-pass paths round the same value differently.
        u32x4 w;
#pragma unroll
        for (int k = 0; k < 4; k++) {
            uint32_t h;
            asm("v_cvt_pk_f16_f32 %0, %1, %2" : "=v"(h) : "v"(o[2 * k]), "v"(o[2 * k + 1]));
            w[k] = h;
        }
        __builtin_nontemporal_store(w, q);
    } else {
        u32x4 a, b;
#pragma unroll
        for (int k = 0; k < 4; k++) {
            a[k] = __float_as_uint(o[k]);
            b[k] = __float_as_uint(o[4 + k]);
        }
        // plain (write-back) stores: with adjacent pieces each instruction
        // covers half of every 32-byte span of the wave's rows, and L2 merges
        // the two halves before the line goes out (streaming stores wrote such
        // lines out twice)
        q[0] = a;
        *reinterpret_cast<u32x4 *>(p + step) = b;
    }
}

// ---- block rotations -------------------------------------------------------
// Full: y = M v with M = L(q_L) R(conj q_R) (the sandwich of Sec. 5.2 as one
// 4x4 orthogonal matrix, precomputed at init); inverse v = M^T y (Prop. 1).
// Fast: y = q_L v through the left-multiplication matrix of q_L = (a,b,c,d);
// inverse conj(q_L) y = L(q_L)^T y.  2-D: y = R(theta) u, inverse R(-theta).
//
// A slot is 4 consecutive coordinates: one quaternion block, or two planar
// pairs.  Its parameters: Full the 16 floats of M (row-major), Fast q_L,
// 2-D (cos, sin) of each pair.  8-D blocks (VAR_BLOCK8) rotate a lane's 8
// coordinates as one block: y = Q v with the block's 8x8 orthogonal matrix Q
// (64 floats, row-major), inverse v = Q^T y.
template <int VAR>
constexpr int kSlotParams = VAR == VAR_FULL ? 16 : 4;

// Parameter floats of a lane's 8 coordinates.
template <int VAR>
constexpr int kLanePL = VAR == VAR_FULL ? 32 : VAR == VAR_BLOCK8 ? 64 : 8;

template <int VAR>
__device__ __forceinline__ void rotate4_forward(const float *P, const float *v, float *y)
{
    if constexpr (VAR == VAR_FULL) {
#pragma unroll
        for (int r = 0; r < 4; r++) {
            float acc = P[4 * r] * v[0];
            acc = fmaf(P[4 * r + 1], v[1], acc);
            acc = fmaf(P[4 * r + 2], v[2], acc);
            acc = fmaf(P[4 * r + 3], v[3], acc);
            y[r] = acc;
        }
    } else if constexpr (VAR == VAR_FAST) {
        const float a = P[0], b = P[1], c = P[2], d = P[3];
        y[0] = fmaf(-d, v[3], fmaf(-c, v[2], fmaf(-b, v[1], a * v[0])));
        y[1] = fmaf(c, v[3], fmaf(-d, v[2], fmaf(a, v[1], b * v[0])));
        y[2] = fmaf(-b, v[3], fmaf(a, v[2], fmaf(d, v[1], c * v[0])));
        y[3] = fmaf(a, v[3], fmaf(b, v[2], fmaf(-c, v[1], d * v[0])));
    } else {
#pragma unroll
        for (int p = 0; p < 2; p++) {
            const float c = P[2 * p], s = P[2 * p + 1];
            y[2 * p] = fmaf(-s, v[2 * p + 1], c * v[2 * p]);
            y[2 * p + 1] = fmaf(c, v[2 * p + 1], s * v[2 * p]);
        }
    }
}

template <int VAR>
__device__ __forceinline__ void rotate4_inverse(const float *P, const float *y, float *o)
{
    if constexpr (VAR == VAR_FULL) {
#pragma unroll
        for (int c = 0; c < 4; c++) {
            float acc = P[c] * y[0];
            acc = fmaf(P[4 + c], y[1], acc);
            acc = fmaf(P[8 + c], y[2], acc);
            acc = fmaf(P[12 + c], y[3], acc);
            o[c] = acc;
        }
    } else if constexpr (VAR == VAR_FAST) {
        const float a = P[0], b = P[1], c = P[2], d = P[3];
        o[0] = fmaf(d, y[3], fmaf(c, y[2], fmaf(b, y[1], a * y[0])));
        o[1] = fmaf(-c, y[3], fmaf(d, y[2], fmaf(a, y[1], -b * y[0])));
        o[2] = fmaf(b, y[3], fmaf(a, y[2], fmaf(-d, y[1], -c * y[0])));
        o[3] = fmaf(a, y[3], fmaf(-b, y[2], fmaf(c, y[1], -d * y[0])));
    } else {
#pragma unroll
        for (int p = 0; p < 2; p++) {
            const float c = P[2 * p], s = P[2 * p + 1];
            o[2 * p] = fmaf(s, y[2 * p + 1], c * y[2 * p]);
            o[2 * p + 1] = fmaf(c, y[2 * p + 1], -s * y[2 * p]);
        }
    }
}

// A lane's 8 coordinates: two slots, or one 8-D block.
template <int VAR>
__device__ __forceinline__ void rotate_forward(const float *P, const float x[8], float y[8])
{
    if constexpr (VAR == VAR_BLOCK8) {
#pragma unroll
        for (int r = 0; r < 8; r++) {
            float acc = P[8 * r] * x[0];
#pragma unroll
            for (int c = 1; c < 8; c++)
                acc = fmaf(P[8 * r + c], x[c], acc);
            y[r] = acc;
        }
    } else {
        rotate4_forward<VAR>(P, x, y);
        rotate4_forward<VAR>(P + kSlotParams<VAR>, x + 4, y + 4);
    }
}

template <int VAR>
__device__ __forceinline__ void rotate_inverse(const float *P, const float y[8], float o[8])
{
    if constexpr (VAR == VAR_BLOCK8) {
#pragma unroll
        for (int c = 0; c < 8; c++) {
            float acc = P[c] * y[0];
#pragma unroll
            for (int r = 1; r < 8; r++)
                acc = fmaf(P[8 * r + c], y[r], acc);
            o[c] = acc;
        }
    } else {
        rotate4_inverse<VAR>(P, y, o);
        rotate4_inverse<VAR>(P + kSlotParams<VAR>, y + 4, o + 4);
    }
}

template <int PL>
__device__ __forceinline__ void load_params(const float *base, float P[PL])
{
    const u32x4 *q = reinterpret_cast<const u32x4 *>(base);
#pragma unroll
    for (int k = 0; k < PL / 4; k++) {
        const u32x4 w = q[k];
        const uint32_t e0 = w[0], e1 = w[1], e2 = w[2], e3 = w[3];
        P[4 * k] = __uint_as_float(e0);
        P[4 * k + 1] = __uint_as_float(e1);
        P[4 * k + 2] = __uint_as_float(e2);
        P[4 * k + 3] = __uint_as_float(e3);
    }
}

}  // namespace
}  // namespace isoq
