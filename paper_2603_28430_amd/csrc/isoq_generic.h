// Stage-1 kernels for vector widths outside {64, 128, 256, 512}: any d from 1 to
// 1024.  Algorithm 1 on the zero-padded vector of Sec. 5.1: when d is not a
// multiple of the block size the last block is filled with zeros, all of its
// rotated coordinates (4g in all, 2-D: 2 g2) are quantized and stored, and
// the padded coordinates are dropped after the inverse rotation.
//
// Layout.  A row spans G lanes (G = 8 .. 64, a power of two) and lane s of
// the row owns the slots s, s + G, ..., s + (BPL - 1) G (a slot is one
// rotation block: 4 coordinates, a quaternion block or two planar pairs, or 8
// coordinates for the 8-D blocks), so consecutive lanes touch consecutive
// slots.  A wave holds 64 / G rows per group and walks
// generic_groups(BPL, SW) groups, issuing every group's loads before computing.  The
// record of a row is written and read bytewise: slot j's SW b index bits start
// at bit SW b j (a whole byte for 8-coordinate slots).  Rows of a width that is a multiple of 4 move in one 8-byte
// (fp16) or 16-byte (fp32) access per slot; fp16 rows of other even widths in
// coordinate pairs (4-byte accesses: such a row starts on a 4-byte boundary,
// PAIRS instantiations); the rest element by element.
//
// Append (MODE_APPEND): the rows are the (token, head) rows of a
// [n_tokens][n_heads][d] tensor in order, row r = token n_heads + head, with
// set r mod n_sets (rows_per_set = 1: set h for head h, or set 0); each row's
// record and norm go to its token's cache row instead of row r.
#pragma once

#include <type_traits>

#include "isoq_device.h"
#include "isoq_stage1.h"

namespace isoq {
namespace {

typedef _Float16 f16x4 __attribute__((ext_vector_type(4)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x8 __attribute__((ext_vector_type(8)));

// Coordinates per slot: one rotation block (two planar pairs for 2-D).
template <int VAR>
constexpr int kGenSW = VAR == VAR_BLOCK8 ? 8 : 4;

// A slot as loaded: SW fp16 values (kept packed until computed) or SW fp32
// values.
template <bool F16, int SW>
using GenRaw = std::conditional_t<F16, std::conditional_t<SW == 8, f16x8, f16x4>,
                                  std::conditional_t<SW == 8, f32x8, f32x4>>;

template <bool F16, int SW>
__device__ __forceinline__ GenRaw<F16, SW> gen_zero()
{
    GenRaw<F16, SW> v;
#pragma unroll
    for (int c = 0; c < SW; c++)
        v[c] = 0;
    return v;
}

// Slot j of a row: one vector access when the row's width is a multiple of
// the slot width (vec), element by element (zero past d) otherwise.
template <bool F16, int SW>
__device__ __forceinline__ GenRaw<F16, SW> gen_load(const char *row, int j, int d, bool vec)
{
    using T = std::conditional_t<F16, _Float16, float>;
    if (vec)
        return *reinterpret_cast<const GenRaw<F16, SW> *>(row + SW * sizeof(T) * j);
    GenRaw<F16, SW> v = gen_zero<F16, SW>();
    const T *e = reinterpret_cast<const T *>(row);
    const int i = SW * j;
#pragma unroll
    for (int c = 0; c < SW; c++)
        if (i + c < d)
            v[c] = e[i + c];
    return v;
}

// fp16 rows of even width d, 2 mod 4: slot j's first pair is inside the row,
// its second unless j is the last slot.
__device__ __forceinline__ f16x4 gen_load_pairs(const char *row, int j, int d)
{
    const f16x2 *q = reinterpret_cast<const f16x2 *>(row) + 2 * j;
    const f16x2 lo = q[0];
    const f16x2 hi = 4 * j + 2 < d ? q[1] : f16x2{(_Float16)0.f, (_Float16)0.f};
    return f16x4{lo[0], lo[1], hi[0], hi[1]};
}

__device__ __forceinline__ void gen_store_pairs(char *row, int j, int d, const float o[4])
{
    f16x2 *q = reinterpret_cast<f16x2 *>(row) + 2 * j;
    q[0] = f16x2{(_Float16)o[0], (_Float16)o[1]};
    if (4 * j + 2 < d)
        q[1] = f16x2{(_Float16)o[2], (_Float16)o[3]};
}

template <bool F16, int SW>
__device__ __forceinline__ void gen_unpack(const GenRaw<F16, SW> &r, float v[SW])
{
#pragma unroll
    for (int c = 0; c < SW; c++)
        v[c] = (float)r[c];
}

template <bool F16, int SW>
__device__ __forceinline__ void gen_store(char *row, int j, int d, bool vec, const float o[SW])
{
    using T = std::conditional_t<F16, _Float16, float>;
    if (vec) {
        GenRaw<F16, SW> h;
#pragma unroll
        for (int c = 0; c < SW; c++)
            h[c] = (T)o[c];
        *reinterpret_cast<GenRaw<F16, SW> *>(row + SW * sizeof(T) * j) = h;
        return;
    }
#pragma unroll
    for (int c = 0; c < SW; c++) {
        const int i = SW * j + c;
        if (i < d) {
            if constexpr (F16)
                reinterpret_cast<_Float16 *>(row)[i] = (_Float16)o[c];
            else
                reinterpret_cast<float *>(row)[i] = o[c];
        }
    }
}

// Where an index record is read from: consecutive bytes, or a paged cache
// (piece-major, as CacheRecRt).
struct RecSrc {
    const uint8_t *rec;
    template <typename T>
    __device__ __forceinline__ T get(int k) const
    {
        return *reinterpret_cast<const T *>(rec + k);
    }
};
struct CacheSrcRt {
    const uint8_t *region;
    int pos, bs, lp, rb;
    template <typename T>
    __device__ __forceinline__ T get(int k) const
    {
        const int64_t o = lp < 0 ? (int64_t)pos * rb + k
                                 : ((((int64_t)(k >> lp)) * bs + pos) << lp) + (k & ((1 << lp) - 1));
        return *reinterpret_cast<const T *>(region + o);
    }
};

// Index bits of slot j (4 coordinates, BITS each) from a record of nb bytes.
template <int BITS, class Src>
__device__ __forceinline__ uint32_t gen_read_slot(const Src &rec, int j, int nb)
{
    auto byte = [&](int k) -> uint32_t { return k < nb ? (uint32_t)rec.template get<uint8_t>(k) : 0u; };
    if constexpr (BITS == 2)
        return byte(j);
    else if constexpr (BITS == 4)
        return byte(2 * j) | (byte(2 * j + 1) << 8);
    else if ((j & 1) == 0)   // bits 12 j .. 12 j + 11 start on a byte boundary
        return byte(3 * j / 2) | ((byte(3 * j / 2 + 1) & 0xFu) << 8);
    else                     // ... or in the middle of byte (3 j - 1) / 2
        return (byte((3 * j - 1) / 2) >> 4) | (byte((3 * j + 1) / 2) << 4);
}

// Write the bytes whose first bit lies in slot j's bit range; `next` is the
// next slot's index bits (only 3 bits per coordinate share a byte between
// slots: the even slot owns it).
template <int BITS, class Dst>
__device__ __forceinline__ void gen_write_slot(const Dst &rec, int j, int nb, uint32_t p, uint32_t next)
{
    auto put = [&](int k, uint32_t v) {
        if (k < nb)
            rec.template put<uint8_t>(k, (uint8_t)v);
    };
    if constexpr (BITS == 2) {
        put(j, p);
    } else if constexpr (BITS == 4) {
        put(2 * j, p);
        put(2 * j + 1, p >> 8);
    } else if ((j & 1) == 0) {
        put(3 * j / 2, p);
        put(3 * j / 2 + 1, (p >> 8) | ((next & 0xFu) << 4));
    } else {
        put((3 * j + 1) / 2, p >> 4);
    }
}

// 8-coordinate slots (8-D blocks): slot j's 8 b bits are bytes [b j, b j + b)
// of the record, so every slot owns whole bytes.
template <int BITS, class Src>
__device__ __forceinline__ uint32_t gen_read_slot8(const Src &rec, int j)
{
    if constexpr (BITS == 2)
        return rec.template get<uint16_t>(2 * j);
    else if constexpr (BITS == 4)
        return rec.template get<uint32_t>(4 * j);
    else
        return (uint32_t)rec.template get<uint8_t>(3 * j) | ((uint32_t)rec.template get<uint8_t>(3 * j + 1) << 8) |
               ((uint32_t)rec.template get<uint8_t>(3 * j + 2) << 16);
}

template <int BITS, class Dst>
__device__ __forceinline__ void gen_write_slot8(const Dst &rec, int j, uint32_t p)
{
    if constexpr (BITS == 2) {
        rec.template put<uint16_t>(2 * j, (uint16_t)p);
    } else if constexpr (BITS == 4) {
        rec.template put<uint32_t>(4 * j, p);
    } else {
        rec.template put<uint8_t>(3 * j, (uint8_t)p);
        rec.template put<uint8_t>(3 * j + 1, (uint8_t)(p >> 8));
        rec.template put<uint8_t>(3 * j + 2, (uint8_t)(p >> 16));
    }
}

// 2 and 3 bits, encoders: the index bits of a slot's 4 coordinates from lane
// masks, as the tuned kernels' ballot_encode does for 8: the top bit of a
// coordinate's index is its sign decision (y > 0) and each lower bit the
// matching bit of the magnitude index (3 bits: a compare with the middle
// positive threshold, then with the one it selects), inverted when y <= 0;
// the masks are pushed into the word from its top, coordinate 3 first.
// Every lane of the wave must call it.
template <int BITS>
__device__ __forceinline__ uint32_t gen_ballot_encode4(const float y[4], const float *ths)
{
    static_assert(BITS == 2 || BITS == 3, "2 or 3 bits");
    uint64_t mk[4 * BITS];
#pragma unroll
    for (int c = 0; c < 4; c++) {
        const int j = 3 - c;
        const float m = fabsf(y[j]);
        uint64_t *o = mk + c * BITS;
        const uint64_t pos = __builtin_amdgcn_ballot_w64(y[j] > 0.f);
        o[0] = pos;
        if constexpr (BITS == 3) {
            const bool hi = m > ths[1];
            const bool lo = m > (hi ? ths[2] : ths[0]);
            o[1] = ~(__builtin_amdgcn_ballot_w64(hi) ^ pos);
            o[2] = ~(__builtin_amdgcn_ballot_w64(lo) ^ pos);
        } else {
            o[1] = ~(__builtin_amdgcn_ballot_w64(m > ths[0]) ^ pos);
        }
    }
    if constexpr (BITS == 3)
        return push_bits12(0u, mk);
    else
        return push_bits8(0u, mk);
}

template <int VAR, int BITS, bool F16, int MODE, int G, int BPL, bool PAIRS>
__global__ __launch_bounds__(kBlockThreads) void generic_kernel(const KArgs a)
{
    constexpr int SW = kGenSW<VAR>;          // coordinates per slot
    static_assert(!PAIRS || (F16 && SW == 4), "pair accesses are for fp16 rows of 4-coordinate slots");
    constexpr int R = 64 / G;                // rows per wave and group
    constexpr int kGenGroups = generic_groups(BPL, SW);
    constexpr int PS = SW == 8 ? 64 : kSlotParams<VAR>;
    constexpr int H = 1 << (BITS - 1);
    constexpr int ESZ = F16 ? 2 : 4;
    constexpr bool kLoadX = MODE != MODE_DEQUANTIZE;
    constexpr bool kAppend = MODE == MODE_APPEND;
    constexpr bool kEncode = MODE == MODE_QUANTIZE || kAppend;
    static_assert(MODE == MODE_ROUNDTRIP || MODE == MODE_QUANTIZE || MODE == MODE_DEQUANTIZE || kAppend, "mode");

    __shared__ float lev_s[16];
    if constexpr (MODE == MODE_DEQUANTIZE) {
        if (threadIdx.x == 0) {
#pragma unroll
            for (int k = 0; k < 2 * H; k++)
                lev_s[k] = a.lev_all[k];
        }
        __syncthreads();
    }

    const int lane = threadIdx.x & 63;
    const int sub = lane & (G - 1);
    const int64_t row0 = ((int64_t)blockIdx.x * (kBlockThreads / 64) + (threadIdx.x >> 6)) * (kGenGroups * R) +
                         lane / G;
    const int d = a.g_d, slots = a.g_slots, nb = a.g_rec;
    const bool vec = a.g_vec != 0;
    const int64_t row_bytes = (int64_t)d * ESZ;
    // the lane's row of group 0; group t is t R rows further (wave-uniform
    // strides, so per-group addresses are one add)
    const char *x0 = kLoadX ? static_cast<const char *>(a.x) + row0 * row_bytes : nullptr;
    char *y0 = !kEncode ? static_cast<char *>(a.y) + row0 * row_bytes : nullptr;
    const uint8_t *ri0 = MODE == MODE_DEQUANTIZE ? a.rec_in + row0 * nb : nullptr;
    uint8_t *ro0 = MODE == MODE_QUANTIZE ? a.rec_out + row0 * nb : nullptr;   // append: per row
    const int64_t xstep = (int64_t)R * row_bytes, rstep = (int64_t)R * nb;

    // ---- loads of every group first
    GenRaw<F16, SW> xr[kLoadX ? kGenGroups : 1][BPL];
    uint32_t pin[kLoadX ? 1 : kGenGroups][BPL];
    float rin[kLoadX ? 1 : kGenGroups];
#pragma unroll
    for (int t = 0; t < kGenGroups; t++) {
        const int64_t row = row0 + (int64_t)t * R;
        const bool ok = row < a.n;
#pragma unroll
        for (int k = 0; k < BPL; k++) {
            const int j = sub + G * k;
            const bool on = ok && j < slots;
            if constexpr (kLoadX) {
                if constexpr (PAIRS)
                    xr[t][k] = on ? gen_load_pairs(x0 + t * xstep, j, d) : gen_zero<F16, SW>();
                else
                    xr[t][k] = on ? gen_load<F16, SW>(x0 + t * xstep, j, d, vec) : gen_zero<F16, SW>();
            } else if constexpr (SW == 8) {
                pin[t][k] = on ? gen_read_slot8<BITS>(RecSrc{ri0 + t * rstep}, j) : 0u;
            } else {
                pin[t][k] = on ? gen_read_slot<BITS>(RecSrc{ri0 + t * rstep}, j, nb) : 0u;
            }
        }
        if constexpr (!kLoadX)
            rin[t] = ok ? a.norms_in[row] : 0.f;
    }

    // ---- rotation parameters of the lane's slots (reloaded when the set changes)
    float P[BPL][PS];
    int64_t pset = -1;
    auto load_set = [&](int64_t set) {
#pragma unroll
        for (int k = 0; k < BPL; k++) {
            const int j = min(sub + G * k, slots - 1);
            load_params<PS>(a.params + set * a.g_set_stride + (int64_t)j * PS, P[k]);
        }
        pset = set;
    };
    if (a.n_sets == 1)
        load_set(0);

#pragma unroll
    for (int t = 0; t < kGenGroups; t++) {
        const int64_t row = row0 + (int64_t)t * R;
        const bool ok = row < a.n;
        if (a.n_sets > 1) {
            const int64_t set = ok ? (row / a.rows_per_set) % a.n_sets : 0;
            if (set != pset)
                load_set(set);
        }
        float yq[BPL][SW];
        uint32_t pk[BPL];
        float rho;
        if constexpr (kLoadX) {
            float xv[BPL][SW];
            float s = 0.f;
#pragma unroll
            for (int k = 0; k < BPL; k++) {
                gen_unpack<F16, SW>(xr[t][k], xv[k]);
#pragma unroll
                for (int c = 0; c < SW; c++)
                    s = fmaf(xv[k][c], xv[k][c], s);
            }
            rho = __builtin_amdgcn_sqrtf(row_sum<G>(s));
            const float rho_e = fmaxf(rho, kEps);
            // thresholds scaled by rho (the rotation is linear, so comparing
            // |T x| with rho t equals comparing |T x / rho| with t); levels
            // scaled by rho give rho * rec directly
            float ths[H > 1 ? H - 1 : 1], lvs[H];
#pragma unroll
            for (int k = 0; k + 1 < H; k++)
                ths[k] = a.thr_pos[k] * rho_e;
#pragma unroll
            for (int k = 0; k < H; k++)
                lvs[k] = a.lev_pos[k] * rho;
#pragma unroll
            for (int k = 0; k < BPL; k++) {
                const int j = sub + G * k;
                float y[SW];
                if constexpr (SW == 8)
                    rotate_forward<VAR>(P[k], xv[k], y);
                else
                    rotate4_forward<VAR>(P[k], xv[k], y);
                uint32_t p = 0;
                if constexpr (kEncode && SW == 4 && BITS <= 3) {
                    p = gen_ballot_encode4<BITS>(y, ths);
                } else {
#pragma unroll
                    for (int c = 0; c < SW; c++) {
                        const float m = fabsf(y[c]);
                        float L = lvs[0];
                        uint32_t cnt = 0;
#pragma unroll
                        for (int q = 0; q + 1 < H; q++) {
                            const bool above = m > ths[q];
                            L = above ? lvs[q + 1] : L;
                            cnt += above ? 1u : 0u;
                        }
                        yq[k][c] = y[c] > 0.f ? L : -L;
                        const uint32_t idx = y[c] > 0.f ? (uint32_t)H + cnt : (uint32_t)(H - 1) - cnt;
                        p |= idx << (BITS * c);
                    }
                }
                // a planar slot past the padded width (its second pair is not
                // a coordinate of the record) and slots past the row carry no bits
                if (VAR == VAR_PLANAR2D && 4 * j + 2 >= a.g_pw)
                    p &= (1u << (2 * BITS)) - 1u;
                pk[k] = (ok && j < slots) ? p : 0u;
            }
        } else {
            rho = rin[t];
#pragma unroll
            for (int k = 0; k < BPL; k++)
#pragma unroll
                for (int c = 0; c < SW; c++)
                    yq[k][c] = lev_s[(pin[t][k] >> (BITS * c)) & (2 * H - 1)] * rho;
        }

        if constexpr (kEncode) {
            // the row's record and norm: row `row`, or (append) the cache
            // row of its token's slot (a skipped slot, < 0 or past the
            // cache, writes nothing)
            bool wr = ok;
            int64_t orow = row;
            int pos = 0;
            if constexpr (kAppend) {
                const uint32_t ru = ok ? (uint32_t)row : 0u;
                const uint32_t token = ru / a.n_heads;
                const uint32_t head = ru - token * a.n_heads;
                orow = cache_slot(a, ok ? a.slots[token] : -1, head, wr, pos);
                wr = wr && ok;
            }
            auto write = [&](const auto &rec) {
#pragma unroll
                for (int k = 0; k < BPL; k++) {
                    const int j = sub + G * k;
                    if constexpr (SW == 8) {
                        if (wr && j < slots)
                            gen_write_slot8<BITS>(rec, j, pk[k]);
                    } else {
                        // the next slot of an even slot sits on the next lane (G is even)
                        const uint32_t next = BITS == 3 ? (uint32_t)__shfl_down((int)pk[k], 1, 64) : 0u;
                        if (wr && j < slots)
                            gen_write_slot<BITS>(rec, j, nb, pk[k], next);
                    }
                }
            };
            if constexpr (kAppend)
                write(CacheRecRt{a.rec_out + (orow - pos) * nb, pos, (int)a.block_size, 0, cache_piece_log2(nb), nb});
            else
                write(RecPtr{ro0 + t * rstep});
            if (wr && sub == 0)
                a.norms_out[orow] = rho;
        } else {
#pragma unroll
            for (int k = 0; k < BPL; k++) {
                const int j = sub + G * k;
                if (ok && j < slots) {
                    float o[SW];
                    if constexpr (SW == 8)
                        rotate_inverse<VAR>(P[k], yq[k], o);
                    else
                        rotate4_inverse<VAR>(P[k], yq[k], o);
                    if constexpr (PAIRS)
                        gen_store_pairs(y0 + t * xstep, j, d, o);
                    else
                        gen_store<F16, SW>(y0 + t * xstep, j, d, vec, o);
                }
            }
        }
    }
}

// Row shape for a padded width of `slots` slots: (G, BPL).
template <int VAR, int BITS, bool F16, int MODE, bool PAIRS>
const void *gen_pick_shape(int slots)
{
    if (slots <= 8)
        return reinterpret_cast<const void *>(&generic_kernel<VAR, BITS, F16, MODE, 8, 1, PAIRS>);
    if (slots <= 16)
        return reinterpret_cast<const void *>(&generic_kernel<VAR, BITS, F16, MODE, 16, 1, PAIRS>);
    if constexpr (kGenSW<VAR> == 4 && !F16) {   // as generic_two_slots
        if (slots <= 32)
            return reinterpret_cast<const void *>(&generic_kernel<VAR, BITS, F16, MODE, 16, 2, PAIRS>);
        if (slots <= 64)
            return reinterpret_cast<const void *>(&generic_kernel<VAR, BITS, F16, MODE, 32, 2, PAIRS>);
    } else {
        if (slots <= 32)
            return reinterpret_cast<const void *>(&generic_kernel<VAR, BITS, F16, MODE, 32, 1, PAIRS>);
        if (slots <= 64)
            return reinterpret_cast<const void *>(&generic_kernel<VAR, BITS, F16, MODE, 64, 1, PAIRS>);
    }
    if (slots <= 128)
        return reinterpret_cast<const void *>(&generic_kernel<VAR, BITS, F16, MODE, 64, 2, PAIRS>);
    // four slots per lane only with 4-coordinate slots (8-coordinate slots
    // of d <= 1024 need at most two)
    if constexpr (kGenSW<VAR> == 4) {
        if (slots <= 256)
            return reinterpret_cast<const void *>(&generic_kernel<VAR, BITS, F16, MODE, 64, 4, PAIRS>);
    }
    return nullptr;
}

template <int VAR, int BITS, bool F16, bool PAIRS>
const void *gen_pick_mode(int slots, int mode)
{
    switch (mode) {
    case MODE_ROUNDTRIP: return gen_pick_shape<VAR, BITS, F16, MODE_ROUNDTRIP, PAIRS>(slots);
    case MODE_QUANTIZE: return gen_pick_shape<VAR, BITS, F16, MODE_QUANTIZE, PAIRS>(slots);
    case MODE_DEQUANTIZE: return gen_pick_shape<VAR, BITS, F16, MODE_DEQUANTIZE, PAIRS>(slots);
    case MODE_APPEND: return gen_pick_shape<VAR, BITS, F16, MODE_APPEND, PAIRS>(slots);
    }
    return nullptr;
}

// pairs: fp16 rows of even width 2 mod 4 (coordinate-pair accesses; not for
// 8-coordinate slots)
template <int VAR, int BITS>
const void *gen_pick_dtype(int slots, bool f16, int mode, bool pairs)
{
    if (!f16)
        return gen_pick_mode<VAR, BITS, false, false>(slots, mode);
    if constexpr (kGenSW<VAR> == 8)
        return pairs ? nullptr : gen_pick_mode<VAR, BITS, true, false>(slots, mode);
    else
        return pairs ? gen_pick_mode<VAR, BITS, true, true>(slots, mode) : gen_pick_mode<VAR, BITS, true, false>(slots, mode);
}

template <int VAR>
const void *gen_pick(int slots, int bits, bool f16, int mode, bool pairs)
{
    switch (bits) {
    case 2: return gen_pick_dtype<VAR, 2>(slots, f16, mode, pairs);
    case 3: return gen_pick_dtype<VAR, 3>(slots, f16, mode, pairs);
    case 4: return gen_pick_dtype<VAR, 4>(slots, f16, mode, pairs);
    }
    return nullptr;
}

}  // namespace
}  // namespace isoq
