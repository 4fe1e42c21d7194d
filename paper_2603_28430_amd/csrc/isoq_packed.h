// Stage-1 kernels for fp16 rows of width d = 16 k up to 504 outside
// {64, 128, 256} (d = 16, 32, 48, 80, 96, 112, 144, 160, 192, ...): the tuned
// kernels' lane work on rows packed back to back across the wave.
//
// A row spans L = d/8 lanes of 8 coordinates (two quaternion blocks or four
// planar pairs, Sec. 5.2-5.4), as in the tuned kernels, but L need not be a
// power of two: a wave holds V rows of a group one after another, lane
// c < V L owning coordinates 8 (c mod L) .. +7 of row c / L, and the lanes
// past V L idle.  Rows, index records and the rows of a group are contiguous,
// so the group is one stretch of V L eight-coordinate chunks: lane c's piece
// of the rows sits 16 c bytes past the group's first row and its index bits
// at bit 8 b c of the group's records, the layout
// the tuned kernels write for a row of V L lanes.  Only the squared norm
// needs the row boundaries: lanes add their pairs by DPP (L is even, so a
// pair never straddles rows), write the pair sums to LDS, and every lane adds
// its row's L/2 pair sums in order.  With 3 bits the four lanes of a quad
// merge their 24-bit pieces into three words, so V L is kept a multiple of 4
// (the host lowers V by one when it is not); in a ragged last group the
// quad that ends the data writes its last word as a half word.
#pragma once

#include "isoq_stage1.h"

namespace isoq {
namespace {

// Index bits of chunk c (8 coordinates) of a group whose first nv chunks hold
// data; 0 past them.  3 bits: a quad's three words, or the chunk's own three
// bytes where those words would reach past the data (ragged last group).
template <int BITS>
__device__ __forceinline__ uint32_t packed_load_bits(const uint8_t *rec, int c, int nv)
{
    if (c >= nv)
        return 0u;
    if constexpr (BITS == 3) {
        if (4 * ((c >> 2) + 1) > nv) {
            const uint8_t *b = rec + 3 * c;
            return (uint32_t)b[0] | ((uint32_t)b[1] << 8) | ((uint32_t)b[2] << 16);
        }
    }
    return load_bits<BITS>(rec, c);
}

// Write chunk c's index bits (p) to the records of a group with nv chunks of
// data.  Every lane of the wave must call it (3 bits exchanges within quads).
template <int BITS>
__device__ __forceinline__ void packed_store_bits(uint8_t *rec, int c, uint32_t p, int nv)
{
    if constexpr (BITS == 3) {
        // lane k < 3 of a quad writes word 3 (c / 4) + k, whose bytes are
        // those of chunks 4 (c / 4) + k and the next; nv is even, so a word
        // is either whole, half inside the data, or past it
        const uint32_t nb = dpp_u<DPP_QUAD_1233>(p);
        const int k = c & 3;
        const int off = 4 * (3 * (c >> 2) + k);
        const uint32_t wv = (p >> (8 * k)) | (nb << (24 - 8 * k));
        if (k < 3) {
            if (off + 4 <= 3 * nv)
                *reinterpret_cast<uint32_t *>(rec + off) = wv;
            else if (off + 2 <= 3 * nv)
                *reinterpret_cast<uint16_t *>(rec + off) = (uint16_t)wv;
        }
    } else if (c < nv) {
        if constexpr (BITS == 2)
            reinterpret_cast<uint16_t *>(rec)[c] = (uint16_t)p;
        else
            reinterpret_cast<uint32_t *>(rec)[c] = p;
    }
}

// Sum of the n (1 .. 32) pair sums at rp, in index order.  n is split into
// blocks of 16, 8, 4, 2 and 1 whose loads are issued together, so a row costs
// at most five LDS round trips (two at d = 80, 96, 160 and 192) rather than
// one per pair.
__device__ __forceinline__ float packed_pair_total(const float *rp, int n)
{
    float tot = 0.f;
    int i = 0;
#pragma unroll
    for (int blk = 16; blk >= 1; blk >>= 1) {
        if (n & blk) {
            float v[16];
#pragma unroll
            for (int j = 0; j < blk; j++)
                v[j] = rp[i + j];
#pragma unroll
            for (int j = 0; j < blk; j++)
                tot += v[j];
            i += blk;
        }
    }
    return tot;
}

template <int VAR, int BITS, bool F16, int MODE>
__global__ __launch_bounds__(kBlockThreads) void packed_kernel(const KArgs a)
{
    constexpr int H = 1 << (BITS - 1);
    constexpr int PL = VAR == VAR_FULL ? 32 : 8;   // parameter floats per lane
    constexpr int LANEB = F16 ? 16 : 32;           // row bytes per lane
    constexpr bool kUseLut = BITS == 4;
    constexpr bool kEncode = MODE == MODE_QUANTIZE;
    constexpr bool kLoadX = MODE != MODE_DEQUANTIZE;
    static_assert(MODE == MODE_ROUNDTRIP || MODE == MODE_QUANTIZE || MODE == MODE_DEQUANTIZE, "mode");

    __shared__ float lds_levels[16];
    __shared__ __align__(16) LutEntry lds_lut[kUseLut && kLoadX ? kLutMaxCells : 1];
    __shared__ float lds_pairs[kBlockThreads / 2];   // 32 pair sums per wave
    // Full's 128 bytes per lane are staged through LDS when the block has one
    // set (per-lane global loads of them move more through the vector memory
    // pipe than the rows do); Fast and 2-D read their 32 bytes directly,
    // which measured faster than a staging barrier
    constexpr bool kStage = VAR == VAR_FULL;
    __shared__ __align__(16) float lds_params[kStage ? kPackedMaxLanes * PL : 4];

    const int L = a.g_d >> 3;   // lanes per row (even)
    const int V = a.g_rows;     // rows per group
    const int lane = threadIdx.x & 63;
    const int q = lane / L;
    const int sub = lane - q * L;         // chunk of the lane within its row
    const int lr = min(q, V - 1);         // row of the lane in the group (idle lanes: the last)
    const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int64_t rowb = (int64_t)a.g_d * (F16 ? 2 : 4);
    const int64_t recb = (int64_t)L * BITS;   // d b / 8
    const int64_t base = (int64_t)blockIdx.x * (kBlockThreads / 64) * kTileGroups;

    if constexpr (MODE == MODE_DEQUANTIZE) {
        if (threadIdx.x < 2 * H)
            lds_levels[threadIdx.x] = a.lev_all[threadIdx.x];
    }
    if constexpr (kUseLut && kLoadX) {
        const u32x4 *s4 = reinterpret_cast<const u32x4 *>(a.lut);
        u32x4 *d4 = reinterpret_cast<u32x4 *>(lds_lut);
        for (int i = threadIdx.x; i < a.lut_cells; i += kBlockThreads)
            d4[i] = s4[i];
    }
    // rotation parameters of the lane's two slots: once, when the whole block
    // has one set; otherwise per group, when the lane's set changes
    const bool uni = a.g_block_set != 0;
    const int64_t bset = a.n_sets == 1 || !uni ? 0 : (base * V / a.rows_per_set) % a.n_sets;
    if (kStage && uni) {
        const u32x4 *s4 = reinterpret_cast<const u32x4 *>(a.params + bset * a.g_set_stride);
        u32x4 *d4 = reinterpret_cast<u32x4 *>(lds_params);
        for (int i = threadIdx.x; i < L * (PL / 4); i += kBlockThreads)
            d4[i] = s4[i];
    }
    if (MODE == MODE_DEQUANTIZE || (kUseLut && kLoadX) || (kStage && uni))
        __syncthreads();
    float P[PL];
    int64_t pset = -1;
    auto load_set = [&](int64_t set) {
        load_params<PL>(a.params + set * a.g_set_stride + (int64_t)sub * PL, P);
        pset = set;
    };
    if (uni) {
        if constexpr (kStage)
            load_params<PL>(lds_params + sub * PL, P);
        else
            load_set(bset);
    }
    float lev[H], thr[H > 1 ? H - 1 : 1];
#pragma unroll
    for (int k = 0; k < H; k++)
        lev[k] = a.lev_pos[k];
#pragma unroll
    for (int k = 0; k < H - 1; k++)
        thr[k] = a.thr_pos[k];

    // ---- the wave's kTileGroups groups (4u + w of the block's): every load
    //      first, then compute and store group by group
    Raw<F16> raw[kLoadX ? kTileGroups : 1];
    uint32_t bin[kLoadX ? 1 : kTileGroups];
    float rin[kLoadX ? 1 : kTileGroups];
#pragma unroll
    for (int u = 0; u < kTileGroups; u++) {
        // a group past the end re-reads group 0 (and is neither computed nor stored)
        const int64_t g0 = (base + 4 * u + w) * V;
        const int64_t grow = g0 < a.n ? g0 : 0;
        const int nv = (int)min((int64_t)V, a.n - grow) * L;   // chunks of data in the group
        const int c = lane < nv ? lane : 0;                    // lanes past them read chunk 0
        if constexpr (kLoadX) {
            load_row_chunk<F16>(static_cast<const char *>(a.x) + grow * rowb + (uint32_t)(c * LANEB), raw[u]);
        } else {
            bin[u] = packed_load_bits<BITS>(a.rec_in + grow * recb, lane, nv);
            rin[u] = (a.norms_in + grow)[lane < nv ? lr : 0];
        }
    }
    __builtin_amdgcn_sched_barrier(0);

    float *pairs = lds_pairs + w * 32;
#pragma unroll
    for (int u = 0; u < kTileGroups; u++) {
        const int64_t grow = (base + 4 * u + w) * V;
        if (grow >= a.n)
            break;
        const int nv = (int)min((int64_t)V, a.n - grow) * L;
        const bool on = lane < nv;
        if (!uni) {
            const int64_t set = ((grow + (on ? lr : 0)) / a.rows_per_set) % a.n_sets;
            if (set != pset)
                load_set(set);
        }
        float yq[8], rho;
        if constexpr (kLoadX) {
            float x[8];
            unpack<F16>(raw[u], x);
            // squared norm: pair sums by DPP, then the row's L/2 pair sums
            // through LDS, added in order by every lane of the row
            float ss = sum_squares<F16>(raw[u], x);
            ss += dpp_f<DPP_QUAD_1032>(ss);
            pairs[lane >> 1] = ss;
            __builtin_amdgcn_wave_barrier();
            const float tot = packed_pair_total(pairs + lr * (L >> 1), L >> 1);
            __builtin_amdgcn_wave_barrier();
            rho = __builtin_amdgcn_sqrtf(tot);
            const float rho_e = fmaxf(rho, kEps);
            float y[8], m[8];
            rotate_forward<VAR>(P, x, y);
#pragma unroll
            for (int j = 0; j < 8; j++)
                m[j] = fabsf(y[j]);
            uint32_t p = 0;
            if constexpr (kUseLut) {
                const float s = a.lut_inv_h * __builtin_amdgcn_rcpf(rho_e);
                p = lut_quantize<BITS, !kEncode, kEncode>(y, m, s, (float)(a.lut_cells - 1), lds_lut, rho, yq);
            } else {
                float ths[H > 1 ? H - 1 : 1];
#pragma unroll
                for (int k = 0; k < H - 1; k++)
                    ths[k] = thr[k] * rho_e;
                if constexpr (kEncode) {
                    p = ballot_encode<BITS, false>(y, m, ths, lev, yq);
                } else {
                    float lvs[H];
#pragma unroll
                    for (int k = 0; k < H; k++)
                        lvs[k] = lev[k] * rho;
                    chain_levels<H>(y, m, ths, lvs, yq);
                }
            }
            if constexpr (kEncode) {
                packed_store_bits<BITS>(a.rec_out + grow * recb, lane, p, nv);
                if (on && sub == 0)
                    (a.norms_out + grow)[lr] = rho;
                continue;
            }
        } else {
            rho = rin[u];
#pragma unroll
            for (int j = 0; j < 8; j++)
                yq[j] = lds_levels[(bin[u] >> (BITS * j)) & (2 * H - 1)] * rho;
        }
        if constexpr (!kEncode) {
            float o[8];
            rotate_inverse<VAR>(P, yq, o);
            if (on)
                store_row_chunk<F16>(static_cast<char *>(a.y) + grow * rowb + (uint32_t)(lane * LANEB), o);
        }
    }
}

template <int VAR, int BITS>
const void *packed_pick_mode(int mode)
{
    switch (mode) {
    case MODE_ROUNDTRIP: return reinterpret_cast<const void *>(&packed_kernel<VAR, BITS, true, MODE_ROUNDTRIP>);
    case MODE_QUANTIZE: return reinterpret_cast<const void *>(&packed_kernel<VAR, BITS, true, MODE_QUANTIZE>);
    case MODE_DEQUANTIZE: return reinterpret_cast<const void *>(&packed_kernel<VAR, BITS, true, MODE_DEQUANTIZE>);
    }
    return nullptr;
}

// fp16 rows only: fp32 rows keep the generic kernels, whose slot-strided
// lanes make every 16-byte access instruction cover one contiguous span
// (measured at d = 96: 0.71 of the HBM roofline for the round trip, against
// 0.60-0.64 with a lane's 32 contiguous bytes)
template <int VAR>
const void *packed_pick(int bits, int mode)
{
    switch (bits) {
    case 2: return packed_pick_mode<VAR, 2>(mode);
    case 3: return packed_pick_mode<VAR, 3>(mode);
    case 4: return packed_pick_mode<VAR, 4>(mode);
    }
    return nullptr;
}

}  // namespace
}  // namespace isoq
