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
//
// Where it keeps more lanes busy (d = 192: 60 lanes instead of 48; d = 320,
// and 288 at 2 and 4 bits) a lane owns two chunks instead, sub and sub + L of
// its row with L = d/16 lanes per row: each 16-byte access instruction then
// covers the first or the second halves of the wave's rows, its index bits go
// to the two halves of the row's record (row-relative addressing; with 3 bits
// L is a multiple of 4, so quads stay inside a row), and a wave walks half as
// many groups so that the same bytes are in flight.
//
// Append (MODE_APPEND, fp16 K/V rows into the slots of a paged cache, at
// d = 80, 96, 160 and 192): block (x, y, z) = (head, token range, K or V) as
// in the tuned append, the rows of a group are consecutive tokens of one head
// (row-relative addressing, input stride n_heads d), and each row's record
// and norm go to its token's cache row.  With 3 bits L is a multiple of 4 at
// 96, 160 and 192, so quads stay inside a row; at 80 (L = 10) lane pairs
// write the record in half-words.
//
// With the stage-2 sketch (MODE_QJL: quantize into rows with one rotation
// set; MODE_APPEND_QJL: into cache slots, one set per head) the width is a
// compile-time D (80, 96, 160, 192): each lane also writes its chunk's
// normalised error e = y / rho' - c[idx] as fp16 to the wave's LDS tile (row
// u V + q for row q of group u, zero columns up to the projection width, a
// multiple of 32), gamma = rho ||e|| is summed over the row like the squared
// norm, and after the tile's groups the wave projects its tile through
// S' = S T^{-1} (qjl_project) and writes the sign bits.  Blocks walk
// g_tpb consecutive tiles, so the staged projection serves several.
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

// 3 bits, rows of a lane count that is even but not a multiple of 4 (d = 80):
// lane sub's 24 bits go to byte 3 sub of the row's record through lane pairs
// (rows start on even lanes): the even lane writes bytes 6 i .. 6 i + 3 (its
// bits and the odd lane's first 8) as two half-words, the odd lane bytes
// 6 i + 4 .. 6 i + 5.  Every lane of the wave must call it (DPP exchange).
template <class Dst>
__device__ __forceinline__ void store_bits3_pairs(const Dst &rec, int sub, uint32_t p, bool ok)
{
    const uint32_t o = dpp_u<DPP_QUAD_1032>(p);   // the pair partner's bits
    const int h = 6 * (sub >> 1);
    if (ok) {
        if ((sub & 1) == 0) {
            rec.template put<uint16_t>(h, (uint16_t)p);
            rec.template put<uint16_t>(h + 2, (uint16_t)((p >> 16) | (o << 8)));
        } else {
            rec.template put<uint16_t>(h + 4, (uint16_t)(p >> 8));
        }
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

template <int VAR, int BITS, int MODE, int C, int D = 0, int QM = 0, int WAVES = kBlockThreads / 64, int LP = 0>
__device__ __forceinline__ void packed_body(const KArgs &a)
{
    constexpr int BT = WAVES * 64;   // threads per block
    constexpr int H = 1 << (BITS - 1);
    constexpr int PL = kLanePL<VAR>;               // parameter floats per chunk
    constexpr bool kQjl = MODE == MODE_QJL || MODE == MODE_APPEND_QJL;
    // groups per wave (4 C chunks in flight per lane; with the sketch a
    // wave's rows fill at most one 16-row projection block)
    constexpr int GPW = packed_groups(kQjl ? packed_shape(D, BITS, true).rows : 1, C, kQjl);
    constexpr bool kUseLut = BITS == 4;
    constexpr bool kAppend = MODE == MODE_APPEND || MODE == MODE_APPEND_QJL;
    constexpr bool kEncode = MODE == MODE_QUANTIZE || MODE == MODE_QJL || kAppend;
    constexpr bool kLoadX = MODE != MODE_DEQUANTIZE;
    static_assert(MODE == MODE_ROUNDTRIP || MODE == MODE_QUANTIZE || MODE == MODE_DEQUANTIZE || kAppend || kQjl,
                  "mode");
    static_assert(C == 1 || C == 2, "one or two chunks per lane");
    // the sketch's tile: QV rows per group, TR rows per wave, rows of ES
    // halfs (DP projected coordinates, then padding)
    static_assert(!kQjl || (D > 0 && QM > 0 && packed_shape(D, BITS, true).chunks == C), "sketch shape");
    constexpr int QV = kQjl ? packed_shape(D, BITS, true).rows : 1;
    constexpr int DP = kQjl ? qjl_proj_width(D) : 32;
    constexpr int TR = kQjl ? GPW * QV : 1;
    // widths whose projection width is a multiple of 64 (d = 192) keep rows
    // unpadded with swizzled chunk positions (err_swizzle), which keeps the
    // block's LDS under half the CU's
    constexpr bool kSwz = DP % 64 == 0;
    constexpr int ES = kSwz ? DP : DP + 8;
    __shared__ __align__(16) _Float16 lds_frag[kQjl ? QM * DP : 8];
    __shared__ __align__(16) _Float16 lds_e[kQjl ? WAVES * TR * ES : 8];
    // append with the sketch: each tile row's cache row (-1: a skipped
    // slot), from the encoder for the sketch's sign rows.  Not at d = 192,
    // whose block sits just under half the CU's LDS (the array would cost
    // the second block: 7% slower); there the sketch finds it from the slot.
    constexpr bool kCrowLds = kQjl && kAppend && !kSwz;
    __shared__ int64_t lds_crow[kCrowLds ? WAVES * TR : 1];

    __shared__ float lds_levels[16];
    __shared__ __align__(16) LutEntry lds_lut[kUseLut && kLoadX ? kLutMaxCells : 1];
    __shared__ float lds_pairs[BT / 2];   // 32 pair sums per wave
    // Full's 128 bytes per chunk (8-D: 256) are staged through LDS when the
    // block has one set (per-lane global loads of them move more through the
    // vector memory pipe than the rows do); Fast and 2-D read their 32 bytes
    // directly, which measured faster than a staging barrier
    constexpr bool kStage = VAR == VAR_FULL || VAR == VAR_BLOCK8;
    __shared__ __align__(16) float lds_params[kStage ? kPackedMaxLanes * PL : 4];

    const int L = a.g_d >> (C + 2);   // lanes per row (even): d / (8 C)
    const int V = a.g_rows;           // rows per group
    const int lane = threadIdx.x & 63;
    const int q = lane / L;
    const int sub = lane - q * L;     // the lane's chunks of its row: sub, sub + L (C = 2)
    const int lr = min(q, V - 1);     // row of the lane in the group (idle lanes: the last)
    const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int64_t rowb = (int64_t)a.g_d * 2;       // fp16 rows
    const int64_t recb = (int64_t)L * C * BITS;    // d b / 8
    const int TPB = kQjl ? a.g_tpb : kAppend ? 1 : packed_tiles_per_block(VAR, C);   // row tiles per block
    const int64_t base0 = (int64_t)(kAppend ? blockIdx.y : blockIdx.x) * TPB * WAVES * GPW;
    // append: the block's head, its input row stride and cache addressing
    const int64_t head = kAppend ? (int64_t)xcd_head(blockIdx.x, a.n_heads, rowb % 128 != 0) : 0;
    const int64_t xstride = kAppend ? (int64_t)a.n_heads * rowb : rowb;

    if constexpr (MODE == MODE_DEQUANTIZE) {
        if (threadIdx.x < 2 * H)
            lds_levels[threadIdx.x] = a.lev_all[threadIdx.x];
    }
    if constexpr (kUseLut && kLoadX) {
        const u32x4 *s4 = reinterpret_cast<const u32x4 *>(a.lut);
        u32x4 *d4 = reinterpret_cast<u32x4 *>(lds_lut);
        for (int i = threadIdx.x; i < a.lut_cells; i += BT)
            d4[i] = s4[i];
    }
    // rotation parameters of the lane's chunks: once, when the whole block
    // has one set; otherwise per group, when the lane's set changes
    const bool uni = kAppend || a.g_block_set != 0;
    const int64_t bset = a.n_sets == 1 || !uni ? 0 : kAppend ? head : (base0 * V / a.rows_per_set) % a.n_sets;
    if (kStage && uni) {
        const u32x4 *s4 = reinterpret_cast<const u32x4 *>(a.params + bset * a.g_set_stride);
        u32x4 *d4 = reinterpret_cast<u32x4 *>(lds_params);
        for (int i = threadIdx.x; i < C * L * (PL / 4); i += BT)
            d4[i] = s4[i];
    }
    if constexpr (kQjl) {
        // the set's projection, and zeros for the error tiles (columns past
        // d, and rows a ragged tile leaves unwritten, stay zero)
        const u32x4 *f4 = reinterpret_cast<const u32x4 *>(a.qjl_frag + bset * (int64_t)(QM * DP));
        u32x4 *g4 = reinterpret_cast<u32x4 *>(lds_frag);
        for (int i = threadIdx.x; i < QM * DP / 8; i += BT)
            g4[i] = f4[i];
        u32x4 *e4 = reinterpret_cast<u32x4 *>(lds_e);
        for (int i = threadIdx.x; i < WAVES * TR * ES / 8; i += BT)
            e4[i] = u32x4{0u, 0u, 0u, 0u};
    }
    if (MODE == MODE_DEQUANTIZE || (kUseLut && kLoadX) || (kStage && uni) || kQjl)
        __syncthreads();
    float P[C][PL];
    int64_t pset = -1;
    auto load_set = [&](int64_t set) {
#pragma unroll
        for (int k = 0; k < C; k++)
            load_params<PL>(a.params + set * a.g_set_stride + (int64_t)(sub + k * L) * PL, P[k]);
        pset = set;
    };
    if (uni) {
        if constexpr (kStage) {
#pragma unroll
            for (int k = 0; k < C; k++)
                load_params<PL>(lds_params + (sub + k * L) * PL, P[k]);
        } else {
            load_set(bset);
        }
    }
    float lev[H], thr[H > 1 ? H - 1 : 1];
#pragma unroll
    for (int k = 0; k < H; k++)
        lev[k] = a.lev_pos[k];
#pragma unroll
    for (int k = 0; k < H - 1; k++)
        thr[k] = a.thr_pos[k];

    // ---- per tile, the wave's GPW groups (WAVES u + w of the tile's): every load
    //      first, then compute and store group by group.  One chunk per
    //      lane: a group is one stretch of V L chunks (flat addressing, chunk
    //      = lane); two: lane sub of row q owns chunks sub and sub + L of that
    //      row.  The tile test is block-uniform (no barrier follows).
    for (int tt = 0; tt < TPB; tt++) {
        const int64_t base = base0 + (int64_t)tt * WAVES * GPW;
        if (base * V >= a.n)
            return;
        Raw<true> raw[kLoadX ? GPW : 1][C];
        uint32_t bin[kLoadX ? 1 : GPW][C];
        float rin[kLoadX ? 1 : GPW];
        int64_t slot[kAppend ? GPW : 1];   // append: each row's cache slot, loaded with the row
#pragma unroll
        for (int u = 0; u < GPW; u++) {
            // a group past the end re-reads group 0 (and is neither computed nor stored)
            const int64_t g0 = (base + WAVES * u + w) * V;
            const int64_t grow = g0 < a.n ? g0 : 0;
            const int rows = (int)min((int64_t)V, a.n - grow);   // rows of data in the group
            const int nv = rows * L;                               // lanes holding data
            const int rq = q < rows ? q : 0;                       // lanes past them read row 0
            if constexpr (kLoadX) {
                const char *row = static_cast<const char *>(a.x) + (grow + rq) * xstride + head * rowb;
#pragma unroll
                for (int k = 0; k < C; k++)
                    load_row_chunk<true>(row + (uint32_t)((sub + k * L) * 16), raw[u][k]);
                if constexpr (kAppend)
                    slot[u] = (a.slots + grow)[rq];
            } else {
                if constexpr (C == 1) {
                    bin[u][0] = packed_load_bits<BITS>(a.rec_in + grow * recb, lane, nv);
                } else {
                    const uint8_t *rec = a.rec_in + (grow + rq) * recb;
#pragma unroll
                    for (int k = 0; k < C; k++)
                        bin[u][k] = load_bits<BITS>(rec + k * L * BITS, sub);
                }
                rin[u] = (a.norms_in + grow)[rq];
            }
        }
        __builtin_amdgcn_sched_barrier(0);

        float *pairs = lds_pairs + w * 32;
#pragma unroll
        for (int u = 0; u < GPW; u++) {
            const int64_t grow = (base + WAVES * u + w) * V;
            if (grow >= a.n)
                break;
            const int rows = (int)min((int64_t)V, a.n - grow);
            const int nv = rows * L;
            const bool on = lane < nv;
            if (!uni) {
                const int64_t set = ((grow + (on ? lr : 0)) / a.rows_per_set) % a.n_sets;
                if (set != pset)
                    load_set(set);
            }
            float yq[C][8], rho;
            float gamma = 0.f;   // with the sketch: rho ||e|| of the lane's row
            if constexpr (kLoadX) {
                float x[C][8];
                // squared norm: the lane's chunks, pair sums by DPP, then the
                // row's L/2 pair sums through LDS, added in order by every lane
                float ss = 0.f;
#pragma unroll
                for (int k = 0; k < C; k++) {
                    unpack<true>(raw[u][k], x[k]);
                    ss += sum_squares<true>(raw[u][k], x[k]);
                }
                ss += dpp_f<DPP_QUAD_1032>(ss);
                pairs[lane >> 1] = ss;
                __builtin_amdgcn_wave_barrier();
                const float tot = packed_pair_total(pairs + lr * (L >> 1), L >> 1);
                __builtin_amdgcn_wave_barrier();
                rho = __builtin_amdgcn_sqrtf(tot);
                const float rho_e = fmaxf(rho, kEps);
                float ths[H > 1 ? H - 1 : 1], lvs[H];
#pragma unroll
                for (int k = 0; k < H - 1; k++)
                    ths[k] = thr[k] * rho_e;
#pragma unroll
                for (int k = 0; k < H; k++)
                    lvs[k] = lev[k] * rho;
                // with the sketch the selected levels are the normalised
                // ones, zero for a zero row (whose y is zero), so that e is
                // zero there
                const float nz = rho > 0.f ? 1.f : 0.f;
                float levq[H];
#pragma unroll
                for (int k = 0; k < H; k++)
                    levq[k] = lev[k] * nz;
                float s2 = 0.f;
                uint32_t p[C];
#pragma unroll
                for (int k = 0; k < C; k++) {
                    float y[8], m[8];
                    rotate_forward<VAR>(P[k], x[k], y);
#pragma unroll
                    for (int j = 0; j < 8; j++)
                        m[j] = fabsf(y[j]);
                    if constexpr (kUseLut) {
                        const float s = a.lut_inv_h * __builtin_amdgcn_rcpf(rho_e);
                        p[k] = lut_quantize<BITS, !kEncode || kQjl, kEncode>(y, m, s, (float)(a.lut_cells - 1),
                                                                             lds_lut, kQjl ? nz : rho, yq[k]);
                    } else if constexpr (kQjl) {
                        p[k] = ballot_encode<BITS, true>(y, m, ths, levq, yq[k]);
                    } else if constexpr (kEncode) {
                        p[k] = ballot_encode<BITS, false>(y, m, ths, lev, yq[k]);
                    } else {
                        chain_levels<H>(y, m, ths, lvs, yq[k]);
                    }
                    if constexpr (kQjl) {
                        // e = y / rho' - c[idx] to the wave's tile as fp16
                        const float inv = __builtin_amdgcn_rcpf(rho_e);
                        float e[8];
#pragma unroll
                        for (int j = 0; j < 8; j++) {
                            e[j] = fmaf(y[j], inv, -yq[k][j]);
                            s2 = fmaf(e[j], e[j], s2);
                        }
                        u32x4 hv;
#pragma unroll
                        for (int i = 0; i < 4; i++) {
                            uint32_t h2;
                            asm("v_cvt_pk_f16_f32 %0, %1, %2" : "=v"(h2) : "v"(e[2 * i]), "v"(e[2 * i + 1]));
                            hv[i] = h2;
                        }
                        if (on) {
                            const int er = u * QV + q, ec = sub + k * L;
                            *reinterpret_cast<u32x4 *>(lds_e + (w * TR + er) * ES +
                                                       8 * (kSwz ? ec ^ err_swizzle(er) : ec)) = hv;
                        }
                    }
                }
                if constexpr (kQjl) {
                    // gamma: the row's sum of e^2 as its squared norm above
                    s2 += dpp_f<DPP_QUAD_1032>(s2);
                    pairs[lane >> 1] = s2;
                    __builtin_amdgcn_wave_barrier();
                    const float t2 = packed_pair_total(pairs + lr * (L >> 1), L >> 1);
                    __builtin_amdgcn_wave_barrier();
                    gamma = rho * __builtin_amdgcn_sqrtf(t2);
                }
                if constexpr (kAppend) {
                    bool ok;
                    int pos;
                    const int64_t cr = cache_slot(a, slot[u], head, ok, pos);
                    if constexpr (kCrowLds) {
                        if (on && sub == 0)
                            lds_crow[w * TR + u * QV + q] = ok ? cr : -1;
                    }
                    auto store = [&](const auto &rec) {
                        if (BITS == 3 && L % 4 != 0) {
                            // d = 80: quads would straddle rows
                            store_bits3_pairs(rec, sub, p[0], on && ok);
                        } else {
#pragma unroll
                            for (int k = 0; k < C; k++)
                                store_bits_to<BITS>(rec.at(k * L * BITS), sub, p[k], on && ok);
                        }
                    };
                    // the cache layout's pieces: from the width where it is a
                    // constant, else from the kernel's LP
                    if constexpr (D > 0)
                        store(cache_rec<(int64_t)D * BITS / 8>(a, cr, pos));
                    else
                        store(CacheRecK<LP>{a.rec_out + (cr - pos) * recb, pos, (int)a.block_size, 0, (int)recb});
                    if (on && ok && sub == 0) {
                        a.norms_out[cr] = rho;
                        if constexpr (kQjl)
                            a.qjl_gamma[cr] = gamma;
                    }
                    continue;
                } else if constexpr (kEncode) {
                    if constexpr (C == 1) {
                        packed_store_bits<BITS>(a.rec_out + grow * recb, lane, p[0], nv);
                    } else {
                        // row-relative: with 3 bits L is a multiple of 4, so quads
                        // stay inside a row and each half record starts on a word
                        uint8_t *rec = a.rec_out + (grow + lr) * recb;
#pragma unroll
                        for (int k = 0; k < C; k++)
                            store_bits<BITS>(rec + k * L * BITS, sub, p[k], on);
                    }
                    if (on && sub == 0) {
                        (a.norms_out + grow)[lr] = rho;
                        if constexpr (kQjl)
                            (a.qjl_gamma + grow)[lr] = gamma;
                    }
                    continue;
                }
            } else {
                rho = rin[u];
#pragma unroll
                for (int k = 0; k < C; k++)
#pragma unroll
                    for (int j = 0; j < 8; j++)
                        yq[k][j] = lds_levels[(bin[u][k] >> (BITS * j)) & (2 * H - 1)] * rho;
            }
            if constexpr (!kEncode) {
                char *row = static_cast<char *>(a.y) + (grow + lr) * rowb;
#pragma unroll
                for (int k = 0; k < C; k++) {
                    float o[8];
                    rotate_inverse<VAR>(P[k], yq[k], o);
                    if (on)
                        store_row_chunk<true>(row + (uint32_t)((sub + k * L) * 16), o);
                }
            }
        }
        if constexpr (kQjl) {
            // the tile's projection: tile row ar is row ar mod QV of group
            // ar / QV of the wave
            qjl_project<DP, QM, TR, ES, kSwz>(lds_frag, lds_e + w * TR * ES, [&](int ar) -> uint32_t * {
                if (ar >= TR)
                    return nullptr;
                const int gu = ar / QV;
                const int64_t row = (base + WAVES * gu + w) * QV + (ar - gu * QV);
                if (row >= a.n)
                    return nullptr;
                int64_t orow = row;
                if constexpr (kCrowLds) {
                    orow = lds_crow[w * TR + ar];   // the encoder's cache row of tile row ar
                    if (orow < 0)
                        return nullptr;
                } else if constexpr (kAppend) {
                    bool ok;
                    int pos;
                    orow = cache_slot(a, a.slots[row], head, ok, pos);
                    if (!ok)
                        return nullptr;
                }
                return reinterpret_cast<uint32_t *>(a.qjl_signs + orow * (QM / 8));
            });
        }
    }
}

template <int VAR, int BITS, int MODE, int C>
__global__ __launch_bounds__(kBlockThreads) void packed_kernel(const KArgs a)
{
    packed_body<VAR, BITS, MODE, C>(a);
}

// K and V in one launch: blockIdx.z = 0 encodes the keys, 1 the values.
// LP: the cache layout's pieces (1 << LP bytes, or records whole for -1).
template <int VAR, int BITS, int C, int LP>
__global__ __launch_bounds__(kBlockThreads) void packed_append_kernel(const KArgs k, const KArgs v)
{
    packed_body<VAR, BITS, MODE_APPEND, C, 0, 0, kBlockThreads / 64, LP>(blockIdx.z == 0 ? k : v);
}

// With the stage-2 sketch: width D, m = QM sign bits, kPackedQjlWaves waves
// per block (one staged projection for twice the waves of the other modes).
template <int VAR, int D, int BITS, int MODE, int QM>
__global__ __launch_bounds__(kPackedQjlWaves * 64) void packed_qjl_kernel(const KArgs a)
{
    packed_body<VAR, BITS, MODE, packed_shape(D, BITS, true).chunks, D, QM, kPackedQjlWaves>(a);
}

template <int VAR, int BITS, int C>
const void *packed_pick_mode(int mode, int cache_lp)
{
    switch (mode) {
    case MODE_ROUNDTRIP: return reinterpret_cast<const void *>(&packed_kernel<VAR, BITS, MODE_ROUNDTRIP, C>);
    case MODE_QUANTIZE: return reinterpret_cast<const void *>(&packed_kernel<VAR, BITS, MODE_QUANTIZE, C>);
    case MODE_DEQUANTIZE: return reinterpret_cast<const void *>(&packed_kernel<VAR, BITS, MODE_DEQUANTIZE, C>);
    case MODE_APPEND:
        return cache_lp == 4   ? reinterpret_cast<const void *>(&packed_append_kernel<VAR, BITS, C, 4>)
               : cache_lp == 3 ? reinterpret_cast<const void *>(&packed_append_kernel<VAR, BITS, C, 3>)
                               : reinterpret_cast<const void *>(&packed_append_kernel<VAR, BITS, C, -1>);
    }
    return nullptr;
}

// fp16 rows only: fp32 rows keep the generic kernels, whose slot-strided
// lanes make every 16-byte access instruction cover one contiguous span
// (measured at d = 96: 0.71 of the HBM roofline for the round trip, against
// 0.60-0.64 with a lane's 32 contiguous bytes)
template <int VAR>
const void *packed_pick(int bits, int mode, int chunks, int cache_lp)
{
    switch (bits * 4 + chunks) {
    case 2 * 4 + 1: return packed_pick_mode<VAR, 2, 1>(mode, cache_lp);
    case 2 * 4 + 2: return packed_pick_mode<VAR, 2, 2>(mode, cache_lp);
    case 3 * 4 + 1: return packed_pick_mode<VAR, 3, 1>(mode, cache_lp);
    case 3 * 4 + 2: return packed_pick_mode<VAR, 3, 2>(mode, cache_lp);
    case 4 * 4 + 1: return packed_pick_mode<VAR, 4, 1>(mode, cache_lp);
    case 4 * 4 + 2: return packed_pick_mode<VAR, 4, 2>(mode, cache_lp);
    }
    return nullptr;
}

}  // namespace
}  // namespace isoq
