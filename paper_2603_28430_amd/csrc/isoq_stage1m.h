// The stage-1 encoder with its forward block rotation on the matrix cores, for
// fp16 rows at d = 64, 128 and 256: round trip (forward half), quantize,
// append into a paged cache, and both with the stage-2 sketch.
//
// Why.  The encoder is bound by VALU issue, not by HBM: a lane's 8
// coordinates cost 32 fp32 multiply-adds for the forward rotation out of
// about 120 VALU instructions per row group.  v_mfma_f32_4x4x4_16b_f16 runs 16
// independent 4x4x4 products per instruction, which is exactly a block
// rotation (Sec. 5.2-5.4: one 4x4 matrix per block, the same for all rows
// of a set): block b of the instruction takes A = the block's matrix, B = four
// rows' 4 coordinates of that block, and returns the four rows' rotated
// coordinates.  The input rows are fp16 and exact in the product; the matrix
// is split into fp16 hi + lo parts (M = hi + lo to about 2^-22 relative), so
// two products per block reproduce M v with fp32 accumulation to within about
// 5e-7 of |v| (fp32 multiply-adds: about 1e-7), well inside the 1e-6 band of
// the parity rule.  8-D blocks take four 4x4 sub-blocks per output half.
//
// Lane layout (the "quad" layout).  The product needs lanes 4b .. 4b + 3 to
// hold the same 8-coordinate chunk of four different rows, so lane l holds
// chunk c of row i = l mod 4 of a row quad, b = l / 4: within a load the 16
// lane quads cover 16 (quad, chunk) pairs; a row's chunks sit on the lanes
// i, i + 4, i + 8, ... (one load at d = 64 and 128; two loads, the two halves
// of the row, at d = 256).  A lane's output of the product is its own row's
// rotated chunk, so quantizing, packing and storing stay lane-local as in the
// VALU encoder (isoq_stage1.h), with two changes: the squared norm is reduced
// over lanes 4 apart (DPP row rotations by 8 and 4, then the permlane swaps),
// and for 3 bits the four lanes of consecutive chunks that merge their 24-bit
// pieces into three words are 4 apart (DPP row_shl:4 instead of a quad
// permutation).  Global memory is read and written in the row order
// (consecutive lanes, consecutive 16-byte pieces of a row) and ds_bpermute
// moves the chunks to the quad order and back; the append kernels, whose
// tokens lie a token stride apart, read in the quad order directly.
//
// Rows with one rotation set each in turn (rows_per_set = 1: row r uses set
// r mod n_sets, as in a [token][head] K/V layout with one set per head) run
// as n_sets interleaved streams (STREAMS): block (s, y) takes tile y of the
// rows s, s + n_sets, s + 2 n_sets, ..., which all use set s, so the lanes of
// an MFMA block still share one matrix.  The append kernels read their rows
// the same way (stream = head), so their records equal isoq_quantize's.
//
// The round trip keeps its inverse rotation in fp32 on the VALU (lane-local,
// the chunk's fp32 parameters), so isoq_roundtrip stays bit-identical to
// isoq_quantize followed by isoq_dequantize: all three see the same
// reduction, the same rotated values and the same quantizer.
#pragma once

#include "isoq_stage1.h"

namespace isoq {
namespace {

typedef _Float16 half4 __attribute__((ext_vector_type(4)));
typedef float f32x4m __attribute__((ext_vector_type(4)));

constexpr int DPP_ROW_SHL4 = 0x104;   // lane i reads lane i + 4 of its 16-lane row
constexpr int DPP_ROW_ROR4 = 0x124;   // lane i reads lane i - 4 (mod 16) of its row
constexpr int DPP_ROW_ROR8 = 0x128;   // lane i reads lane i + 8 (mod 16) of its row

// Sum over the N (8 or 16) lanes 4 apart that hold one row's chunks in the
// quad layout (lanes i, i + 4, ..., i + 4 (N - 1) of the wave, i < 4, or of
// its half for N = 8).  Rotating by 8 first pairs lanes symmetrically, so all
// N lanes add the same two partial sums in the same order and get the same
// bits; the permlane swaps then add whole 16-lane rows as row_sum does.
template <int N>
__device__ __forceinline__ float quad_row_sum(float v)
{
    static_assert(N == 8 || N == 16, "8 or 16 lanes");
    v += dpp_f<DPP_ROW_ROR8>(v);
    v += dpp_f<DPP_ROW_ROR4>(v);
    {
        const auto s = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
        v = __uint_as_float(s[0]) + __uint_as_float(s[1]);
    }
    if constexpr (N == 16) {
        const auto s = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
        v = __uint_as_float(s[0]) + __uint_as_float(s[1]);
    }
    return v;
}

template <int VAR, int D, int BITS, int MODE, int QM = 0, int WAVES = 4, bool STREAMS = false>
struct Stage1M {
    static constexpr int C = D / kCoordsPerLane;       // chunks per row
    static constexpr int SPQ = C > 16 ? C / 16 : 1;    // loads holding one row quad
    static constexpr int QPS = C < 16 ? 16 / C : 1;    // row quads per load
    static constexpr int NRL = C < 16 ? C : 16;        // lanes of one row in one load
    static constexpr int RT = kTileGroups * 64 / C;    // rows per wave tile
    static constexpr int H = 1 << (BITS - 1);
    static constexpr int PL = kLanePL<VAR>;            // fp32 parameters per chunk (round trip inverse)
    static constexpr int PB = VAR == VAR_BLOCK8 ? 4 : 2;  // 16-byte matrix pieces per (chunk, quad row)
    static constexpr int64_t ROWB = (int64_t)D * 2;
    static constexpr int64_t RECB = (int64_t)D * BITS / 8;
    static constexpr bool kUseLut = BITS == 4;
    static constexpr bool kQjl = MODE == MODE_QJL || MODE == MODE_APPEND_QJL;
    static constexpr bool kAppend = MODE == MODE_APPEND || MODE == MODE_APPEND_QJL;
    static constexpr bool kRoundtrip = MODE == MODE_ROUNDTRIP;
    static constexpr bool kEncode = !kRoundtrip;
    static constexpr int kTileRows = RT;
    static constexpr int kEStride = D;   // unpadded, chunk positions swizzled (err_swizzle)
    static_assert(quad_layout(VAR, D, BITS), "quad layout variants and widths");
    static_assert(MODE != MODE_DEQUANTIZE, "the decoder keeps the VALU layout");
    static_assert(kTileGroups % SPQ == 0, "a row quad's loads fit in a tile");
    static_assert(!STREAMS || MODE == MODE_ROUNDTRIP || MODE == MODE_QUANTIZE, "streams: round trip and quantize");
    // block (x, y) = (stream or head, tile of its rows)
    static constexpr bool kByHead = kAppend || STREAMS;
    // global memory in the row order (below); the append kernels read their
    // tokens in the quad order, where four consecutive lanes read four
    // tokens' chunks of one head: measured faster there (their rows are
    // scattered over the token stride, so the row order gains no lines)
    static constexpr bool kPerm = !kAppend;
    static constexpr bool kEarly = !kQjl;

    // Geometry of load u for the lane of MFMA block b (= lane / 4) in wave w:
    // its chunk, its quad in the wave's tile and its quad in the block's tile
    // (block quad q holds block-tile rows 4 q .. 4 q + 3; the waves' loads u
    // together cover consecutive quads).
    __device__ static __forceinline__ int chunk_of(int u, int b) { return C <= 16 ? b % C : 16 * (u % SPQ) + b; }
    __device__ static __forceinline__ int wquad_of(int u, int b) { return C <= 16 ? QPS * u + b / C : u / SPQ; }
    __device__ static __forceinline__ int bquad_of(int u, int b, int w)
    {
        return C <= 16 ? (WAVES * u + w) * QPS + b / C : WAVES * (u / SPQ) + w;
    }
    // block quad of wave quad wq (the inverse of wquad_of, for the sketch)
    __device__ static __forceinline__ int bquad_of_wquad(int wq, int w)
    {
        return C <= 16 ? (WAVES * (wq / QPS) + w) * QPS + wq % QPS : WAVES * wq + w;
    }

    struct In {
        u32x4 raw;
        int64_t slot;   // append modes: the token's cache slot
    };

    // Lane orders of a load.  A load instruction of the wave covers the same
    // rows and chunks in two orders: in the row order lane l holds chunk
    // l mod NRL of the load's row l / NRL (consecutive lanes, consecutive
    // 16-byte pieces of a row: each quarter-wave covers whole 128-byte lines),
    // in the quad order lane 4 b + i holds chunk b mod C (d = 256: chunk b of
    // the half) of the load's row 4 (b / C) + i.  Global memory is read and
    // written in the row order (with the quad order, four consecutive lanes
    // touch four rows and the L1 cache counted four times the accesses);
    // ds_bpermute moves the chunks between the orders (the LDS crossbar, no
    // VALU).  The load's first row in the tile, and the lane maps:
    __device__ static __forceinline__ int load_row_base(int u, int w)
    {
        return C <= 16 ? 4 * QPS * (WAVES * u + w) : 4 * (WAVES * (u / SPQ) + w);
    }
    // the row-order lane holding quad-order lane (b, i)'s chunk
    __device__ static __forceinline__ int row_lane_of(int b, int i)
    {
        const int rin = (C <= 16 ? 4 * (b / C) : 0) + i, cin = C <= 16 ? b % C : b;
        return rin * NRL + cin;
    }
    // the quad-order lane holding row-order lane l's chunk
    __device__ static __forceinline__ int quad_lane_of(int l)
    {
        const int rin = l / NRL, cin = l % NRL;
        const int b = C <= 16 ? (rin / 4) * C + cin : cin;
        return 4 * b + rin % 4;
    }
    // chunk of row-order lane l in load u
    __device__ static __forceinline__ int row_chunk_of(int u, int l)
    {
        return C <= 16 ? l % NRL : 16 * (u % SPQ) + l % NRL;
    }

    __device__ static __forceinline__ u32x4 permute(const u32x4 &v, int addr)
    {
        u32x4 r;
#pragma unroll
        for (int k = 0; k < 4; k++)
            r[k] = (uint32_t)__builtin_amdgcn_ds_bpermute(addr, (int)v[k]);
        return r;
    }

    // Row addressing: row (or token, or stream row) row0 + roff of the
    // block's sequence, row0 wave-uniform and roff < the rows of a tile, so
    // addresses are a scalar base plus a 32-bit lane offset.  In memory the
    // row is row0 + roff, or (row0 + roff) n_sets + s for stream s, and a
    // token's row is (token n_heads + head).
    __device__ static __forceinline__ int64_t mem_row0(const KArgs &a, int64_t row0)
    {
        return STREAMS ? row0 * a.n_sets + blockIdx.x : row0;
    }
    __device__ static __forceinline__ uint32_t mem_roff(const KArgs &a, int roff)
    {
        return STREAMS ? (uint32_t)roff * (uint32_t)a.n_sets : (uint32_t)roff;
    }

    // chunk c of row (or token) row0 + roff, read in the row order
    __device__ static __forceinline__ u32x4 fetch(const KArgs &a, int64_t row0, int roff, int c)
    {
        if constexpr (kAppend) {
            // token row0 + roff, head blockIdx.x of rows [n_tokens][n_heads][d]
            const int64_t tstride = (int64_t)a.n_heads * ROWB;
            return __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(
                static_cast<const char *>(a.x) + row0 * tstride + (int64_t)blockIdx.x * ROWB +
                (uint32_t)((uint32_t)roff * (uint32_t)tstride + c * 16)));
        } else {
            return __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(
                static_cast<const char *>(a.x) + mem_row0(a, row0) * ROWB +
                (uint32_t)(mem_roff(a, roff) * (uint32_t)ROWB + c * 16)));
        }
    }

    // y = M v for the lane's chunk: four (8-D: eight) products of 16 blocks.
    // Am: the chunk's matrix rows for this lane's quad row, fp16 (hi, lo)
    // pieces.
    __device__ static __forceinline__ void rotate(const u32x4 *Am, const u32x4 &raw, float y[8])
    {
        half4 xb[2];
        xb[0] = __builtin_bit_cast(half4, u32x2{raw[0], raw[1]});
        xb[1] = __builtin_bit_cast(half4, u32x2{raw[2], raw[3]});
        f32x4m acc[2];
#pragma unroll
        for (int s = 0; s < 2; s++) {
            acc[s] = f32x4m{0.f, 0.f, 0.f, 0.f};
            if constexpr (VAR == VAR_BLOCK8) {
                // output half s: sub-blocks (s, 0) and (s, 1), each hi then lo
#pragma unroll
                for (int t = 0; t < 2; t++) {
                    const u32x4 q = Am[2 * s + t];
                    const half4 hi = __builtin_bit_cast(half4, u32x2{q[0], q[1]});
                    const half4 lo = __builtin_bit_cast(half4, u32x2{q[2], q[3]});
                    acc[s] = __builtin_amdgcn_mfma_f32_4x4x4f16(hi, xb[t], acc[s], 0, 0, 0);
                    acc[s] = __builtin_amdgcn_mfma_f32_4x4x4f16(lo, xb[t], acc[s], 0, 0, 0);
                }
            } else {
                const u32x4 q = Am[s];
                const half4 hi = __builtin_bit_cast(half4, u32x2{q[0], q[1]});
                const half4 lo = __builtin_bit_cast(half4, u32x2{q[2], q[3]});
                acc[s] = __builtin_amdgcn_mfma_f32_4x4x4f16(hi, xb[s], acc[s], 0, 0, 0);
                acc[s] = __builtin_amdgcn_mfma_f32_4x4x4f16(lo, xb[s], acc[s], 0, 0, 0);
            }
        }
#pragma unroll
        for (int k = 0; k < 4; k++) {
            y[k] = acc[0][k];
            y[4 + k] = acc[1][k];
        }
    }

    // Record bits of chunk c (coordinates 8 c .. 8 c + 7, bits [8 c b, 8 (c + 1) b)):
    // a half-word (2 bits), a word (4 bits), or for 3 bits 24 bits that the
    // lanes of chunks 4 k .. 4 k + 3 (4 lanes apart) merge into three words.
    template <class Dst>
    __device__ static __forceinline__ void store_bits(const Dst &rec, int c, uint32_t p, bool ok)
    {
        if constexpr (BITS == 2) {
            if (ok)
                rec.template put<uint16_t>(2 * c, (uint16_t)p);
        } else if constexpr (BITS == 4) {
            if (ok)
                rec.template put<uint32_t>(4 * c, p);
        } else {
            const uint32_t nb = dpp_u<DPP_ROW_SHL4>(p);   // the next chunk's bits
            const int k = c & 3;
            if (ok && k < 3)
                rec.template put<uint32_t>(4 * (3 * (c >> 2) + k), (p >> (8 * k)) | (nb << (24 - 8 * k)));
        }
    }

    // LDS for the block's rotation set, staged once per block: the matrix
    // pieces piece-major ([piece][chunk][quad row], 16 bytes each, so a
    // wave's reads of one piece cover consecutive 16-byte words), and for the
    // round trip the fp32 parameters chunk-minor ([16-byte piece][chunk], the
    // four lanes of a chunk reading one word).
    // the round trip stages its set in LDS (its fp32 inverse parameters are
    // read there); the encoders load their matrix rows straight from global
    // memory (no barrier before a short block's loads)
    static constexpr bool kStage = kRoundtrip;
    static constexpr int kLdsA = kStage ? PB * C * 4 : 0;                 // 16-byte words
    static constexpr int kLdsP = kStage && kRoundtrip ? PL / 4 * C : 0;  // 16-byte words
    static constexpr int kLdsWords = kLdsA + kLdsP > 0 ? kLdsA + kLdsP : 1;

    __device__ static void run(const KArgs &a, LutEntry *lds_lut, u32x4 *lds_par, _Float16 *lds_frag = nullptr,
                               _Float16 *lds_e = nullptr, int64_t *lds_crow = nullptr)
    {
        constexpr int BT = WAVES * 64;
        const int lane = threadIdx.x & 63;
        const int b = lane >> 2, qi = lane & 3;
        const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
        const int64_t tile0 = kByHead ? blockIdx.y : blockIdx.x;
        const int64_t rows_per_tile = (int64_t)WAVES * RT;
        // rows of the block's sequence: all rows, the tokens (append), or the
        // rows of stream blockIdx.x
        const int64_t nrows = STREAMS ? (a.n - blockIdx.x + a.n_sets - 1) / a.n_sets : a.n;

        // 1. block-wide tables: the 4-bit lookup table and the sketch's
        //    projection of the block's set, staged through LDS
        if constexpr (kUseLut) {
            const u32x4 *s4 = reinterpret_cast<const u32x4 *>(a.lut);
            u32x4 *d4 = reinterpret_cast<u32x4 *>(lds_lut);
            for (int i = threadIdx.x; i < a.lut_cells; i += BT)
                d4[i] = s4[i];
        }
        // the block's rotation set (every block's rows share one: the host
        // launches these kernels only then); append: every set is a head
        const int64_t set = a.n_sets <= 1 ? 0
                            : kByHead   ? (int64_t)blockIdx.x
                                        : (tile0 * rows_per_tile / a.rows_per_set) % a.n_sets;
        if constexpr (kQjl) {
            const u32x4 *f4 = reinterpret_cast<const u32x4 *>(a.qjl_frag + set * (int64_t)(QM * D));
            u32x4 *g4 = reinterpret_cast<u32x4 *>(lds_frag);
            for (int i = threadIdx.x; i < QM * D / 8; i += BT)
                g4[i] = f4[i];
        }
        if constexpr (kStage) {
            // the set's matrix pieces ([chunk][quad row][piece] in memory)
            // and fp32 parameters ([chunk][PL floats]), transposed on the way
            const u32x4 *am = reinterpret_cast<const u32x4 *>(a.mfma) + set * (int64_t)(C * 4 * PB);
            for (int j = threadIdx.x; j < kLdsA; j += BT) {
                const int k = j / (C * 4), cq = j - k * (C * 4);
                lds_par[j] = am[cq * PB + k];
            }
            if constexpr (kRoundtrip) {
                const u32x4 *pp = reinterpret_cast<const u32x4 *>(a.params + set * (int64_t)(C * PL));
                for (int j = threadIdx.x; j < kLdsP; j += BT) {
                    const int k = j / C, c = j - k * C;
                    lds_par[kLdsA + j] = pp[c * (PL / 4) + k];
                }
            }
        }
        if constexpr (kStage || kUseLut || kQjl)
            __syncthreads();

        // 2. the lane's matrix rows (quad row qi) of its SPQ chunks (the
        //    round trip reads its fp32 inverse parameters from LDS where it
        //    uses them, which keeps them out of the registers)
        u32x4 Am[SPQ][PB];
#pragma unroll
        for (int h = 0; h < SPQ; h++) {
            const int c = chunk_of(h, b);
            if constexpr (kStage) {
#pragma unroll
                for (int k = 0; k < PB; k++)
                    Am[h][k] = lds_par[(k * C + c) * 4 + qi];
            } else {
                const u32x4 *src = reinterpret_cast<const u32x4 *>(a.mfma) + (set * C + c) * (4 * PB) + qi * PB;
#pragma unroll
                for (int k = 0; k < PB; k++)
                    Am[h][k] = src[k];
            }
        }
        float lev[H], thr[H > 1 ? H - 1 : 1];
#pragma unroll
        for (int k = 0; k < H; k++)
            lev[k] = a.lev_pos[k];
#pragma unroll
        for (int k = 0; k < H - 1; k++)
            thr[k] = a.thr_pos[k];

        // 3. tiles: one per block, or with the sketch a stride of them (the
        //    staged projection then serves several).  A wave whose first row
        //    is past the end has nothing left.
        _Float16 *eq = kQjl ? lds_e + w * RT * kEStride : nullptr;
        // append with the sketch: the cache row of each tile row (-1: a
        // skipped slot), written by the encoder and read by the sketch
        int64_t *crq = kQjl && kAppend ? lds_crow + w * RT : nullptr;
        const int64_t tstride = kQjl ? (int64_t)(kAppend ? gridDim.y : gridDim.x) : (int64_t)1 << 40;
        const int64_t first_quad = C <= 16 ? (int64_t)w * QPS : w;   // bquad_of(0, 0, w)
        In buf[kTileGroups];
        int roffs[kTileGroups];   // the lane's row in the tile, per load (quad order)
        for (int64_t tb = tile0;; tb += tstride) {
            const int64_t row0 = tb * rows_per_tile;
            if (row0 + 4 * first_quad >= nrows)
                return;
            if (row0 + rows_per_tile <= nrows) {
                load<false>(a, row0, nrows, b, qi, w, buf, roffs);
                process<false>(a, Am, lds_par, lev, thr, lds_lut, row0, nrows, b, qi, w, eq, crq, buf, roffs);
            } else {
                load<true>(a, row0, nrows, b, qi, w, buf, roffs);
                process<true>(a, Am, lds_par, lev, thr, lds_lut, row0, nrows, b, qi, w, eq, crq, buf, roffs);
            }
            if constexpr (kQjl)
                sketch(a, lds_frag, eq, crq, row0, w);
            else
                return;
        }
    }

    // A tile: the wave's kTileGroups loads first (rows past the end re-read
    // the last row, compute it again and store the same bits), then compute
    // and store row quad by row quad (SPQ loads each).
    template <bool TAIL>
    __device__ static __forceinline__ void load(const KArgs &a, int64_t row0, int64_t nrows, int b, int qi, int w,
                                                In *buf, int *roffs)
    {
        const int lane = threadIdx.x & 63;
#pragma unroll
        for (int u = 0; u < kTileGroups; u++) {
            int r = 4 * bquad_of(u, b, w) + qi;
            int rl = load_row_base(u, w) + lane / NRL;   // the same in the row order
            if (TAIL) {
                r = (int)min((int64_t)r, nrows - 1 - row0);
                rl = (int)min((int64_t)rl, nrows - 1 - row0);
            }
            roffs[u] = r;
            if constexpr (kPerm)
                buf[u].raw = fetch(a, row0, rl, row_chunk_of(u, lane));
            else
                buf[u].raw = fetch(a, row0, r, chunk_of(u, b));
            if constexpr (kAppend)
                buf[u].slot = (a.slots + row0)[r];
        }
    }

    template <bool TAIL>
    __device__ static __forceinline__ void process(const KArgs &a, const u32x4 (*Am)[PB], const u32x4 *lds_par,
                                                   const float *lev, const float *thr, const LutEntry *lut,
                                                   int64_t row0, int64_t nrows, int b, int qi, int w, _Float16 *eq,
                                                   int64_t *crq, In *buf, const int *roffs)
    {
        const int lane = threadIdx.x & 63;
        __builtin_amdgcn_sched_barrier(0);
        // the loaded chunks in the quad order
        if constexpr (kPerm) {
            const int to_quad = 4 * row_lane_of(b, qi);
#pragma unroll
            for (int u = 0; u < kTileGroups; u++)
                buf[u].raw = permute(buf[u].raw, to_quad);
        }
        // every load's matrix products and squared-norm part first (the
        // products' latency then overlaps the rest of the tile's work)
        float yy[kEarly ? kTileGroups : 1][8], sq[kTileGroups];
#pragma unroll
        for (int u = 0; u < kTileGroups; u++) {
            float x8[8];
            Raw<true> r;
            r.w[0] = buf[u].raw;
            sq[u] = sum_squares<true>(r, x8);
            if constexpr (kEarly)
                rotate(Am[u % SPQ], buf[u].raw, yy[u]);
        }
#pragma unroll
        for (int k = 0; k < kTileGroups / SPQ; k++) {
            const int u0 = k * SPQ;
            // squared norm: the row's chunks in this quad's loads
            float part[SPQ];
#pragma unroll
            for (int h = 0; h < SPQ; h++)
                part[h] = quad_row_sum<NRL>(sq[u0 + h]);
            float ss = part[0];
            if constexpr (SPQ == 2)
                ss = part[0] + part[1];
            const float rho = __builtin_amdgcn_sqrtf(ss);
            const float rho_e = fmaxf(rho, kEps);
            float e2[SPQ];
            int64_t crow = -1;   // append: the row's cache row (-1: skipped slot)
#pragma unroll
            for (int h = 0; h < SPQ; h++) {
                // the row order's row and chunk of this load (round trip store)
                int rl = load_row_base(u0 + h, w) + lane / NRL;
                if (TAIL)
                    rl = (int)min((int64_t)rl, nrows - 1 - row0);
                float ylate[kEarly ? 1 : 8];
                if constexpr (!kEarly)
                    rotate(Am[h], buf[u0 + h].raw, ylate);
                e2[h] = compute(a, lds_par, lev, thr, lut, buf[u0 + h], row0, roffs[u0 + h],
                                chunk_of(u0 + h, b), rho, rho_e, eq, 4 * wquad_of(u0 + h, b) + qi,
                                kEarly ? yy[u0 + h] : ylate, rl, row_chunk_of(u0 + h, lane), crq, crow);
            }
            if constexpr (kQjl) {
                // gamma = rho ||e|| over the row's chunks (T is orthogonal:
                // ||x - x_hat|| in the input space)
                float s2 = quad_row_sum<NRL>(e2[0]);
                if constexpr (SPQ == 2)
                    s2 = s2 + quad_row_sum<NRL>(e2[1]);
                const float gamma = rho * __builtin_amdgcn_sqrtf(s2);
                if (chunk_of(u0, b) == 0)   // the lane of the row's chunk 0
                    emit_gamma(a, row0 + roffs[u0], crow, gamma);
            }
        }
    }

    __device__ static __forceinline__ void emit_gamma(const KArgs &a, int64_t row, int64_t crow, float gamma)
    {
        if constexpr (kAppend) {
            if (crow >= 0)
                a.qjl_gamma[crow] = gamma;
        } else {
            a.qjl_gamma[row] = gamma;
        }
    }

    // One chunk (its rotated values y_in): quantize, write the record bits and rho (encoders) or
    // the reconstruction (round trip); with the sketch the error e goes to
    // the wave's LDS tile (row erow) and its squared norm is returned.
    __device__ static __forceinline__ float compute(const KArgs &a, const u32x4 *lds_par,
                                                    const float *lev, const float *thr, const LutEntry *lut,
                                                    const In &in, int64_t row0, int roff, int c, float rho,
                                                    float rho_e, _Float16 *eq, int erow, const float *y_in,
                                                    int rl_roff, int rl_chunk, int64_t *crq, int64_t &crow)
    {
        float y[8], m[8], yq[8];
#pragma unroll
        for (int j = 0; j < 8; j++)
            y[j] = y_in[j];
#pragma unroll
        for (int j = 0; j < 8; j++)
            m[j] = fabsf(y[j]);
        // with the sketch the levels are the normalised ones, and zero for a
        // zero row (whose y is exactly zero), so that e below is zero there
        const float lscale = kQjl ? (rho > 0.f ? 1.f : 0.f) : rho;
        uint32_t p = 0;
        if constexpr (kUseLut) {
            const float s = a.lut_inv_h * __builtin_amdgcn_rcpf(rho_e);
            p = lut_quantize<BITS, kRoundtrip || kQjl, kEncode>(y, m, s, (float)(a.lut_cells - 1), lut, lscale, yq);
        } else {
            float ths[H > 1 ? H - 1 : 1];
#pragma unroll
            for (int k = 0; k < H - 1; k++)
                ths[k] = thr[k] * rho_e;
            if constexpr (kRoundtrip) {
                float lvs[H];
#pragma unroll
                for (int k = 0; k < H; k++)
                    lvs[k] = lev[k] * lscale;
                chain_levels<H>(y, m, ths, lvs, yq);
            } else if constexpr (kQjl) {
                float lvs[H];
#pragma unroll
                for (int k = 0; k < H; k++)
                    lvs[k] = lev[k] * lscale;
                p = ballot_encode<BITS, kQjl>(y, m, ths, lvs, yq);
            } else {
                p = ballot_encode<BITS, kQjl>(y, m, ths, lev, yq);
            }
        }
        if constexpr (kEncode) {
            // the row's record and norm: its row, or the token's cache row
            if constexpr (kAppend) {
                bool ok;
                int pos;
                const int64_t orow = cache_slot(a, in.slot, blockIdx.x, ok, pos);
                store_bits(cache_rec<RECB>(a, orow, pos), c, p, ok);
                if (ok && c == 0)
                    a.norms_out[orow] = rho;
                crow = ok ? orow : -1;
                if constexpr (kQjl) {
                    if (c == 0)
                        crq[erow] = crow;
                }
            } else {
                const uint32_t mr = mem_roff(a, roff);
                store_bits(RecPtr{a.rec_out + mem_row0(a, row0) * RECB + (uint32_t)(mr * (uint32_t)RECB)}, c, p, true);
                if (c == 0)
                    (a.norms_out + mem_row0(a, row0))[mr] = rho;
            }
        }
        if constexpr (kRoundtrip) {
            // the chunk's fp32 parameters from LDS ([16-byte piece][chunk])
            float P[PL];
#pragma unroll
            for (int k = 0; k < PL / 4; k++) {
                const u32x4 v = lds_par[kLdsA + k * C + c];
                const uint32_t e0 = v[0], e1 = v[1], e2 = v[2], e3 = v[3];
                P[4 * k] = __uint_as_float(e0);
                P[4 * k + 1] = __uint_as_float(e1);
                P[4 * k + 2] = __uint_as_float(e2);
                P[4 * k + 3] = __uint_as_float(e3);
            }
            float o[8];
            rotate_inverse<VAR>(P, yq, o);
            // fp16, round to nearest even (one explicit conversion, as
            // store_row_chunk does), then to the row order and out
            u32x4 hv;
#pragma unroll
            for (int k = 0; k < 4; k++) {
                uint32_t h;
                asm("v_cvt_pk_f16_f32 %0, %1, %2" : "=v"(h) : "v"(o[2 * k]), "v"(o[2 * k + 1]));
                hv[k] = h;
            }
            const int lane = threadIdx.x & 63;
            hv = permute(hv, 4 * quad_lane_of(lane));
            __builtin_nontemporal_store(hv, reinterpret_cast<u32x4 *>(
                                                static_cast<char *>(a.y) + mem_row0(a, row0) * ROWB +
                                                (uint32_t)(mem_roff(a, rl_roff) * (uint32_t)ROWB + rl_chunk * 16)));
        }
        float s2 = 0.f;
        if constexpr (kQjl) {
            // e = y / rho' - c[idx], the normalised rotated-domain error (zero
            // for a zero row), to the wave's LDS tile as fp16
            const float inv = __builtin_amdgcn_rcpf(rho_e);
            float e[8];
#pragma unroll
            for (int j = 0; j < 8; j++) {
                e[j] = fmaf(y[j], inv, -yq[j]);
                s2 = fmaf(e[j], e[j], s2);
            }
            u32x4 hv;
#pragma unroll
            for (int k = 0; k < 4; k++) {
                uint32_t v;
                asm("v_cvt_pk_f16_f32 %0, %1, %2" : "=v"(v) : "v"(e[2 * k]), "v"(e[2 * k + 1]));
                hv[k] = v;
            }
            *reinterpret_cast<u32x4 *>(eq + erow * kEStride + 8 * (c ^ err_swizzle(erow))) = hv;
        }
        return s2;
    }

    // Stage-2 sketch of the wave's tile: tile row 4 wq + i is row i of the
    // wave's quad wq.
    __device__ static __forceinline__ void sketch(const KArgs &a, const _Float16 *frag, const _Float16 *eq,
                                                  const int64_t *crq, int64_t row0, int w)
    {
        qjl_project<D, QM, kTileRows, kEStride, true>(frag, eq, [&](int ar) -> uint32_t * {
            const int64_t row = row0 + 4 * bquad_of_wquad(ar >> 2, w) + (ar & 3);
            if (ar >= kTileRows || row >= a.n)
                return nullptr;
            int64_t orow = row;
            if constexpr (kAppend) {
                orow = crq[ar];   // the encoder's cache row of tile row ar
                if (orow < 0)
                    return nullptr;
            }
            return reinterpret_cast<uint32_t *>(a.qjl_signs + orow * (QM / 8));
        });
    }
};

}  // namespace
}  // namespace isoq
