// Attention logits against a paged cache of quantized keys, for decoding.
//
// A key stored by isoq_kv_append is x_hat = rho T^{-1}(c[idx]) with T the
// block rotation of its head.  T is orthogonal (Prop. 1), so for a query q
//     <q, x_hat> = rho <T q, c[idx]>:
// the query is rotated once and the keys are never inverse-rotated or
// dequantized.  With the query fixed, <T q, c[idx]> is a sum of table lookups
// (asymmetric distance computation): the record is cut into fields of F
// coordinates (F b bits: pairs for 2 and 3 bits, single coordinates for 4
// bits, so a table has at most 64 entries) and field j of value e contributes
// table[j][e] = sum_f (T q)_{F j + f} c[e_f].
//
// Workgroup (key head h, chunk of kScoreChunk positions, sequence s):
//   0. load the block-table entries of the lane's keys and the first batch
//      of records;
//   1. rotate the group's query heads (scale folded in) into LDS;
//   2. build the group's tables in LDS (d/F tables of 2^(F b) floats each);
//   3. one key per lane: its record (one load per piece of the cache
//      layout, up to 16 bytes) and norm, the d/F
//      lookups summed, rho * sum written.  All lanes read the same field's
//      table at the same time; a 64-entry table on 32 four-byte banks makes
//      entries e and e + 32 share a bank, which measured as no cost: the
//      record loads set the speed.
// With the stage-2 sketch (QM > 0 sign bits per key, Sec. 8) each logit also
// gets the residual correction sqrt(pi/2)/m gamma <S q, 2 z - 1>: S q is
// computed once per workgroup and cut into groups of 4 signs, each with a
// 16-entry table sum_b (+-1) (S q)_{4 i + b}, summed like the stage-1 fields.
// The roofline is HBM bandwidth on the records (d b / 8 + 4 bytes per key,
// plus m / 8 + 4 with the sketch, and the 4-byte logit); no MFMA: there is no
// dense contraction left once q is rotated.
#pragma once

#include <hip/hip_runtime.h>

#include "isoq_device.h"
#include "isoq_internal.h"

namespace isoq {
namespace {

template <int D, int BITS, int QM = 0>
struct ScoreShape {
    static constexpr int K = 1 << BITS;
    static constexpr int F = BITS == 4 ? 1 : 2;   // coordinates per lookup field
    static constexpr int FB = F * BITS;           // bits per field
    static constexpr int E = 1 << FB;             // entries per table
    static constexpr int NF = D / F;              // fields (tables) per key
    static constexpr int RW = (D * BITS + 31) / 32;  // record words (the last one partial at 3 bits, d = 80)
    static constexpr int RH = D * BITS / 16;         // record half-words
    static_assert(RH * 16 == D * BITS, "records are a whole number of half-words");
    // words per record load: 16, 8 or 4 bytes, the largest that divides the
    // record (a record of d b / 8 bytes starts on such a boundary); 0: a
    // record of an odd number of half-words, read in 2-byte loads
    static constexpr int LW = RW * 32 != D * BITS ? 0 : RW % 4 == 0 ? 4 : RW % 2 == 0 ? 2 : 1;
    static constexpr int RV = LW ? RW / LW : RH;   // loads per record
    // bytes per load, and the piece size of the cache layout (cache_piece):
    // one load per piece (16 or 8 bytes), or several per record stored whole
    static constexpr int PB = LW ? 4 * LW : 2;
    static constexpr int CP = cache_piece(D * BITS / 8);
    static_assert(CP % PB == 0, "loads tile the pieces of the cache layout");
    // keys per lane and batch
    static constexpr int KPT = RW <= 12 ? 2 : 1;
    static constexpr int SW = QM / 32;             // sketch words per key
    static constexpr int NQ = QM / 4;              // 4-sign groups (16-entry tables) per key
    // LDS floats for g query heads: tables, codebook, rotated queries; with
    // the sketch also the sign tables, S q and the raw queries
    static constexpr int lds_floats(int g) { return g * NF * E + 16 + g * D + (QM ? g * (16 * NQ + QM + D) : 0); }
};

// A compile-time group size whose LDS fits 64 KB uses a static array (its
// address is a constant the reads take as immediate offsets); otherwise the
// group size comes at run time with dynamic LDS.
template <int D, int BITS, int GT, int QM>
constexpr bool kStaticLds = GT > 0 && ScoreShape<D, BITS, QM>::lds_floats(GT) * 4 <= 65536;

// Sum of the table entries selected by the fields of one record.  `base` is
// the LDS byte address of the query head's first table, a multiple of the
// head's table block, so the byte address of entry e of table j is
// (4 e | base) + 4 E j: one shift and one and-or per field, the table offset
// an immediate of the read.  The reads go out in groups of 16 with two
// partial sums: group i adds into sum i mod 2, and that sum is forced to be
// complete before group i + 2 is issued, so at most 32 reads are in flight
// (left alone, the compiler issues all d/F reads before the first add and
// holds every result in a register).
// NF fields of FB bits each, tables of 2^FB entries.
template <int NF, int FB>
__device__ __forceinline__ float lookup_sum(const char *lds, uint32_t base, const uint32_t *w)
{
    constexpr int E = 1 << FB;
    constexpr uint32_t kMask = (uint32_t)(E - 1) << 2;
    float acc[2] = {0.f, 0.f};
#pragma unroll
    for (int j = 0; j < NF; j++) {
        const int o = j * FB;
        const int k = o >> 5, sh = o & 31;
        uint32_t x;
        if (sh + FB > 32)
            x = __builtin_amdgcn_alignbit(w[k + 1], w[k], sh - 2);  // straddles two words (sh >= 26)
        else if (sh >= 2)
            x = w[k] >> (sh - 2);
        else
            x = w[k] << (2 - sh);
        const uint32_t addr = (x & kMask) | base;
        acc[(j >> 4) & 1] += *reinterpret_cast<const float *>(lds + addr + 4 * E * j);
        if ((j & 15) == 15) {
            __builtin_amdgcn_sched_barrier(0);
            if (j >= 31)
                asm volatile("" : "+v"(acc[((j >> 4) + 1) & 1]));
        }
    }
    return acc[0] + acc[1];
}

// GT: query heads per key head as a compile-time constant (the table base of
// every head then folds into the reads' immediate offsets), or 0 for any
// group size given at run time.
template <int VAR, int D, int BITS, bool F16, int GT, int QM>
__global__ __launch_bounds__(256) void score_kernel(const SArgs a)
{
    using S = ScoreShape<D, BITS, QM>;
    constexpr int LPQ = D / kCoordsPerLane;          // 8-coordinate chunks per query
    constexpr int PL = kLanePL<VAR>;
    constexpr int64_t RB = (int64_t)D * BITS / 8;    // record bytes
    // LDS: tables[G][NF][E] | levels[16] | q~[G][D] | (sketch) sign tables
    // [G][NQ][16] | S q [G][QM] | q [G][D]
    float *smem;
    if constexpr (kStaticLds<D, BITS, GT, QM>) {
        __shared__ __align__(16) float sm[S::lds_floats(GT)];
        smem = sm;
    } else {
        extern __shared__ __align__(16) float dyn[];
        smem = dyn;
    }
    // a head's records of one cache block: block_size records of RB bytes
    const int h = (int)xcd_head(blockIdx.x, (uint32_t)a.n_kv_heads, a.block_size * RB % 128 != 0);
    const int s = blockIdx.z;
    const int G = GT > 0 ? GT : a.group;
    int64_t len = a.seq_lens[s];
    len = min(len, a.max_len);
    len = min(len, (int64_t)a.max_blocks * a.block_size);
    const int64_t t0 = (int64_t)blockIdx.y * kScoreChunk;
    if (t0 >= len)
        return;  // block-uniform: the whole workgroup leaves before any barrier
    float *tab = smem;
    float *lev = tab + G * S::NF * S::E;
    float *qt = lev + 16;
    float *tab2 = qt + G * D;
    float *sqv = tab2 + G * 16 * S::NQ;
    float *qraw = sqv + G * QM;
    const int set = a.n_sets == 1 ? 0 : h;

    // 0. keys t0 + threadIdx.x + 256 i, in batches of KPT keys per lane.  A
    //    record's address depends on its block-table entry, so the entries
    //    of all of the lane's keys are loaded first; the first batch's
    //    records are then in flight while the tables are built, and each
    //    later batch is loaded while the previous one is summed.  The cache
    //    stores records piece-major, so one load instruction (piece v of
    //    the wave's 64 keys) reads consecutive bytes of each cache block;
    //    with records stored whole, the lanes of an instruction were a
    //    record apart and every instruction touched every line of the span.
    //    Pieces of 8 and 16 bytes are read non-temporally; records stored
    //    whole (sizes not a multiple of 8) with ordinary 2- or 4-byte loads,
    //    whose lanes are a record apart (the second and later loads of a
    //    line then hit L1).
    const int64_t tend = min(t0 + (int64_t)kScoreChunk, len);
    const int32_t *table = a.block_table + (int64_t)s * a.max_blocks;
    constexpr int NB = kScoreChunk / 256 / S::KPT;
    static_assert(NB * S::KPT * 256 == kScoreChunk, "batches tile the chunk");
    int32_t bt[NB][S::KPT];
#pragma unroll
    for (int b = 0; b < NB; b++)
#pragma unroll
        for (int u = 0; u < S::KPT; u++) {
            const int64_t t = t0 + threadIdx.x + 256 * (b * S::KPT + u);
            const uint32_t tt = (uint32_t)min(t, len - 1);
            bt[b][u] = table[fast_div(tt, a.div_block)];
        }
    struct Batch {
        uint32_t w[S::KPT][S::RW];
        uint32_t z[S::KPT][S::SW > 0 ? S::SW : 1];   // sign sketch
        float gam[S::KPT];
        float rho[S::KPT];
        int64_t t[S::KPT];
        bool ok[S::KPT];
    };
    auto issue = [&](int b, Batch &k) {
#pragma unroll
        for (int u = 0; u < S::KPT; u++) {
            const int64_t t = t0 + threadIdx.x + 256 * (b * S::KPT + u);
            const uint32_t tt = (uint32_t)min(t, len - 1);
            const uint32_t bi = fast_div(tt, a.div_block);
            const int32_t blk = bt[b][u];
            k.ok[u] = t < tend && blk >= 0 && blk < a.n_blocks;
            // an invalid key reads record 0 of block 0 (always present) and is not stored
            const int pos = k.ok[u] ? (int)(tt - bi * a.block_size) : 0;
            const int64_t krow = k.ok[u] ? ((int64_t)blk * a.n_kv_heads + h) * a.block_size + pos : 0;
            // load v of the record: byte v PB, in piece v PB / CP of the
            // head's block region (piece-major: consecutive keys' pieces are
            // adjacent), at byte v PB mod CP of the piece
            const uint8_t *pc0 = a.k_idx + (krow - pos) * RB + (int64_t)pos * S::CP;
            const int64_t pstep = (int64_t)a.block_size * S::CP;
            auto at = [&](int v) { return pc0 + (v * S::PB / S::CP) * pstep + (v * S::PB % S::CP); };
            if constexpr (S::LW == 4) {
#pragma unroll
                for (int v = 0; v < S::RV; v++) {
                    const u32x4 q4 = __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(at(v)));
#pragma unroll
                    for (int c = 0; c < 4; c++) {
                        const uint32_t e = q4[c];
                        k.w[u][4 * v + c] = e;
                    }
                }
            } else if constexpr (S::LW == 0) {
                // records of an odd number of half-words: 2-byte loads, paired
                // into words (the upper half of the last word is zero)
#pragma unroll
                for (int c = 0; c < S::RW; c++) {
                    const uint32_t lo = *reinterpret_cast<const uint16_t *>(at(2 * c));
                    const uint32_t hi = 2 * c + 1 < S::RH ? (uint32_t)*reinterpret_cast<const uint16_t *>(at(2 * c + 1)) : 0u;
                    k.w[u][c] = lo | (hi << 16);
                }
            } else if constexpr (S::LW == 1) {
                // records of an odd number of words: 4-byte loads
#pragma unroll
                for (int v = 0; v < S::RV; v++)
                    k.w[u][v] = *reinterpret_cast<const uint32_t *>(at(v));
            } else {
                // records of 8 (mod 16) bytes: 8-byte loads
#pragma unroll
                for (int v = 0; v < S::RV; v++) {
                    const u32x2 q2 = __builtin_nontemporal_load(reinterpret_cast<const u32x2 *>(at(v)));
                    const uint32_t e0 = q2[0], e1 = q2[1];
                    k.w[u][2 * v] = e0;
                    k.w[u][2 * v + 1] = e1;
                }
            }
            k.rho[u] = a.k_rho[krow];
            k.t[u] = t;
            if constexpr (QM > 0) {
                const uint32_t *zp = reinterpret_cast<const uint32_t *>(a.k_signs + krow * (QM / 8));
#pragma unroll
                for (int c = 0; c < S::SW; c++)
                    k.z[u][c] = zp[c];
                k.gam[u] = a.k_gamma[krow];
            }
        }
    };
    Batch kb[2];
    issue(0, kb[0]);

    // 1. rotated queries q~_g = scale * T_h q_g and the codebook
    if (threadIdx.x < S::K)
        lev[threadIdx.x] = a.lev_all[threadIdx.x];
    for (int i = threadIdx.x; i < G * LPQ; i += blockDim.x) {
        const int g = i / LPQ, l = i - g * LPQ;
        const char *qrow = static_cast<const char *>(a.q) +
                           ((int64_t)s * a.n_q_heads + (int64_t)h * G + g) * D * (F16 ? 2 : 4);
        Raw<F16> r;
        load_row_chunk<F16>(qrow + l * (F16 ? 16 : 32), r);
        float x[8], y[8], P[PL];
        unpack<F16>(r, x);
        load_params<PL>(a.params + ((int64_t)set * LPQ + l) * PL, P);
        rotate_forward<VAR>(P, x, y);
#pragma unroll
        for (int k = 0; k < 8; k++)
            qt[g * D + 8 * l + k] = y[k] * a.scale;
        if constexpr (QM > 0) {
#pragma unroll
            for (int k = 0; k < 8; k++)
                qraw[g * D + 8 * l + k] = x[k];
        }
    }
    __syncthreads();

    // 2. tables: tab[g][j][e] = sum_f q~_g[F j + f] * c[(e >> f b) mod K].
    //    A work item fills 16 consecutive entries of one table: with
    //    e = 16 m + k, the first coordinate's level index e mod K is k mod K
    //    (K <= 16 divides 16), a constant, and the second's, e >> b, takes at
    //    most two values per item.
    constexpr int EPT = S::E < 16 ? S::E : 16;
    for (int i = threadIdx.x; i < G * S::NF * (S::E / EPT); i += blockDim.x) {
        const int m = i % (S::E / EPT);
        const int gj = i / (S::E / EPT);  // g * NF + j
        const int g = gj / S::NF, j = gj - g * S::NF;
        const float *qg = qt + g * D + S::F * j;
        const float qa = qg[0];
        float out[EPT];
        if constexpr (S::F == 2) {
            const float qb = qg[1];
#pragma unroll
            for (int k = 0; k < EPT; k++)
                out[k] = fmaf(qb, lev[(EPT * m + k) >> BITS], qa * a.lev_all[k & (S::K - 1)]);
        } else {
#pragma unroll
            for (int k = 0; k < EPT; k++)
                out[k] = qa * a.lev_all[k];
        }
        float4 *dst = reinterpret_cast<float4 *>(tab + (int64_t)gj * S::E + EPT * m);
#pragma unroll
        for (int k = 0; k < EPT / 4; k++)
            dst[k] = make_float4(out[4 * k], out[4 * k + 1], out[4 * k + 2], out[4 * k + 3]);
    }
    if constexpr (QM > 0) {
        // (S q_g)_r for every query head of the group, S fp32 [QM][D]
        for (int i = threadIdx.x; i < G * QM; i += blockDim.x) {
            const int g = i / QM, r = i - g * QM;
            const float4 *srow = reinterpret_cast<const float4 *>(a.qjl_S + (int64_t)r * D);
            const float4 *qv = reinterpret_cast<const float4 *>(qraw + g * D);
            float acc = 0.f;
#pragma unroll 8
            for (int j = 0; j < D / 4; j++) {
                const float4 sv = srow[j], q4 = qv[j];
                acc = fmaf(sv.x, q4.x, acc);
                acc = fmaf(sv.y, q4.y, acc);
                acc = fmaf(sv.z, q4.z, acc);
                acc = fmaf(sv.w, q4.w, acc);
            }
            sqv[g * QM + r] = acc * a.qjl_scale;
        }
        __syncthreads();
        // sign tables: entry e of group i is sum_b (bit b of e ? 1 : -1) (S q)_{4 i + b}
        for (int i = threadIdx.x; i < G * S::NQ; i += blockDim.x) {
            const float *v = sqv + 4 * i;  // i = g * NQ + group
            const float v0 = v[0], v1 = v[1], v2 = v[2], v3 = v[3];
            float out[16];
#pragma unroll
            for (int e = 0; e < 16; e++)
                out[e] = ((e & 1) ? v0 : -v0) + ((e & 2) ? v1 : -v1) + ((e & 4) ? v2 : -v2) + ((e & 8) ? v3 : -v3);
            float4 *dst = reinterpret_cast<float4 *>(tab2 + 16 * i);
#pragma unroll
            for (int k = 0; k < 4; k++)
                dst[k] = make_float4(out[4 * k], out[4 * k + 1], out[4 * k + 2], out[4 * k + 3]);
        }
    }
    __syncthreads();

    auto consume = [&](Batch &k) {
#pragma unroll
        for (int u = 0; u < S::KPT; u++) {
            float *dst = a.scores + ((int64_t)s * a.n_q_heads + (int64_t)h * G) * a.max_len + k.t[u];
            // compile-time group sizes unroll fully; a run-time one loops
            constexpr int GU = GT > 0 ? GT : 1;
            for (int g0 = 0; g0 < G; g0 += GU)
#pragma unroll
            for (int gi = 0; gi < GU; gi++) {
                const int g = g0 + gi;
                // Empty asm statements keep the register footprint small: the
                // record words look modified per query head, so the field
                // offsets are not hoisted out of this loop (d/F registers),
                // and the sum is complete before the branch, so the lookups
                // are not sunk into it and held all at once.
#pragma unroll
                for (int c = 0; c < S::RW; c++)
                    asm volatile("" : "+v"(k.w[u][c]));
                const float acc = lookup_sum<S::NF, S::FB>(reinterpret_cast<const char *>(tab),
                                                           (uint32_t)(g * S::NF * S::E * 4), k.w[u]);
                float val = k.rho[u] * acc;
                if constexpr (QM > 0) {
#pragma unroll
                    for (int c = 0; c < S::SW; c++)
                        asm volatile("" : "+v"(k.z[u][c]));
                    const float acc2 = lookup_sum<S::NQ, 4>(reinterpret_cast<const char *>(tab2),
                                                             (uint32_t)(g * S::NQ * 16 * 4), k.z[u]);
                    val = fmaf(k.gam[u], acc2, val);
                }
                asm volatile("" ::"v"(val));
                if (k.ok[u])
                    dst[(int64_t)g * a.max_len] = val;
            }
        }
    };
    // 3. sums, batch by batch (the next batch's loads issued first)
#pragma unroll
    for (int b = 0; b < NB; b++) {
        if (t0 + 256 * b * S::KPT >= tend)  // block-uniform
            break;
        if (b + 1 < NB && t0 + 256 * (b + 1) * S::KPT < tend)
            issue(b + 1, kb[(b + 1) & 1]);
        consume(kb[b & 1]);
    }
}

}  // namespace
}  // namespace isoq
