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
//   1. rotate the group's query heads (scale folded in) into LDS;
//   2. build the group's tables in LDS (d/F tables of 2^(F b) floats each);
//   3. one key per lane: load its record (16-byte loads) and norm, sum the
//      d/F lookups, write rho * sum.  All lanes read the same field's table at
//      the same time, so lanes that read different entries never collide on
//      an LDS bank (a table has at most 64 entries).
// The path is bound by HBM bandwidth on the records (d b / 8 + 4 bytes per
// key); no MFMA: there is no dense contraction left once q is rotated.
#include <hip/hip_runtime.h>

#include "isoq_device.h"
#include "isoq_internal.h"

namespace isoq {
namespace {

template <int D, int BITS>
struct ScoreShape {
    static constexpr int K = 1 << BITS;
    static constexpr int F = BITS == 4 ? 1 : 2;   // coordinates per lookup field
    static constexpr int FB = F * BITS;           // bits per field
    static constexpr int E = 1 << FB;             // entries per table
    static constexpr int NF = D / F;              // fields (tables) per key
    static constexpr int RW = D * BITS / 32;      // record words
    static constexpr int RV = RW / 4;             // 16-byte loads per record
    // keys per lane and batch
    static constexpr int KPT = RW <= 12 ? 2 : 1;
    static_assert(RW % 4 == 0, "records are a whole number of 16-byte vectors");
    // LDS floats for g query heads: tables, codebook, rotated queries
    static constexpr int lds_floats(int g) { return g * NF * E + 16 + g * D; }
};

// A compile-time group size whose LDS fits 64 KB uses a static array (its
// address is a constant the reads take as immediate offsets); otherwise the
// group size comes at run time with dynamic LDS.
template <int D, int BITS, int GT>
constexpr bool kStaticLds = GT > 0 && ScoreShape<D, BITS>::lds_floats(GT) * 4 <= 65536;

// Sum of the table entries selected by the fields of one record.  `base` is
// the LDS byte address of the query head's first table, a multiple of the
// head's table block, so the byte address of entry e of table j is
// (4 e | base) + 4 E j: one shift and one and-or per field, the table offset
// an immediate of the read.
template <int D, int BITS>
__device__ __forceinline__ float lookup_sum(const char *lds, uint32_t base, const uint32_t *w)
{
    using S = ScoreShape<D, BITS>;
    constexpr uint32_t kMask = (uint32_t)(S::E - 1) << 2;
    float acc = 0.f;
#pragma unroll
    for (int j = 0; j < S::NF; j++) {
        const int o = j * S::FB;
        const int k = o >> 5, sh = o & 31;
        uint32_t x;
        if (sh + S::FB > 32)
            x = __builtin_amdgcn_alignbit(w[k + 1], w[k], sh - 2);  // straddles two words (sh >= 26)
        else if (sh >= 2)
            x = w[k] >> (sh - 2);
        else
            x = w[k] << (2 - sh);
        const uint32_t addr = (x & kMask) | base;
        acc += *reinterpret_cast<const float *>(lds + addr + 4 * S::E * j);
        // at most 16 lookups in flight: left alone, the scheduler issues all
        // d/F reads first and holds every result in a register
        if ((j & 15) == 15)
            __builtin_amdgcn_sched_barrier(0);
    }
    return acc;
}

// GT: query heads per key head as a compile-time constant (the table base of
// every head then folds into the reads' immediate offsets), or 0 for any
// group size given at run time.
template <int VAR, int D, int BITS, bool F16, int GT>
__global__ __launch_bounds__(256) void score_kernel(const SArgs a)
{
    using S = ScoreShape<D, BITS>;
    constexpr int LPQ = D / kCoordsPerLane;          // 8-coordinate chunks per query
    constexpr int PL = VAR == VAR_FULL ? 32 : 8;
    constexpr int64_t RB = (int64_t)D * BITS / 8;    // record bytes
    // LDS: tables[G][NF][E] | levels[16] | q~[G][D]
    float *smem;
    if constexpr (kStaticLds<D, BITS, GT>) {
        __shared__ __align__(16) float sm[S::lds_floats(GT)];
        smem = sm;
    } else {
        extern __shared__ __align__(16) float dyn[];
        smem = dyn;
    }
    const int h = blockIdx.x, s = blockIdx.z;
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
    const int set = a.n_sets == 1 ? 0 : h;

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
    __syncthreads();

    // 3. keys t0 + threadIdx.x + 256 i, in batches of KPT keys per lane: the
    //    batch's records are loaded together, then summed.  (Prefetching the
    //    next batch during the sums measured slower: the extra registers cost
    //    more occupancy than the overlap gained.)
    const int64_t tend = min(t0 + (int64_t)kScoreChunk, len);
    const int32_t *table = a.block_table + (int64_t)s * a.max_blocks;
    constexpr int NB = kScoreChunk / 256 / S::KPT;
    static_assert(NB * S::KPT * 256 == kScoreChunk, "batches tile the chunk");
    struct Batch {
        uint32_t w[S::KPT][S::RW];
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
            const int32_t blk = table[bi];
            k.ok[u] = t < tend && blk >= 0 && blk < a.n_blocks;
            // an invalid key reads record 0 of block 0 (always present) and is not stored
            const int64_t krow =
                k.ok[u] ? ((int64_t)blk * a.n_kv_heads + h) * a.block_size + (tt - bi * a.block_size) : 0;
            const u32x4 *rp = reinterpret_cast<const u32x4 *>(a.k_idx + krow * RB);
#pragma unroll
            for (int v = 0; v < S::RV; v++) {
                const u32x4 q4 = __builtin_nontemporal_load(rp + v);
#pragma unroll
                for (int c = 0; c < 4; c++) {
                    const uint32_t e = q4[c];
                    k.w[u][4 * v + c] = e;
                }
            }
            k.rho[u] = a.k_rho[krow];
            k.t[u] = t;
        }
    };
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
                const float acc = lookup_sum<D, BITS>(reinterpret_cast<const char *>(tab),
                                                      (uint32_t)(g * S::NF * S::E * 4), k.w[u]);
                const float val = k.rho[u] * acc;
                asm volatile("" ::"v"(val));
                if (k.ok[u])
                    dst[(int64_t)g * a.max_len] = val;
            }
        }
    };
#pragma unroll 1
    for (int b = 0; b < NB; b++) {
        if (t0 + 256 * b * S::KPT >= tend)  // block-uniform
            break;
        Batch k;
        issue(b, k);
        consume(k);
    }
}

template <int VAR, int D, int BITS, bool F16, int GT>
ScoreKernel entry(int group)
{
    using S = ScoreShape<D, BITS>;
    if constexpr (kStaticLds<D, BITS, GT>)
        return {reinterpret_cast<const void *>(&score_kernel<VAR, D, BITS, F16, GT>), 0};
    return {reinterpret_cast<const void *>(&score_kernel<VAR, D, BITS, F16, 0>),
            sizeof(float) * (size_t)S::lds_floats(group)};
}

template <int VAR, int D, int BITS, bool F16>
ScoreKernel pick_group(int group)
{
    switch (group) {
    case 1: return entry<VAR, D, BITS, F16, 1>(group);
    case 4: return entry<VAR, D, BITS, F16, 4>(group);
    }
    return entry<VAR, D, BITS, F16, 0>(group);
}

template <int VAR, int D, int BITS>
ScoreKernel pick_dtype(bool f16, int group)
{
    return f16 ? pick_group<VAR, D, BITS, true>(group) : pick_group<VAR, D, BITS, false>(group);
}

template <int VAR, int D>
ScoreKernel pick_bits(int bits, bool f16, int group)
{
    switch (bits) {
    case 2: return pick_dtype<VAR, D, 2>(f16, group);
    case 3: return pick_dtype<VAR, D, 3>(f16, group);
    case 4: return pick_dtype<VAR, D, 4>(f16, group);
    }
    return {nullptr, 0};
}

template <int VAR>
ScoreKernel pick_d(int d, int bits, bool f16, int group)
{
    switch (d) {
    case 128: return pick_bits<VAR, 128>(bits, f16, group);
    case 256: return pick_bits<VAR, 256>(bits, f16, group);
    case 512: return pick_bits<VAR, 512>(bits, f16, group);
    }
    return {nullptr, 0};
}

}  // namespace

ScoreKernel score_kernel_for(int variant, int d, int bits, bool f16, int group)
{
    switch (variant) {
    case VAR_FULL: return pick_d<VAR_FULL>(d, bits, f16, group);
    case VAR_FAST: return pick_d<VAR_FAST>(d, bits, f16, group);
    case VAR_PLANAR2D: return pick_d<VAR_PLANAR2D>(d, bits, f16, group);
    }
    return {nullptr, 0};
}

}  // namespace isoq
