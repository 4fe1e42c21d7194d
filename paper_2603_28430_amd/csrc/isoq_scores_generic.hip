// Attention logits at key widths without a tuned logit kernel.  The identity
// is the tuned kernels' (Prop. 1: T is orthogonal, so <q, x_hat> =
// rho <T q_pad, c[idx]> with q_pad the query zero-padded to the record's
// padded width, Sec. 5.1), evaluated directly: the workgroup's query is
// rotated once into LDS (scale folded in), then each lane takes one key and
// sums (T q)_j c[idx_j] over the padded coordinates, reading its record slot
// by slot as the generic stage-1 kernels write it (through the cache's
// piece-major layout).  This is the compatibility
// path for widths no model family of the paper uses; it is not tuned.
//
// Workgroup (query head, chunk of kScoreChunk positions, sequence).  Query
// head hq reads key head hq / group.  Positions at or past the sequence's
// length, and keys whose block-table entry is out of range, are not written.
#include "isoq_scores_generic.h"

#include "isoq_generic.h"

namespace isoq {
namespace {

template <int VAR, int BITS, bool F16>
__global__ __launch_bounds__(256) void generic_score_kernel(const SArgs a, const GenScoreShape g)
{
    constexpr int SW = kGenSW<VAR>;
    constexpr int PS = SW == 8 ? 64 : kSlotParams<VAR>;
    constexpr int K = 1 << BITS;
    extern __shared__ __align__(16) float gsm[];
    float *lev = gsm;       // c_0 .. c_{K-1}
    float *qt = gsm + 16;   // scale * T q_pad, slots * SW floats

    const int hq = blockIdx.x;
    const int h = hq / a.group;
    const int s = blockIdx.z;
    int64_t len = a.seq_lens[s];
    len = min(len, a.max_len);
    len = min(len, (int64_t)a.max_blocks * a.block_size);
    const int64_t t0 = (int64_t)blockIdx.y * kScoreChunk;
    if (t0 >= len)
        return;  // block-uniform: the whole workgroup leaves before the barrier
    const int set = a.n_sets == 1 ? 0 : h;

    if (threadIdx.x < K)
        lev[threadIdx.x] = a.lev_all[threadIdx.x];
    const int64_t qoff = ((int64_t)s * a.n_q_heads + hq) * g.d;
    for (int j = threadIdx.x; j < g.slots; j += blockDim.x) {
        float x[SW], y[SW], P[PS];
#pragma unroll
        for (int c = 0; c < SW; c++) {
            const int i = SW * j + c;
            if constexpr (F16)
                x[c] = i < g.d ? (float)static_cast<const _Float16 *>(a.q)[qoff + i] : 0.f;
            else
                x[c] = i < g.d ? static_cast<const float *>(a.q)[qoff + i] : 0.f;
        }
        load_params<PS>(a.params + set * g.set_stride + (int64_t)j * PS, P);
        if constexpr (SW == 8)
            rotate_forward<VAR>(P, x, y);
        else
            rotate4_forward<VAR>(P, x, y);
#pragma unroll
        for (int c = 0; c < SW; c++)
            qt[SW * j + c] = y[c] * a.scale;
    }
    __syncthreads();

    const int64_t tend = min(t0 + (int64_t)kScoreChunk, len);
    const int32_t *table = a.block_table + (int64_t)s * a.max_blocks;
    float *dst = a.scores + ((int64_t)s * a.n_q_heads + hq) * a.max_len;
    for (int64_t t = t0 + threadIdx.x; t < tend; t += blockDim.x) {
        const uint32_t bi = fast_div((uint32_t)t, a.div_block);
        const int32_t blk = table[bi];
        if (blk < 0 || blk >= a.n_blocks)
            continue;
        const int pos = (int)((uint32_t)t - bi * a.block_size);
        const int64_t krow = ((int64_t)blk * a.n_kv_heads + h) * a.block_size + pos;
        // the record, piece-major in its head's block region
        const CacheSrcRt rec{a.k_idx + (krow - pos) * g.rec, pos, a.block_size, g.rec_lp, g.rec};
        float acc = 0.f;
#pragma unroll 4
        for (int j = 0; j < g.slots; j++) {
            uint32_t p;
            if constexpr (SW == 8)
                p = gen_read_slot8<BITS>(rec, j);
            else
                p = gen_read_slot<BITS>(rec, j, g.rec);
#pragma unroll
            for (int c = 0; c < SW; c++)
                acc = fmaf(qt[SW * j + c], lev[(p >> (BITS * c)) & (K - 1)], acc);
        }
        dst[t] = a.k_rho[krow] * acc;
    }
}

template <int VAR, int BITS>
const void *gen_score_dtype(bool f16)
{
    return f16 ? reinterpret_cast<const void *>(&generic_score_kernel<VAR, BITS, true>)
               : reinterpret_cast<const void *>(&generic_score_kernel<VAR, BITS, false>);
}

template <int VAR>
const void *gen_score_bits(int bits, bool f16)
{
    switch (bits) {
    case 2: return gen_score_dtype<VAR, 2>(f16);
    case 3: return gen_score_dtype<VAR, 3>(f16);
    case 4: return gen_score_dtype<VAR, 4>(f16);
    }
    return nullptr;
}

}  // namespace

const void *generic_score_kernel_for(int variant, int bits, bool f16)
{
    switch (variant) {
    case VAR_FULL: return gen_score_bits<VAR_FULL>(bits, f16);
    case VAR_FAST: return gen_score_bits<VAR_FAST>(bits, f16);
    case VAR_PLANAR2D: return gen_score_bits<VAR_PLANAR2D>(bits, f16);
    case VAR_BLOCK8: return gen_score_bits<VAR_BLOCK8>(bits, f16);
    }
    return nullptr;
}

}  // namespace isoq
