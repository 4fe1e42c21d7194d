// Internal declarations shared by the library's host code (isoq_api.cpp,
// isoq_host_params.cpp) and its kernels (isoq_kernels.hip).
#pragma once

#include <stddef.h>
#include <stdint.h>

#include <vector>

namespace isoq {

enum Mode {
    MODE_ROUNDTRIP = 0,
    MODE_QUANTIZE = 1,
    MODE_DEQUANTIZE = 2,
    MODE_APPEND = 3,      // quantize into the slots of a paged cache
    MODE_QJL = 4,         // quantize with the stage-2 sketch
    MODE_APPEND_QJL = 5,  // both: records, norms, signs and gamma into cache slots
    // kernel_m_for only: round trip and quantize of rows whose set is the row
    // number mod n_sets (rows_per_set = 1), as n_sets interleaved streams
    MODE_STREAMS_ROUNDTRIP = 6,
    MODE_STREAMS_QUANTIZE = 7
};
// VAR_BLOCK8: 8-D grouped blocks, one 8x8 orthogonal matrix per 8 coordinates
enum Variant { VAR_FULL = 0, VAR_FAST = 1, VAR_PLANAR2D = 2, VAR_BLOCK8 = 3 };

// Every lane owns 8 consecutive coordinates of a row (two quaternion blocks or
// four planar pairs), so a row spans d/8 lanes and a wave holds 512/d rows.
constexpr int kCoordsPerLane = 8;
constexpr int kBlockThreads = 256;

// Row groups per wave in one block (a block covers 4 * kTileGroups groups,
// i.e. 64 rows of d = 128): four 16-byte loads in flight per lane.
constexpr int kTileGroups = 4;

// Device rotation parameters per lane, in floats: Full keeps the two 4x4
// matrices M = L(q_L) R(conj q_R) row-major, Fast the two unit quaternions,
// 2-D (cos, sin) of the four pairs, 8-D the block's 8x8 matrix row-major.
inline int params_per_lane(int variant) { return variant == VAR_FULL ? 32 : variant == VAR_BLOCK8 ? 64 : 8; }

// The same per 4-coordinate slot (one quaternion block, two planar pairs, or
// half of an 8-D block: its matrix rows 0..3, then rows 4..7), and the slots
// of a set: ceil(d/4) for Full and Fast, ceil(ceil(d/2) / 2) for 2-D (an odd
// pair count leaves an identity pair in the last slot), 2 ceil(d/8) for 8-D.
inline int params_per_slot(int variant) { return variant == VAR_FULL ? 16 : variant == VAR_BLOCK8 ? 32 : 4; }
inline int padded_width(int variant, int d)
{
    return variant == VAR_PLANAR2D ? 2 * ((d + 1) / 2) : variant == VAR_BLOCK8 ? 8 * ((d + 7) / 8) : 4 * ((d + 3) / 4);
}
inline int slots_per_set(int variant, int d) { return (padded_width(variant, d) + 3) / 4; }

// Division of 32-bit unsigned integers by a run-time constant d >= 1 through
// one multiply-high, two shifts and two adds (Granlund and Montgomery,
// "Division by invariant integers using multiplication", PLDI 1994, Fig. 4.1):
// t = mulhi(n, m), n / d = (t + ((n - t) >> s1)) >> s2, with
// l = ceil(log2 d), m = floor(2^32 (2^l - d) / d) + 1, s1 = min(l, 1),
// s2 = max(l - 1, 0).  Exact for every n < 2^32.
struct FastDiv {
    uint32_t m, s1, s2;
};

inline FastDiv make_fastdiv(uint32_t d)
{
    int l = 0;
    while ((1ull << l) < d)
        l++;
    const uint64_t m = ((1ull << 32) * ((1ull << l) - d)) / d + 1;
    return FastDiv{(uint32_t)m, (uint32_t)(l < 1 ? l : 1), (uint32_t)(l > 1 ? l - 1 : 0)};
}

// Kernel arguments, passed by value (they land in scalar registers).
struct KArgs {
    const void *x;           // roundtrip / quantize: input rows
    void *y;                 // roundtrip / dequantize: output rows
    uint8_t *rec_out;        // quantize: packed index records
    const uint8_t *rec_in;   // dequantize: packed index records
    float *norms_out;        // quantize: rho per row
    const float *norms_in;   // dequantize: rho per row
    const float *params;     // [n_sets][d/8][params_per_lane]
    int64_t n;               // rows
    int64_t rows_per_set;    // rows per parameter set (>= 1)
    int32_t n_sets;
    int32_t g_block_set;     // packed-row kernels: the rows of each block share one set
    const float *lut;        // magnitude lookup table (4-bit codebooks), [lut_cells][4]
    float lut_inv_h;         // 1 / cell width, in units of the normalised coordinate
    int32_t lut_cells;
    float lev_pos[8];        // c_{K/2} .. c_{K-1}   (positive half of the codebook)
    float thr_pos[8];        // t_{K/2} .. t_{K-2}   (positive thresholds; t_{K/2-1} = 0)
    float lev_all[16];       // c_0 .. c_{K-1}
    // append into a paged cache (n = tokens; the head is blockIdx.y)
    const int64_t *slots;    // [n_tokens] cache slot of each token
    int64_t n_slots;         // cache capacity in slots (n_blocks * block_size)
    uint32_t n_heads, block_size;
    FastDiv div_block;
    // the forward rotation on the matrix cores (isoq_stage1m.h): per set,
    // chunk and quad row, the fp16 (hi, lo) rows of the chunk's 4x4 matrices
    const uint32_t *mfma;
    // stage-2 residual sketch (quantize with QJL)
    const uint16_t *qjl_frag;  // [n_sets][m/16][dp/32][64][8] fp16: S' = S T^{-1} in fragment order,
                               // dp = d rounded up to a multiple of 32 (zero columns past d)
    uint8_t *qjl_signs;        // [n][m/8] sign bits of S (x - x_hat)
    float *qjl_gamma;          // [n] ||x - x_hat||
    // widths outside {64, 128, 256, 512} (isoq_generic.h)
    int32_t g_d;               // coordinates per row
    int32_t g_pw;              // padded width: 4 ceil(d/4), 2-D 2 ceil(d/2)
    int32_t g_slots;           // 4-coordinate slots per row, ceil(g_pw / 4)
    int32_t g_rec;             // record bytes, ceil(g_pw * bits / 8)
    int32_t g_vec;             // rows move in whole slots (d a multiple of 4)
    int32_t g_rows;            // packed-row kernels (isoq_packed.h): rows per wave group
    int32_t g_tpb;             // packed-row kernels with the sketch: row tiles per block
    int64_t g_set_stride;      // floats per parameter set, kSlotParams * g_slots
};

// Attention logits against a paged cache of quantized keys (isoq_scores.hip).
struct SArgs {
    const void *q;               // [n_seqs][n_q_heads][d] queries
    const uint8_t *k_idx;        // [n_blocks][n_kv_heads][block_size][record]
    const float *k_rho;          // [n_blocks][n_kv_heads][block_size]
    const int32_t *block_table;  // [n_seqs][max_blocks]
    const int32_t *seq_lens;     // [n_seqs]
    float *scores;               // [n_seqs][n_q_heads][max_len]
    const float *params;         // rotation parameters, device layout of the stage-1 kernels
    int64_t max_len, n_blocks;
    int32_t n_q_heads, n_kv_heads, group, block_size, max_blocks, n_sets;
    float scale;
    int32_t pad0;
    FastDiv div_block;
    float lev_all[16];           // c_0 .. c_{K-1}
    // stage-2 residual correction (kernels with a sketch only)
    const float *qjl_S;          // [m][d] fp32 projection
    const uint8_t *k_signs;      // [n_blocks][n_kv_heads][block_size][m/8]
    const float *k_gamma;        // [n_blocks][n_kv_heads][block_size]
    float qjl_scale;             // scale * sqrt(pi/2) / m
    int32_t pad1;
};

// Keys per workgroup of the score kernel.
constexpr int kScoreChunk = 1024;

// Score kernel for (variant, d, bits, fp16 queries?, query heads per key
// head) and the dynamic LDS bytes it needs (0 when its LDS is static), or
// {nullptr, 0}.
struct ScoreKernel {
    const void *fn;
    size_t dyn_lds;
};
ScoreKernel score_kernel_for(int variant, int d, int bits, bool f16, int group);
ScoreKernel score_kernel_for_block8(int d, int bits, bool f16, int group);
// The same with the stage-2 residual correction of m sign bits (isoq_scores_qjl.hip).
ScoreKernel score_qjl_kernel_for(int variant, int d, int bits, bool f16, int group, int m);

// Paged caches (isoq_kv_append, isoq_kv_scores) hold a head's records of
// one cache block piece-major: a record of R bytes is cut into pieces of
// P = cache_piece(R) bytes, and piece j of position pos lies at byte
// (j block_size + pos) P of the head's block region, so consecutive
// positions' pieces are adjacent.  P is 16 or 8 when that divides R; other
// records are one piece (P = R: stored whole, one after the other).
constexpr int cache_piece(int64_t R) { return R % 16 == 0 ? 16 : R % 8 == 0 ? 8 : (int)R; }

// Variants and widths whose fp16 encoders (round trip, quantize, append,
// sketch) rotate on the matrix cores in the quad layout (isoq_stage1m.h), and
// the kernel for (variant, d, bits, mode) there (round trip, quantize,
// append), or nullptr.  2-D rows at 4 bits keep the VALU encoder (its round
// trip measured 5% faster there; at 2 and 3 bits the matrix cores are
// faster, quantize by up to 6%).
constexpr bool quad_layout(int variant, int d, int bits)
{
    return (d == 64 || d == 128 || d == 256) && (variant != VAR_PLANAR2D || bits != 4);
}
const void *kernel_m_for(int variant, int d, int bits, int mode);
// Bytes of the matrix-core parameters per set: d/8 chunks x 4 quad rows x
// (2 slots, 8-D: 4 sub-blocks) x 16 bytes of fp16 (hi, lo) rows.
inline size_t mfma_bytes_per_set(int variant, int d) { return (size_t)(d / 8) * 4 * (variant == VAR_BLOCK8 ? 4 : 2) * 16; }
// Build them from a set's device-layout fp32 parameters (isoq_host_params.cpp).
void build_mfma_params(int variant, int d, const float *set_layout, uint16_t *out);

// Kernel entry for (variant, d, bits, fp16 rows?, generic set indexing?, mode),
// or nullptr.  Generic set indexing is needed when there is more than one
// set and rows_per_set is not a multiple of the rows of a block.
const void *kernel_for(int variant, int d, int bits, bool f16, bool generic_sets, int mode);
// The same for 8-D blocks (isoq_kernels_8d.hip).
const void *kernel_for_block8(int d, int bits, bool f16, bool generic_sets, int mode);
// Stage-1 kernels for the other widths (d = 1 .. 1024) with `slots` slots
// per padded row (4 coordinates; 8 for 8-D blocks), one per variant
// (isoq_generic_*.hip); nullptr when no kernel fits.  Rows of one block:
// 4 waves x generic_rows_per_wave.
// pairs: fp16 rows whose width is even and not a multiple of 4 move in
// coordinate pairs (separate instantiations)
const void *generic_kernel_full(int slots, int bits, bool f16, int mode, bool pairs);
const void *generic_kernel_fast(int slots, int bits, bool f16, int mode, bool pairs);
const void *generic_kernel_2d(int slots, int bits, bool f16, int mode, bool pairs);
const void *generic_kernel_8d(int slots, int bits, bool f16, int mode, bool pairs);
// Row shape of the generic kernels for a row of `slots` slots of sw
// coordinates: G lanes per row, BPL slots per lane, and row groups per wave
// (every group's loads are in flight together: 8 groups of one 4-coordinate
// slot, 4 groups of several; half as many for 8-coordinate slots, whose 64
// parameters per slot fill the registers).
// fp32 rows of 17 to 64 four-coordinate slots take two slots per lane on
// half the lanes (measured at d = 96: Full quantize 0.52 -> 0.56, the round
// trips 1-2% faster); fp16 rows there lost up to 17% that way and keep one.
inline bool generic_two_slots(int slots, int sw, bool f16) { return !f16 && sw == 4 && slots > 16 && slots <= 64; }
inline int generic_lanes(int slots, int sw, bool f16)
{
    if (generic_two_slots(slots, sw, f16))
        return slots <= 32 ? 16 : 32;
    return slots <= 8 ? 8 : slots <= 16 ? 16 : slots <= 32 ? 32 : 64;
}
inline int generic_bpl(int slots, int sw, bool f16)
{
    if (generic_two_slots(slots, sw, f16))
        return 2;
    return slots <= 64 ? 1 : slots <= 128 ? 2 : 4;
}
constexpr int generic_groups(int bpl, int sw) { return (bpl == 1 ? 8 : 4) / (sw == 8 ? 2 : 1); }
inline int generic_rows_per_wave(int slots, int sw, bool f16)
{
    return generic_groups(generic_bpl(slots, sw, f16), sw) * (64 / generic_lanes(slots, sw, f16));
}
constexpr int kGenericMaxD = 1024;
// Packed-row kernels (isoq_packed.h) for fp16 rows of width d = 16 k up to
// 504 outside the tuned widths.  One 8-coordinate chunk per lane: L = d/8
// lanes per row, V = floor(64 / L) rows per wave group, one fewer for 3 bits
// when V L is not a multiple of 4 (a quad of lanes writes whole words).  Two
// chunks per lane (one in each half of the row, L = d/16 lanes per row, L
// even and, for 3 bits, a multiple of 4) where that keeps more lanes busy:
// d = 192 and 320 (and 288 at 2 and 4 bits).  rows = 0 where the family does
// not apply (the generic kernels take those widths and every fp32 row).
constexpr int kPackedMaxLanes = 63;   // d/8 at d = 504
struct PackedShape {
    int rows;     // rows per wave group
    int chunks;   // 8-coordinate chunks per lane
};
constexpr PackedShape packed_shape(int d, int bits, bool f16)
{
    if (!f16 || d % 16 != 0 || d > 8 * kPackedMaxLanes || d == 64 || d == 128 || d == 256)
        return {0, 0};
    const int l1 = d / 8;
    int v1 = 64 / l1;
    if (bits == 3 && (v1 * l1) % 4 != 0)
        v1--;
    const int l2 = d / 16;
    if (d % 32 == 0 && (bits != 3 || l2 % 4 == 0)) {
        const int v2 = 64 / l2;
        if (v2 * l2 > v1 * l1)
            return {v2, 2};
    }
    return {v1, 1};
}
// Row tiles (4 waves x kTileGroups / chunks groups) per block: two for Full
// (and 8-D blocks) with two chunks per lane, which halves its LDS staging per tile (measured
// 4% faster at d = 192; one chunk per lane measured 2-4% slower with two).
constexpr int packed_tiles_per_block(int variant, int chunks)
{
    return (variant == VAR_FULL || variant == VAR_BLOCK8) && chunks == 2 ? 2 : 1;
}
// (cache_lp, append only: the cache layout's pieces, 1 << cache_lp bytes, or
// records whole for cache_lp < 0)
const void *packed_kernel_full(int bits, int mode, int chunks, int cache_lp = -1);
const void *packed_kernel_fast(int bits, int mode, int chunks, int cache_lp = -1);
const void *packed_kernel_2d(int bits, int mode, int chunks, int cache_lp = -1);
const void *packed_kernel_8d(int bits, int mode, int chunks, int cache_lp = -1);
// Packed-row kernels with the stage-2 sketch of m bits (isoq_packed_qjl.hip):
// quantize into rows (one rotation set) or, with `append`, into the slots of
// a paged cache, for fp16 rows at d = 80, 96, 160 and 192; or nullptr.
const void *packed_qjl_kernel_for(int variant, int d, int bits, int m, bool append);
// Projection width of the sketch: d rounded up to a multiple of 32 (the
// k-step of the projection's matrix instruction).
constexpr int qjl_proj_width(int d) { return (d + 31) / 32 * 32; }
// Waves per block of the packed-row kernels with the sketch.
constexpr int kPackedQjlWaves = 8;
// Row groups per wave of the packed-row kernels: kTileGroups / chunks, and
// with the sketch at most 16 / rows, so that a wave's tile fits one 16-row
// block of the projection.
constexpr int packed_groups(int rows, int chunks, bool sketch)
{
    return sketch && 16 / rows < kTileGroups / chunks ? 16 / rows : kTileGroups / chunks;
}
// Blocks of the stage-2 sketch kernel with a single rotation set (each walks
// several tiles).
constexpr int64_t kQjlBlocks = 1024;
// Quantize with the stage-2 sketch of m bits (isoq_qjl.hip), or nullptr;
// with `append`, the kernel that writes into the slots of a paged cache.
const void *qjl_kernel_for(int variant, int d, int bits, bool f16, int m, bool append, int waves);
// Waves per block of the sketch kernels: 8, so that one staged copy of the
// projection serves twice the waves (at d = 128, m = 128 LDS admits 12 waves
// of 4-wave blocks per CU, 16 of 8-wave blocks; the 8-wave kernels also take
// fewer registers); 4 for quantize into rows with several sets (a block's
// rows share one set, and rows_per_set must stay a multiple of the smaller
// block).
inline int qjl_waves(int m, bool append, int n_sets) { return append || n_sets == 1 ? 8 : 4; }

// Magnitude lookup table, used for 4-bit codebooks.  The magnitude axis of
// the normalised coordinate is cut into cells of width h, h smaller than every
// gap between consecutive positive thresholds (and than the first one), so a
// cell holds at most one threshold.  Entry c = {threshold inside the cell in
// cell units (+inf if none), level below it, level above it, magnitude index
// below it}; values past the last cell use the last entry.
constexpr int kLutMaxCells = 256;
struct LutEntry {
    float t, lo, hi;
    uint32_t m;
};
static_assert(sizeof(LutEntry) == 16, "LUT entries are 16 bytes");

// ---- host-side parameter construction (isoq_host_params.cpp) -------------
// Build the table from the positive thresholds tau[0..H-2] and the positive
// levels lev[0..H-1] (H = 2^(bits-1)).  Returns false if more than
// kLutMaxCells cells would be needed.
bool build_magnitude_lut(int H, const double *tau, const double *lev, double *inv_h,
                         std::vector<LutEntry> &lut);
// Lloyd-Max levels for N(0, sigma^2) (ascending, symmetrised).
bool lloyd_levels(int bits, double sigma, int iters, double *levels);
// Seeded raw draws (Philox4x32-10 + Box-Muller), layout of the public header.
void seeded_draws(int variant, int d, int n_sets, uint64_t seed, double *out);
size_t raw_per_set(int variant, int d);
size_t export_per_set(int variant, int d);
// Seeded stage-2 projection S [m][d] (Philox4x32-10 stream 3 + Box-Muller).
void seeded_projection(int m, int d, uint64_t seed, double *out);
// The forward block rotation of one set (exported unit parameters, Table 1
// layout) applied to `rows` vectors of length d.
void rotate_rows_forward(int variant, int d, const float *unit_set, const double *in, int rows, double *out);
// From raw draws to (a) the exported unit parameters and (b) the device
// layout.  Returns false when a quaternion draw is zero or not finite.
bool build_rotation(int variant, int d, int n_sets, const double *raw, std::vector<float> &exported,
                    std::vector<float> &device_layout);

}  // namespace isoq
