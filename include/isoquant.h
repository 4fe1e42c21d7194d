/*
 * isoquant.h -- C ABI of the IsoQuant stage-1 quantize/dequantize library for
 * AMD Instinct MI355X (gfx950).
 *
 * IsoQuant (arXiv 2603.28430) compresses a d-dimensional vector x in four
 * steps (Algorithm 1): split off the norm rho = ||x|| (Sec. 3); rotate the
 * direction block by block, with 4-D quaternion blocks v -> q_L v conj(q_R)
 * (IsoQuant-Full, Sec. 5.2), v -> q_L v (IsoQuant-Fast, Sec. 5.3), 2-D
 * planar rotations (Sec. 5.4) or 8-D grouped blocks (Table 3's block-size
 * axis, Haar(SO(8)) blocks as in Sec. 5.7); quantize every rotated coordinate with one
 * shared b-bit Lloyd-Max codebook; then dequantize, rotate back and multiply
 * by rho.
 *
 * Conventions shared by every call:
 *   - Status codes are returned, never exceptions.  Arguments are validated
 *     before any device work; a call that returns an error launched nothing.
 *   - Rows are contiguous, row-major [n][d].  Coordinate 4i of a row is the
 *     real part of quaternion block i; the 2-D case pairs (2j, 2j+1); 8-D
 *     block i holds coordinates 8i .. 8i+7.
 *   - Device buffers are owned by the caller and must live on the device that
 *     was current at isoq_params_init.  Row buffers (fp16/fp32) must be
 *     16-byte aligned, index records and norm arrays 4-byte aligned.
 *   - `stream` is a hipStream_t (NULL = the null stream).  Calls are
 *     asynchronous on it and never synchronise the device.  n = 0 is a valid
 *     no-op.  Output buffers must not overlap inputs, except that the
 *     reconstruction may be written in place over the input of
 *     isoq_roundtrip (x_hat == x exactly).
 *   - A parameter handle is immutable after init; concurrent calls that share
 *     it are safe.  Only init and destroy allocate or free device memory.
 *   - Supported shapes in this version: bits in {2, 3, 4}, fp16 or fp32 rows
 *     (arithmetic is fp32 in every case); d from 1 to 1024 for quantize,
 *     dequantize and round trip (tuned kernels for d in {64, 128, 256, 512},
 *     packed-row kernels for fp16 rows at other multiples of 16 up to 504, a
 *     generic kernel family for every other width), d in {64, 128, 256, 512}
 *     for the KV-cache append (and, fp16 rows only, 80, 96, 160 and 192), d in
 *     {64, 80, 96, 128, 160, 192, 256, 512} for the attention-score call
 *     without the sketch, d in {64, 128, 256, 512} and (fp16 rows, or any
 *     query type for the scores) 80, 96, 160 and 192 for the stage-2 sketch
 *     and the calls that use it (Full, Fast and 2-D handles; every other call
 *     takes all four variants).
 *   - Widths that are not a multiple of the block size (4; 2-D: 2; 8-D: 8)
 *     follow Sec. 5.1: the last block is zero padded, all pw rotated
 *     coordinates are quantized and stored (pw = 4 ceil(d/4); 2-D:
 *     2 ceil(d/2); 8-D: 8 ceil(d/8)), and the padded coordinates are dropped
 *     after the inverse rotation.
 *   - Rows must be finite.  The squared norm is accumulated in fp32, so an
 *     fp32 row must have 1e-18 <= ||x|| <= 1e18 or be exactly zero (every fp16
 *     row qualifies); a zero row gives rho = 0, x_hat = 0 and every index
 *     2^(bits-1) - 1.
 */
#ifndef ISOQUANT_H
#define ISOQUANT_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum isoq_status {
    ISOQ_OK = 0,
    ISOQ_E_INVALID = 1,     /* bad enum value, n < 0, rows_per_set < 1, bad codebook  */
    ISOQ_E_UNSUPPORTED = 2, /* valid request outside the shapes listed above           */
    ISOQ_E_NULL = 3,        /* required pointer is NULL                                */
    ISOQ_E_ALIGN = 4,       /* pointer misaligned                                      */
    ISOQ_E_HIP = 5,         /* HIP runtime error (launch failure, no device, ...)      */
    ISOQ_E_NOMEM = 6,       /* device or host allocation failed                        */
    ISOQ_E_DEVICE = 7       /* called with a device other than the handle's            */
} isoq_status;

/* variants (Sec. 5.2, 5.3, 5.4; ISOQ_BLOCK8: 8-D grouped blocks, Table 3 and
 * Sec. 5.7) */
enum { ISOQ_FULL = 0, ISOQ_FAST = 1, ISOQ_PLANAR2D = 2, ISOQ_BLOCK8 = 3 };
/* row element types */
enum { ISOQ_F32 = 0, ISOQ_F16 = 1 };

typedef struct isoq_params isoq_params;

/*
 * isoq_params_init -- build the rotation parameters and the codebook of one
 * quantizer and copy them to the current device.
 *
 *   variant   ISOQ_FULL, ISOQ_FAST, ISOQ_PLANAR2D or ISOQ_BLOCK8.
 *   d, bits   vector width and bits per coordinate.
 *   n_sets    number of independent rotation sets (e.g. one per attention
 *             head); row r of a later call uses set (r / rows_per_set) mod
 *             n_sets.  The codebook is shared by all sets.
 *   rot_host  NULL, or host array of raw draws (Sec. 5.5: unconstrained
 *             vectors normalised on the fly), n_sets * isoq_raw_params_per_set
 *             doubles: Full, per set and block i, u_L[4] then u_R[4]; Fast,
 *             u_L[4] per block; 2-D, one angle theta (radians) per coordinate
 *             pair; 8-D, a raw 8x8 matrix G per block of 8 coordinates
 *             (row-major).  Quaternions are normalised here (u / ||u||); a zero
 *             u is ISOQ_E_INVALID.  An 8-D block rotates by the orthogonal
 *             factor Q of G = QR with a positive diagonal in R (Haar on O(8)
 *             for Gaussian G), with column 0 negated when det Q = -1 (so Q is
 *             in SO(8)); G with dependent columns is ISOQ_E_INVALID.
 *             NULL: draw them from `seed` (Haar sampling, Sec. 5.5): u ~ N(0,I4)
 *             and theta ~ U[0, 2 pi) from Philox4x32-10 with key = seed and
 *             counter (block, set, stream, 0), stream 0 for u_L, 1 for u_R, 2 for
 *             theta (8-D: G ~ N(0,1) entries 4q .. 4q+3 from counter
 *             (block, set, 4, q), q = 0..15); Box-Muller maps the four 32-bit words (w0..w3) to
 *             (z0, z1) = sqrt(-2 ln U1) (cos 2 pi U2, sin 2 pi U2) with
 *             U1 = (w0 + 1/2) / 2^32, U2 = w1 / 2^32, likewise (z2, z3) from
 *             (w2, w3); theta = 2 pi w0 / 2^32.
 *   codebook_host  NULL, or host array of 2^bits levels, strictly increasing
 *             and symmetric about 0 (|c_k + c_{K-1-k}| <= 1e-6 max|c|; they are
 *             then symmetrised exactly).  NULL: Lloyd-Max levels for N(0, 1/d)
 *             after 200 Lloyd iterations from levels evenly spaced on
 *             [-3/sqrt(d), 3/sqrt(d)].  Decision thresholds are the midpoints
 *             of adjacent levels.  The kernels take the sign of a rotated
 *             value y (y > 0) and compare |y| with the positive thresholds
 *             (|y| > t), so a value exactly on a threshold goes to the level
 *             of smaller magnitude: the lower level for y > 0, the upper one
 *             for y < 0 (0 itself goes to level 2^(bits-1) - 1).
 *   out       receives the handle (set to NULL on error).
 * Host arrays are only read during the call; the caller keeps ownership.
 */
isoq_status isoq_params_init(isoq_params **out, int variant, int d, int bits, int n_sets,
                             const double *rot_host, const double *codebook_host, uint64_t seed);

/* Free the handle and its device memory (NULL is accepted).  Must not race
 * with calls still running on the GPU that use the handle: synchronise their
 * streams first. */
isoq_status isoq_params_destroy(isoq_params *p);

/*
 * isoq_params_export -- copy out the values the device uses (fp32).  Any
 * output may be NULL.
 *   rot_out        n_sets * isoq_export_params_per_set floats: Full, per
 *                  block q_L[4] then q_R[4] (unit); Fast q_L[4]; 2-D
 *                  (cos theta, sin theta) per pair; 8-D the block's
 *                  orthogonal Q (64 floats, row-major).  These are the
 *                  parameter counts of Table 1 (8 g4, 4 g4, 2 g2 per set;
 *                  8-D, not in Table 1: 64 g8).
 *   levels_out     2^bits levels, ascending.
 *   thresholds_out 2^bits - 1 decision thresholds, ascending.
 */
isoq_status isoq_params_export(const isoq_params *p, float *rot_out, float *levels_out,
                               float *thresholds_out);

/* Read back the shape of a handle (any output may be NULL). */
isoq_status isoq_params_info(const isoq_params *p, int *variant, int *d, int *bits, int *n_sets);

/*
 * isoq_quantize -- encoder half of Algorithm 1: norm split, blockwise rotation,
 * scalar quantization.
 *   x          device, [n][d] rows of `dtype`.
 *   idx_packed device, [n][isoq_record_bytes(variant, d, bits)] bytes: per row
 *              one record of the pw rotated coordinates in which coordinate j
 *              occupies bits [j*bits, (j+1)*bits), bit m being bit (m mod 8) of
 *              byte m/8 (least significant first); bits past pw*bits are 0.
 *   norms      device, [n] fp32 rho = ||x||_2.
 * Index of a coordinate y: number of thresholds t_k with y > t_k applied to the
 * direction x / max(rho, 1e-12).
 */
isoq_status isoq_quantize(const isoq_params *p, int dtype, const void *x, int64_t n,
                          int64_t rows_per_set, uint8_t *idx_packed, float *norms, void *stream);

/*
 * isoq_dequantize -- decoder half of Algorithm 1: level lookup, inverse block
 * rotation, multiplication by rho.  Inputs as produced by isoq_quantize; output
 * x_hat device [n][d] rows of `dtype` (fp16 is rounded to nearest even).
 */
isoq_status isoq_dequantize(const isoq_params *p, int dtype, const uint8_t *idx_packed,
                            const float *norms, int64_t n, int64_t rows_per_set, void *x_hat,
                            void *stream);

/*
 * isoq_roundtrip -- the fused stage-1 path x -> x_hat of Algorithm 1 with no
 * index traffic to memory.  Bitwise equal to isoq_quantize followed by
 * isoq_dequantize on the same handle, rows_per_set and dtype.
 */
isoq_status isoq_roundtrip(const isoq_params *p, int dtype, const void *x, int64_t n,
                           int64_t rows_per_set, void *x_hat, void *stream);

/*
 * isoq_kv_append -- quantize-on-append into a paged K/V cache, for
 * autoregressive decoding (the fused KV-cache compression the paper names as
 * its next step, Sec. 10): the new key and value rows are encoded as by
 * isoq_quantize (Algorithm 1's encoder) and their index records and norms are
 * written straight into the cache slots of their tokens.  Any d in 1..1024:
 * d in {64, 128, 256, 512}, and fp16 rows at 80, 96, 160 and 192, take one
 * launch for both tensors; other widths, and fp32 rows at those four, one
 * launch of the width-generic encoder per tensor.
 *
 *   pk, pv      handles of the K and V quantizers.  They must agree in variant,
 *               d and bits; each has n_sets == 1 or n_sets == n_heads, and the
 *               row of (token t, head h) uses set h (resp. set 0).  pv may be
 *               pk.  pv, v_new, v_idx and v_rho all NULL: keys only.
 *   dtype       ISOQ_F16 or ISOQ_F32, the element type of k_new and v_new.
 *   k_new, v_new  device, [n_tokens][n_heads][d] rows (16-byte aligned).
 *   slot_mapping  device, int64 [n_tokens] (8-byte aligned): cache slot of
 *               token t; a slot < 0 or >= n_blocks * block_size skips the token
 *               (padding), its rows are not written.
 *   k_idx, v_idx  device, n_blocks * n_heads * block_size * R bytes (R =
 *               isoq_packed_bytes; 4-byte aligned): slot s is position s mod
 *               block_size of cache block s / block_size, and (block b, head
 *               h) owns the block_size * R bytes from (b n_heads + h)
 *               block_size R on.  Inside that region the records are stored
 *               piece-major: record byte k of position p lies at byte
 *               (floor(k / P) block_size + p) P + k mod P, with P = 16 if 16
 *               divides R, else 8 if 8 divides R, else P = R (records stored
 *               whole, position after position).  Pieces of consecutive
 *               positions are adjacent, which the logit kernel reads in one
 *               coalesced load.  Record bytes as in isoq_quantize.
 *   k_rho, v_rho  device, fp32 [n_blocks][n_heads][block_size].
 * Limits: n_tokens * n_heads < 2^31, n_blocks * block_size < 2^31, n_heads and
 * block_size >= 1, and for the one-launch shapes at most 65,535 launch blocks
 * of tokens (n_tokens up to 8,388,480 at d = 64, 4,194,240 at d = 128,
 * 2,097,120 at d = 256, 1,048,560 at d = 512; fp16 rows: 6,291,360 at d = 80,
 * 5,242,800 at d = 96, 3,145,680 at d = 160, 2,621,400 at d = 192); beyond
 * that ISOQ_E_UNSUPPORTED.  Distinct tokens must map to distinct slots (a repeated slot
 * is written by both rows in an unspecified order).  Slots not named are left
 * untouched.  n_tokens = 0 is a no-op.
 */
isoq_status isoq_kv_append(const isoq_params *pk, const isoq_params *pv, int dtype,
                           const void *k_new, const void *v_new, const int64_t *slot_mapping,
                           int64_t n_tokens, int n_heads, uint8_t *k_idx, float *k_rho,
                           uint8_t *v_idx, float *v_rho, int64_t n_blocks, int block_size,
                           void *stream);

/*
 * isoq_kv_scores -- attention logits of decoding queries against the keys of
 * a paged cache written by isoq_kv_append, without dequantizing the keys.  A
 * key's reconstruction is rho T^{-1}(c[idx]) and T is orthogonal (Prop. 1), so
 * <q, k_hat> = rho <T q, c[idx]>: each query is rotated once and the logits
 * are sums of table lookups over the packed index records.  Any d in 1..1024:
 * at d in {64, 80, 96, 128, 160, 192, 256, 512} with lookup tables; at other
 * widths a width-generic kernel sums (T q_pad)_j c[idx_j] over the record's
 * zero-padded coordinates (q_pad: q with zeros past d), one workgroup per
 * query head.
 *
 *   pk          the K quantizer (n_sets == 1 or n_sets == n_kv_heads; key head h
 *               uses set h, resp. 0).
 *   dtype       ISOQ_F16 or ISOQ_F32, the element type of q.
 *   q           device, [n_seqs][n_q_heads][d] (16-byte aligned).  Query head hq
 *               reads key head hq / (n_q_heads / n_kv_heads) (grouped-query
 *               attention; n_q_heads must be a multiple of n_kv_heads).
 *   k_idx, k_rho  the cache, laid out as in isoq_kv_append (k_idx 16-byte
 *               aligned), n_blocks cache blocks of block_size positions.
 *   block_table device, int32 [n_seqs][max_blocks_per_seq]: cache block of the
 *               sequence's positions [j * block_size, (j+1) * block_size).
 *   seq_lens    device, int32 [n_seqs]: positions of each sequence.
 *   scores      device, fp32 [n_seqs][n_q_heads][max_len]:
 *               scores[s][hq][t] = scale * <q[s][hq], k_hat(s, t)> for
 *               t < min(seq_lens[s], max_len, max_blocks_per_seq * block_size).
 *               Other positions, and positions whose block id lies outside
 *               [0, n_blocks), are not written.
 * Limits: n_seqs <= 65535, max_blocks_per_seq * block_size < 2^31, and at the
 * table widths the tables of one key head's query group must fit in LDS:
 * group * (d/F * 2^(F bits) + d) * 4 bytes with F = 2 for 2 and 3 bits, F = 1
 * for 4 bits (ISOQ_E_UNSUPPORTED otherwise; e.g. at d = 128, 3 bits, 16.9 KB
 * per query head).  Logits are accumulated in fp32.
 */
isoq_status isoq_kv_scores(const isoq_params *pk, int dtype, const void *q, int n_seqs,
                           int n_q_heads, int n_kv_heads, const uint8_t *k_idx, const float *k_rho,
                           int64_t n_blocks, int block_size, const int32_t *block_table,
                           int max_blocks_per_seq, const int32_t *seq_lens, float scale,
                           float *scores, int64_t max_len, void *stream);

/*
 * Stage-2 residual sketch (Sec. 8: the stage-1 residual r = x - x_hat is
 * projected by a quantized Johnson-Lindenstrauss transform and corrects inner
 * products without bias).  A sketch handle holds a Gaussian projection S
 * [m][d]; a row is stored as its stage-1 record and rho plus the m sign bits
 * z_i = [(S r)_i > 0] and gamma = ||r||, and <q, x> is estimated by
 *     <q, x_hat> + sqrt(pi/2) / m * gamma * <S q, 2 z - 1>.
 *
 * isoq_sketch_init -- build the sketch of quantizer p on the current device.
 *   m       sketch bits per row: 64 or 128 at d = 64, 80, 96, 128, 160 and
 *           192; 64 at d = 256 and 512 (the projection, m d fp16, is staged in
 *           LDS).  Other d, other m, or an 8-D handle: ISOQ_E_UNSUPPORTED.
 *   S_host  NULL, or host array [m][d] of doubles (row-major).  NULL: S is
 *           drawn from `seed`: S[i][4g .. 4g+3] is the Box-Muller quadruple of
 *           Philox4x32-10 with key = seed and counter (g, i, 3, 0) (the
 *           mapping of isoq_params_init).
 * The sketch is bound to p's rotation (it stores S T^{-1} for every set); use
 * it only with the handle it was built from.  Only init and destroy allocate.
 */
typedef struct isoq_sketch isoq_sketch;
isoq_status isoq_sketch_init(isoq_sketch **out, const isoq_params *p, int m, const double *S_host,
                             uint64_t seed);
isoq_status isoq_sketch_destroy(isoq_sketch *sk);
/* m and the projection S as used (fp32, [m][d]); any output may be NULL. */
isoq_status isoq_sketch_export(const isoq_sketch *sk, int *m, float *S_out);

/*
 * isoq_quantize_qjl -- isoq_quantize plus the stage-2 sketch of every row.
 *   idx_packed, norms  as isoq_quantize (bitwise the same records and norms).
 *   signs   device, [n][m/8] bytes (4-byte aligned): bit i of a row's record
 *           (bit i mod 8 of byte i / 8) is z_i.  The projection runs in fp16
 *           with fp32 accumulation, so a sign whose exact projection lies
 *           within about 2^-9 sum_j |S'_ij| |e_j| rho of zero may differ from
 *           an exact computation (S' = S T^{-1}, e the normalised rotated error).
 *   gamma   device, [n] fp32 ||x - x_hat||.
 * Needs one rotation set per block of rows: n_sets == 1, or rows_per_set a
 * multiple of 64 rows at d = 128 (32 at d = 256); ISOQ_E_UNSUPPORTED otherwise.
 * At d = 80, 96, 160 and 192: fp16 rows and n_sets == 1 only.
 */
isoq_status isoq_quantize_qjl(const isoq_params *p, const isoq_sketch *sk, int dtype, const void *x,
                              int64_t n, int64_t rows_per_set, uint8_t *idx_packed, float *norms,
                              uint8_t *signs, float *gamma, void *stream);

/*
 * isoq_kv_append_qjl -- quantize-on-append of key rows with the stage-2
 * residual sketch (Sec. 8): each new key row is encoded as by
 * isoq_quantize_qjl (records, norms, m sign bits and gamma, bit for bit the
 * same) and all four go straight into the cache slot of its token, in one
 * launch.  Values need no sketch: append them with isoq_kv_append.
 *
 *   pk, sk      the K quantizer and its sketch (same variant, d, sets and
 *               device); pk->n_sets == 1 or n_heads (head h uses set h).
 *   dtype, k_new, slot_mapping, n_tokens, n_heads, k_idx, k_rho, n_blocks,
 *   block_size  as in isoq_kv_append.
 *   k_signs     device, [n_blocks][n_heads][block_size][m/8] bytes (4-byte
 *               aligned), the sign sketch of each slot, bit i of byte i/8 =
 *               [(S (x - x_hat))_i > 0].
 *   k_gamma     device, fp32 [n_blocks][n_heads][block_size], ||x - x_hat||.
 * Skipped slots (< 0 or >= n_blocks * block_size) are not written; other
 * slots not named are untouched.  Limits as in isoq_kv_append; the widths and
 * sketch sizes are those of isoq_sketch_init.
 */
isoq_status isoq_kv_append_qjl(const isoq_params *pk, const isoq_sketch *sk, int dtype, const void *k_new,
                               const int64_t *slot_mapping, int64_t n_tokens, int n_heads, uint8_t *k_idx,
                               float *k_rho, uint8_t *k_signs, float *k_gamma, int64_t n_blocks, int block_size,
                               void *stream);

/*
 * isoq_kv_scores_qjl -- isoq_kv_scores with the stage-2 residual correction:
 *   scores[s][hq][t] = scale * (rho <T q, c[idx]> + sqrt(pi/2) / m * gamma
 *                               * <S q, 2 z - 1>)
 * for keys stored with their sketch: k_signs device [n_blocks][n_kv_heads]
 * [block_size][m/8] bytes and k_gamma device fp32 [n_blocks][n_kv_heads]
 * [block_size] (4-byte aligned), in the layout of k_idx / k_rho (sign
 * records as written by isoq_quantize_qjl).  sk is the keys' sketch (built
 * from pk).  Other arguments and limits as isoq_kv_scores; S q is computed
 * in fp32.
 */
isoq_status isoq_kv_scores_qjl(const isoq_params *pk, const isoq_sketch *sk, int dtype, const void *q,
                               int n_seqs, int n_q_heads, int n_kv_heads, const uint8_t *k_idx,
                               const float *k_rho, const uint8_t *k_signs, const float *k_gamma,
                               int64_t n_blocks, int block_size, const int32_t *block_table,
                               int max_blocks_per_seq, const int32_t *seq_lens, float scale, float *scores,
                               int64_t max_len, void *stream);

/* Sizes: bytes of one packed index record, ceil(pw * bits / 8) with the
 * padded width pw = 4 g4 (Full, Fast) or 2 g2 (2-D); isoq_packed_bytes is
 * ceil(d * bits / 8), the same number whenever d is a multiple of 4.  Raw
 * draws per set for rot_host (Full 8 g4, Fast 4 g4, 2-D g2); exported
 * parameters per set (Full 8 g4, Fast 4 g4, 2-D 2 g2), with g4 = ceil(d/4),
 * g2 = ceil(d/2).  Return 0 for invalid arguments. */
size_t isoq_record_bytes(int variant, int d, int bits);
size_t isoq_packed_bytes(int d, int bits);
size_t isoq_raw_params_per_set(int variant, int d);
size_t isoq_export_params_per_set(int variant, int d);

/*
 * Host-only helpers (no device needed), the same computations init performs:
 *   isoq_codebook_lloyd   2^bits Lloyd-Max levels for N(0, 1/d) after `iters`
 *                         iterations (see isoq_params_init), as doubles.
 *   isoq_rotation_draws   the seeded raw draws init uses when rot_host is NULL,
 *                         n_sets * isoq_raw_params_per_set doubles.
 */
isoq_status isoq_codebook_lloyd(int bits, int d, int iters, double *levels_out);
isoq_status isoq_rotation_draws(int variant, int d, int n_sets, uint64_t seed, double *out);

/* Static text for a status code. */
const char *isoq_status_string(isoq_status s);

/* The HIP call and error text behind the last ISOQ_E_HIP (or a hipMalloc
 * ISOQ_E_NOMEM) returned on the calling thread; "" if none.  Valid until the
 * next call on the same thread. */
const char *isoq_last_hip_error(void);

#ifdef __cplusplus
}
#endif

#endif /* ISOQUANT_H */
