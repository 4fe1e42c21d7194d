/*
 * IsoQuant stage-1 oracle: a plain, slow, double-precision CPU model of the
 * quantize -> dequantize path of "IsoQuant: Hardware-Aligned SO(4) Isoclinic
 * Rotations for LLM KV Cache Compression" (arXiv 2603.28430).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may include, link or
 * call this file: only the test suite, the smoke check and the CPU-baseline leg
 * of the benchmark use it.  It shares no code, header, table or constant
 * generator with the HIP library; it is compiled by gcc on its own.
 *
 * Every routine follows the paper's definitions in the order the paper states
 * them.  There is no blocking, fusion or reordering.  All arithmetic is IEEE
 * double with contraction disabled (the build passes -ffp-contract=off).
 *
 * Readings where the paper is silent (each one is listed in the design notes):
 *   - quantizer Q: one scalar codebook of 2^b levels shared by all rotated
 *     coordinates; index = number of decision thresholds strictly below the
 *     value (a tie goes to the lower cell); thresholds are the midpoints of
 *     adjacent levels (nearest-level rule);
 *   - codebook: Lloyd iteration on the continuous density N(0, 1/d), started
 *     from levels evenly spaced on [-3 sigma, 3 sigma], then symmetrised;
 *   - epsilon in max(rho, eps) is 1e-12;
 *   - quaternion block i holds coordinates 4i..4i+3 with coordinate 4i the
 *     real part; the 2-D case pairs coordinates (2j, 2j+1);
 *   - Full evaluates (q_L v) conj(q_R) left to right (associative, Prop. 1);
 *   - raw rotation draws are normalised here, u / ||u||  (Sec. 5.5);
 *   - 8-D grouped blocks (the block-size axis of Table 3; Sec. 5.7 states the
 *     law of a Haar block rotation for any block size k): coordinates 8i..8i+7
 *     form block i, rotated by its own R_i ~ Haar(SO(8)).  A raw draw is an
 *     8x8 matrix G of i.i.d. N(0,1) entries; R_i is the orthogonal factor Q of
 *     G = QR with diag(R) > 0 (Haar on O(8)), with its first column negated
 *     when det Q = -1 (a fixed reflection maps that coset onto SO(8) and
 *     keeps the measure).
 *
 * Pins: every public function is checked in the CPU test suite against facts
 * that do not come from this file (defining relations of H, the textbook
 * rotation formula, orthogonality, Max's Lloyd-Max tables, library routines,
 * brute force, closed-form integrals, the counts of Table 1).
 */
#include <math.h>
#include <stddef.h>
#include <stdint.h>
#include <string.h>

#define ORC_FULL 0
#define ORC_FAST 1
#define ORC_PLANAR2D 2
#define ORC_BLOCK8 3

static const double ORC_EPS = 1e-12;

/* ---------------------------------------------------------------------------
 * Multiplication counter for the rotation arithmetic (Sec. 6, Table 1: one
 * quaternion product is counted as 16 multiply-adds).  Thread-local so that
 * row-parallel callers do not race.
 * ------------------------------------------------------------------------- */
static _Thread_local uint64_t orc_muls;

static double cmul(double a, double b)
{
    orc_muls++;
    return a * b;
}

uint64_t orc_mul_count(void) { return orc_muls; }
void orc_mul_count_reset(void) { orc_muls = 0; }

/* ---------------------------------------------------------------------------
 * Quaternion algebra (Sec. 4).  A quaternion is q[0] + q[1] i + q[2] j + q[3] k.
 * The product is expanded term by term from the basis rules
 * i^2 = j^2 = k^2 = ijk = -1, which give ij = k, jk = i, ki = j and
 * ji = -k, kj = -i, ik = -j.
 * ------------------------------------------------------------------------- */

/* basis product e_r * e_s = sign * e_index, basis order (1, i, j, k) */
static const int BASIS_INDEX[4][4] = {
    {0, 1, 2, 3}, /* 1*1=1   1*i=i   1*j=j   1*k=k  */
    {1, 0, 3, 2}, /* i*1=i   i*i=-1  i*j=k   i*k=-j */
    {2, 3, 0, 1}, /* j*1=j   j*i=-k  j*j=-1  j*k=i  */
    {3, 2, 1, 0}, /* k*1=k   k*i=j   k*j=-i  k*k=-1 */
};
static const int BASIS_SIGN[4][4] = {
    {+1, +1, +1, +1},
    {+1, -1, +1, -1},
    {+1, -1, -1, +1},
    {+1, +1, -1, -1},
};

/* out = p * q (Hamilton product): 16 scalar multiplications, 12 additions. */
void orc_qmul(const double p[4], const double q[4], double out[4])
{
    double acc[4] = {0.0, 0.0, 0.0, 0.0};
    for (int r = 0; r < 4; r++)
        for (int s = 0; s < 4; s++)
            acc[BASIS_INDEX[r][s]] += BASIS_SIGN[r][s] * cmul(p[r], q[s]);
    memcpy(out, acc, sizeof acc);
}

/* conj(q) = a - b i - c j - d k (Sec. 4). */
void orc_qconj(const double q[4], double out[4])
{
    out[0] = q[0];
    out[1] = -q[1];
    out[2] = -q[2];
    out[3] = -q[3];
}

/* q = u / ||u||_2 (Sec. 5.5, unconstrained vector normalised on the fly). */
void orc_qnormalize(const double u[4], double q[4])
{
    double n = sqrt(u[0] * u[0] + u[1] * u[1] + u[2] * u[2] + u[3] * u[3]);
    for (int c = 0; c < 4; c++)
        q[c] = u[c] / n;
}

/* ---------------------------------------------------------------------------
 * Block transforms (Sec. 5.2, 5.3, 5.4; inverse from Proposition 1).
 * ------------------------------------------------------------------------- */

/* IsoQuant-Full forward: T(v) = q_L v conj(q_R). */
void orc_full_forward(const double qL[4], const double qR[4], const double v[4], double out[4])
{
    double qRc[4], t[4];
    orc_qconj(qR, qRc);
    orc_qmul(qL, v, t);
    orc_qmul(t, qRc, out);
}

/* IsoQuant-Full inverse: T^-1(v) = conj(q_L) v q_R. */
void orc_full_inverse(const double qL[4], const double qR[4], const double v[4], double out[4])
{
    double qLc[4], t[4];
    orc_qconj(qL, qLc);
    orc_qmul(qLc, v, t);
    orc_qmul(t, qR, out);
}

/* IsoQuant-Fast forward: v -> q_L v. */
void orc_fast_forward(const double qL[4], const double v[4], double out[4])
{
    orc_qmul(qL, v, out);
}

/* IsoQuant-Fast inverse: v -> conj(q_L) v. */
void orc_fast_inverse(const double qL[4], const double v[4], double out[4])
{
    double qLc[4];
    orc_qconj(qL, qLc);
    orc_qmul(qLc, v, out);
}

/* 2-D case: u -> R(theta) u with R = [[cos, -sin], [sin, cos]]. */
void orc_planar_forward(double theta, const double u[2], double out[2])
{
    double c = cos(theta), s = sin(theta);
    out[0] = cmul(c, u[0]) - cmul(s, u[1]);
    out[1] = cmul(s, u[0]) + cmul(c, u[1]);
}

/* 2-D case inverse: u -> R(-theta) u. */
void orc_planar_inverse(double theta, const double u[2], double out[2])
{
    orc_planar_forward(-theta, u, out);
}

/* ---------------------------------------------------------------------------
 * 8-D grouped blocks (Table 3; Sec. 5.7 with k = 8).
 * ------------------------------------------------------------------------- */

/* Determinant of a row-major 8x8 matrix by Gaussian elimination with partial
 * pivoting (the product of the pivots, sign flipped once per row swap). */
double orc_det8(const double M[64])
{
    double a[8][8];
    for (int r = 0; r < 8; r++)
        for (int c = 0; c < 8; c++)
            a[r][c] = M[8 * r + c];
    double det = 1.0;
    for (int k = 0; k < 8; k++) {
        int piv = k;
        for (int r = k + 1; r < 8; r++)
            if (fabs(a[r][k]) > fabs(a[piv][k]))
                piv = r;
        if (a[piv][k] == 0.0)
            return 0.0;
        if (piv != k) {
            for (int c = 0; c < 8; c++) {
                double t = a[k][c];
                a[k][c] = a[piv][c];
                a[piv][c] = t;
            }
            det = -det;
        }
        det *= a[k][k];
        for (int r = k + 1; r < 8; r++) {
            double f = a[r][k] / a[k][k];
            for (int c = k; c < 8; c++)
                a[r][c] -= f * a[k][c];
        }
    }
    return det;
}

/*
 * The rotation of one 8-D block from its raw draw G (row-major 8x8): the
 * columns of G orthonormalised in order by Gram-Schmidt, which is the Q of
 * G = QR with a positive diagonal in R (each column loses its components along
 * the earlier ones, a second pass removing what rounding left, then is scaled
 * to unit length); then det Q = +1 by negating column 0 when it is -1.
 * Q is written row-major.  Returns 0, or -1 when the columns are linearly
 * dependent (a column left with less than 1e-12 of G's largest column norm
 * after the projections: rounding leaves that in place of 0).
 */
int orc_orthonormalize8(const double G[64], double Q[64])
{
    double col[8][8]; /* col[c][r] = entry (r, c) */
    double cmax = 0.0;
    for (int r = 0; r < 8; r++)
        for (int c = 0; c < 8; c++)
            col[c][r] = G[8 * r + c];
    for (int c = 0; c < 8; c++) {
        double ss = 0.0;
        for (int r = 0; r < 8; r++)
            ss += col[c][r] * col[c][r];
        if (sqrt(ss) > cmax)
            cmax = sqrt(ss);
    }
    for (int c = 0; c < 8; c++) {
        for (int pass = 0; pass < 2; pass++)
            for (int p = 0; p < c; p++) {
                double dot = 0.0;
                for (int r = 0; r < 8; r++)
                    dot += col[p][r] * col[c][r];
                for (int r = 0; r < 8; r++)
                    col[c][r] -= dot * col[p][r];
            }
        double ss = 0.0;
        for (int r = 0; r < 8; r++)
            ss += col[c][r] * col[c][r];
        double n = sqrt(ss);
        if (!(n > 1e-12 * cmax) || !isfinite(n))
            return -1;
        for (int r = 0; r < 8; r++)
            col[c][r] /= n;
    }
    for (int r = 0; r < 8; r++)
        for (int c = 0; c < 8; c++)
            Q[8 * r + c] = col[c][r];
    if (orc_det8(Q) < 0.0)
        for (int r = 0; r < 8; r++)
            Q[8 * r] = -Q[8 * r];
    return 0;
}

/* y = Q v for one 8-D block (64 multiplications, counted). */
void orc_block8_forward(const double G[64], const double v[8], double out[8])
{
    double Q[64];
    if (orc_orthonormalize8(G, Q) != 0) {
        for (int r = 0; r < 8; r++)
            out[r] = NAN;
        return;
    }
    for (int r = 0; r < 8; r++) {
        double acc = 0.0;
        for (int c = 0; c < 8; c++)
            acc += cmul(Q[8 * r + c], v[c]);
        out[r] = acc;
    }
}

/* v = Q^T y, the inverse of a block rotation (Q is orthogonal). */
void orc_block8_inverse(const double G[64], const double y[8], double out[8])
{
    double Q[64];
    if (orc_orthonormalize8(G, Q) != 0) {
        for (int c = 0; c < 8; c++)
            out[c] = NAN;
        return;
    }
    for (int c = 0; c < 8; c++) {
        double acc = 0.0;
        for (int r = 0; r < 8; r++)
            acc += cmul(Q[8 * r + c], y[r]);
        out[c] = acc;
    }
}

/* ---------------------------------------------------------------------------
 * Scalar Lloyd-Max quantizer Q (Sec. 1 and 7.2 name it; fit procedure is the
 * reading stated in the header).
 * ------------------------------------------------------------------------- */

static double std_pdf(double z) { return exp(-0.5 * z * z) / sqrt(2.0 * M_PI); }

/* P(a < Z <= b) for Z ~ N(0,1), computed with erfc to keep tail cells exact. */
static double std_mass(double a, double b)
{
    /* Phi(z) = erfc(-z / sqrt 2) / 2 */
    double pa = isinf(a) ? 0.0 : 0.5 * erfc(-a / M_SQRT2);
    double pb = isinf(b) ? 1.0 : 0.5 * erfc(-b / M_SQRT2);
    if (a > 0.0) {
        /* upper tail: use the complementary form to avoid cancellation */
        double qa = 0.5 * erfc(a / M_SQRT2);
        double qb = isinf(b) ? 0.0 : 0.5 * erfc(b / M_SQRT2);
        return qa - qb;
    }
    return pb - pa;
}

/* Decision thresholds of the nearest-level rule: t_k = (c_k + c_{k+1}) / 2. */
void orc_thresholds(int bits, const double *levels, double *thr)
{
    int K = 1 << bits;
    for (int k = 0; k + 1 < K; k++)
        thr[k] = 0.5 * (levels[k] + levels[k + 1]);
}

/*
 * Lloyd iteration for N(0, sigma^2): alternate the nearest-level partition
 * (midpoint thresholds) and the centroid condition
 *     c_k = E[X | t_{k-1} < X <= t_k]
 *         = sigma * (pdf(a) - pdf(b)) / (Phi(b) - Phi(a)),  a = t_{k-1}/sigma, b = t_k/sigma,
 * with t_{-1} = -inf and t_{K-1} = +inf.  Returns 0 on success.
 */
int orc_lloyd_max_gaussian(int bits, double sigma, int iters, double *levels)
{
    if (bits < 1 || bits > 8 || !(sigma > 0.0) || iters < 0)
        return -1;
    int K = 1 << bits;
    double z[256], t[257];
    for (int k = 0; k < K; k++)
        z[k] = (K == 1) ? 0.0 : -3.0 + 6.0 * (double)k / (double)(K - 1);
    for (int it = 0; it < iters; it++) {
        t[0] = -INFINITY;
        for (int k = 1; k < K; k++)
            t[k] = 0.5 * (z[k - 1] + z[k]);
        t[K] = INFINITY;
        for (int k = 0; k < K; k++) {
            double a = t[k], b = t[k + 1];
            double pa = isinf(a) ? 0.0 : std_pdf(a);
            double pb = isinf(b) ? 0.0 : std_pdf(b);
            z[k] = (pa - pb) / std_mass(a, b);
        }
    }
    /* the density is symmetric, so the optimal codebook is: enforce it */
    for (int k = 0; k < K / 2; k++) {
        double m = 0.5 * (z[K - 1 - k] - z[k]);
        z[k] = -m;
        z[K - 1 - k] = m;
    }
    for (int k = 0; k < K; k++)
        levels[k] = sigma * z[k];
    return 0;
}

/* Q: index = #{k : y > t_k}; value = c[index]. */
static int quantize_index(int bits, const double *thr, double y)
{
    int K = 1 << bits, idx = 0;
    for (int k = 0; k + 1 < K; k++)
        if (y > thr[k])
            idx++;
    return idx;
}

/* ---------------------------------------------------------------------------
 * Geometry of the partition (Sec. 4.1, Sec. 5.1, Sec. 6).
 * ------------------------------------------------------------------------- */

/* number of local blocks: g4 = ceil(d/4) for Full/Fast, g2 = ceil(d/2) for 2-D,
 * g8 = ceil(d/8) for 8-D blocks */
int orc_num_blocks(int variant, int d)
{
    return variant == ORC_PLANAR2D ? (d + 1) / 2 : variant == ORC_BLOCK8 ? (d + 7) / 8 : (d + 3) / 4;
}

/* raw parameters per set: Full 8 g4 (u_L, u_R), Fast 4 g4 (u_L), 2-D g2 angles,
 * 8-D 64 g8 (one raw 8x8 matrix per block) */
int orc_raw_params_per_set(int variant, int d)
{
    int g = orc_num_blocks(variant, d);
    return variant == ORC_FULL ? 8 * g : variant == ORC_FAST ? 4 * g : variant == ORC_BLOCK8 ? 64 * g : g;
}

/* rotation parameters counted as in Table 1: 8 g4 / 4 g4 / 2 g2 (cos, sin);
 * 8-D blocks (not in Table 1) store their 64 matrix entries per block */
int orc_table1_params(int variant, int d)
{
    int g = orc_num_blocks(variant, d);
    return variant == ORC_FULL ? 8 * g : variant == ORC_FAST ? 4 * g : variant == ORC_BLOCK8 ? 64 * g : 2 * g;
}

/* ---------------------------------------------------------------------------
 * Encoder / decoder transforms on a whole normalised vector (Sec. 5.1: the
 * block-diagonal element of (SO(4))^g, of (SO(2))^g2 or of (SO(8))^g8, applied block by
 * block on the zero-padded vector).  `pad` holds blk*g coordinates.
 * ------------------------------------------------------------------------- */
static void block_forward(int variant, const double *rot, int i, const double *vin, double *vout)
{
    if (variant == ORC_FULL) {
        double qL[4], qR[4];
        orc_qnormalize(rot + 8 * i, qL);
        orc_qnormalize(rot + 8 * i + 4, qR);
        orc_full_forward(qL, qR, vin, vout);
    } else if (variant == ORC_FAST) {
        double qL[4];
        orc_qnormalize(rot + 4 * i, qL);
        orc_fast_forward(qL, vin, vout);
    } else if (variant == ORC_BLOCK8) {
        orc_block8_forward(rot + 64 * i, vin, vout);
    } else {
        orc_planar_forward(rot[i], vin, vout);
    }
}

static void block_inverse(int variant, const double *rot, int i, const double *vin, double *vout)
{
    if (variant == ORC_FULL) {
        double qL[4], qR[4];
        orc_qnormalize(rot + 8 * i, qL);
        orc_qnormalize(rot + 8 * i + 4, qR);
        orc_full_inverse(qL, qR, vin, vout);
    } else if (variant == ORC_FAST) {
        double qL[4];
        orc_qnormalize(rot + 4 * i, qL);
        orc_fast_inverse(qL, vin, vout);
    } else if (variant == ORC_BLOCK8) {
        orc_block8_inverse(rot + 64 * i, vin, vout);
    } else {
        orc_planar_inverse(rot[i], vin, vout);
    }
}

static int block_width(int variant) { return variant == ORC_PLANAR2D ? 2 : variant == ORC_BLOCK8 ? 8 : 4; }

/*
 * Encoder E on one normalised vector: out[0 .. blk*g) = blockwise rotation of
 * the zero-padded input.  Multiplications are counted (Table 1 pin).
 */
void orc_encode(int variant, int d, const double *rot, const double *xbar, double *out)
{
    int blk = block_width(variant), g = orc_num_blocks(variant, d);
    for (int i = 0; i < g; i++) {
        double v[8] = {0, 0, 0, 0, 0, 0, 0, 0};
        for (int c = 0; c < blk; c++)
            v[c] = (blk * i + c < d) ? xbar[blk * i + c] : 0.0;
        block_forward(variant, rot, i, v, out + blk * i);
    }
}

/* Decoder: inverse block rotations of the padded vector, padding dropped. */
void orc_decode(int variant, int d, const double *rot, const double *yhat, double *rec)
{
    int blk = block_width(variant), g = orc_num_blocks(variant, d);
    for (int i = 0; i < g; i++) {
        double r[8];
        block_inverse(variant, rot, i, yhat + blk * i, r);
        for (int c = 0; c < blk; c++)
            if (blk * i + c < d)
                rec[blk * i + c] = r[c];
    }
}

static int64_t set_of_row(int64_t row, int n_sets, int64_t rows_per_set)
{
    if (n_sets <= 1)
        return 0;
    return (row / rows_per_set) % n_sets;
}

/* ---------------------------------------------------------------------------
 * Algorithm 1 (stage-1 quantization) for rows [row_begin, row_end) of x.
 *   x      : [n][d] input rows (row r at x + r*d)
 *   rot    : raw draws, [n_sets][orc_raw_params_per_set]
 *   levels : 2^bits codebook, ascending
 * Outputs (each may be NULL):
 *   idx    : [n][pg] codebook index per rotated coordinate, pg = blk*g (padded)
 *   rho    : [n] norms
 *   xhat   : [n][d] reconstruction
 * The set of row r is (r / rows_per_set) mod n_sets.
 * ------------------------------------------------------------------------- */
static int stage1_args_ok(int variant, int d, int bits, int n_sets, int64_t rows_per_set)
{
    return !(variant < 0 || variant > 3 || d < 1 || d > 4096 || bits < 1 || bits > 8 || n_sets < 1 ||
             (n_sets > 1 && rows_per_set < 1));
}

/* Algorithm 1 on one row.  xr: d inputs; rs: raw draws of the row's set;
 * outputs idx_row[pg], *rho_out, xhat_row[d] and the rotated normalised
 * coordinates ytil_row[pg] (each may be NULL). */
static void stage1_row(int variant, int d, int bits, const double *rs, const double *levels,
                       const double *thr, const double *xr, uint8_t *idx_row, double *rho_out,
                       double *xhat_row, double *ytil_row)
{
    int blk = block_width(variant), g = orc_num_blocks(variant, d), pg = blk * g;
    double xbar[4096], ytil[4100], yhat[4100], rec[4096];
    /* step: norm and direction (Sec. 3) */
    double ss = 0.0;
    for (int j = 0; j < d; j++)
        ss += xr[j] * xr[j];
    double p = sqrt(ss);
    double den = p > ORC_EPS ? p : ORC_EPS;
    for (int j = 0; j < d; j++)
        xbar[j] = xr[j] / den;
    /* steps: partition into zero-padded blocks and rotate each block */
    orc_encode(variant, d, rs, xbar, ytil);
    if (ytil_row)
        memcpy(ytil_row, ytil, sizeof(double) * (size_t)pg);
    /* step: coordinate-wise scalar quantization in the rotated basis */
    for (int j = 0; j < pg; j++) {
        int q = quantize_index(bits, thr, ytil[j]);
        if (idx_row)
            idx_row[j] = (uint8_t)q;
        yhat[j] = levels[q];
    }
    /* steps: inverse rotation, concatenation, padding dropped, norm restored */
    orc_decode(variant, d, rs, yhat, rec);
    if (rho_out)
        *rho_out = p;
    if (xhat_row)
        for (int j = 0; j < d; j++)
            xhat_row[j] = p * rec[j];
}

/* ---------------------------------------------------------------------------
 * Algorithm 1 (stage-1 quantization) for rows [row_begin, row_end) of x.
 *   x      : [n][d] input rows (row r at x + r*d)
 *   rot    : raw draws, [n_sets][orc_raw_params_per_set]
 *   levels : 2^bits codebook, ascending
 * Outputs (each may be NULL), indexed by row number:
 *   idx    : [n][pg] codebook index per rotated coordinate, pg = blk*g (padded)
 *   rho    : [n] norms
 *   xhat   : [n][d] reconstruction
 *   ytil   : [n][pg] rotated coordinates of the normalised row (before Q)
 * The set of row r is (r / rows_per_set) mod n_sets.
 * ------------------------------------------------------------------------- */
int orc_stage1(int variant, int d, int bits, int n_sets, int64_t rows_per_set,
               const double *rot, const double *levels, const double *x,
               int64_t row_begin, int64_t row_end,
               uint8_t *idx, double *rho, double *xhat, double *ytil)
{
    if (!stage1_args_ok(variant, d, bits, n_sets, rows_per_set))
        return -1;
    int pg = block_width(variant) * orc_num_blocks(variant, d);
    int rp = orc_raw_params_per_set(variant, d);
    double thr[255];
    orc_thresholds(bits, levels, thr);
    for (int64_t r = row_begin; r < row_end; r++)
        stage1_row(variant, d, bits, rot + set_of_row(r, n_sets, rows_per_set) * rp, levels, thr,
                   x + r * d, idx ? idx + r * pg : NULL, rho ? rho + r : NULL,
                   xhat ? xhat + r * d : NULL, ytil ? ytil + r * pg : NULL);
    return 0;
}

/* Same as orc_stage1 for m selected rows: xs[t] is the input row whose global
 * row number is rows[t]; outputs are written at position t. */
int orc_stage1_rows(int variant, int d, int bits, int n_sets, int64_t rows_per_set,
                    const double *rot, const double *levels, const int64_t *rows, int64_t m,
                    const double *xs, uint8_t *idx, double *rho, double *xhat, double *ytil)
{
    if (!stage1_args_ok(variant, d, bits, n_sets, rows_per_set))
        return -1;
    int pg = block_width(variant) * orc_num_blocks(variant, d);
    int rp = orc_raw_params_per_set(variant, d);
    double thr[255];
    orc_thresholds(bits, levels, thr);
    for (int64_t t = 0; t < m; t++)
        stage1_row(variant, d, bits, rot + set_of_row(rows[t], n_sets, rows_per_set) * rp, levels,
                   thr, xs + t * d, idx ? idx + t * pg : NULL, rho ? rho + t : NULL,
                   xhat ? xhat + t * d : NULL, ytil ? ytil + t * pg : NULL);
    return 0;
}

/* Dequantize rows [row_begin, row_end) from indices and norms (the decoder
 * half of Algorithm 1). */
int orc_dequantize(int variant, int d, int bits, int n_sets, int64_t rows_per_set,
                   const double *rot, const double *levels, const uint8_t *idx, const double *rho,
                   int64_t row_begin, int64_t row_end, double *xhat)
{
    if (!stage1_args_ok(variant, d, bits, n_sets, rows_per_set))
        return -1;
    int K = 1 << bits;
    int blk = block_width(variant), g = orc_num_blocks(variant, d), pg = blk * g;
    int rp = orc_raw_params_per_set(variant, d);
    double yhat[4100], rec[4096];
    for (int64_t r = row_begin; r < row_end; r++) {
        const double *rs = rot + set_of_row(r, n_sets, rows_per_set) * rp;
        for (int j = 0; j < pg; j++) {
            int q = idx[r * pg + j];
            if (q >= K)
                return -2;
            yhat[j] = levels[q];
        }
        orc_decode(variant, d, rs, yhat, rec);
        for (int j = 0; j < d; j++)
            xhat[r * d + j] = rho[r] * rec[j];
    }
    return 0;
}

/* ---------------------------------------------------------------------------
 * Packed index record (reading: the paper only says indices are b-bit).
 * Row r occupies bytes [r*rb, (r+1)*rb), rb = ceil(m*bits/8) for m indices per
 * row; index j occupies bits [j*bits, (j+1)*bits) of the record, bit n being
 * bit (n mod 8) of byte floor(n/8) (least significant bit first).
 * ------------------------------------------------------------------------- */
int64_t orc_record_bytes(int m, int bits) { return ((int64_t)m * bits + 7) / 8; }

void orc_pack(const uint8_t *idx, int64_t n, int m, int bits, uint8_t *out)
{
    int64_t rb = orc_record_bytes(m, bits);
    memset(out, 0, (size_t)(n * rb));
    for (int64_t r = 0; r < n; r++)
        for (int j = 0; j < m; j++)
            for (int t = 0; t < bits; t++) {
                int64_t bit = (int64_t)j * bits + t;
                if ((idx[r * m + j] >> t) & 1)
                    out[r * rb + bit / 8] |= (uint8_t)(1u << (bit % 8));
            }
}

void orc_unpack(const uint8_t *in, int64_t n, int m, int bits, uint8_t *idx)
{
    int64_t rb = orc_record_bytes(m, bits);
    for (int64_t r = 0; r < n; r++)
        for (int j = 0; j < m; j++) {
            int v = 0;
            for (int t = 0; t < bits; t++) {
                int64_t bit = (int64_t)j * bits + t;
                v |= ((in[r * rb + bit / 8] >> (bit % 8)) & 1) << t;
            }
            idx[r * m + j] = (uint8_t)v;
        }
}
