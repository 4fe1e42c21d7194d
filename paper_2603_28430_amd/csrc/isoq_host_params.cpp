// Host-side construction of the quantizer state: Lloyd-Max codebook, seeded
// rotation draws, normalisation (Sec. 5.5) and the per-lane device layout.
// All of it runs once, at isoq_params_init, in double precision.
#include <algorithm>
#include <cmath>
#include <cstring>

#include "isoq_internal.h"

namespace isoq {

// ---------------------------------------------------------------- codebook
// Lloyd's fixed-point iteration for a Gaussian source N(0, sigma^2), in units
// of sigma: the decision points are the midpoints of neighbouring levels, and
// each level moves to the conditional mean of its cell,
//   E[Z | a < Z <= b] = (phi(a) - phi(b)) / (Phi(b) - Phi(a)).
// Start: levels evenly spaced on [-3, 3].  The source is symmetric, so the
// result is made exactly odd before scaling.
namespace {
double gauss_pdf(double z) { return std::exp(-0.5 * z * z) * 0.39894228040143267794; }

// P(Z > z) with Z ~ N(0,1); +inf and -inf handled
double gauss_sf(double z)
{
    if (std::isinf(z))
        return z > 0 ? 0.0 : 1.0;
    return 0.5 * std::erfc(z * 0.70710678118654752440);
}
}  // namespace

bool lloyd_levels(int bits, double sigma, int iters, double *levels)
{
    if (bits < 1 || bits > 4 || !(sigma > 0) || iters < 0)
        return false;
    const int K = 1 << bits;
    double c[16], edge[17];
    for (int k = 0; k < K; k++)
        c[k] = K > 1 ? 6.0 * k / (K - 1) - 3.0 : 0.0;
    for (int it = 0; it < iters; it++) {
        edge[0] = -INFINITY;
        edge[K] = INFINITY;
        for (int k = 1; k < K; k++)
            edge[k] = 0.5 * (c[k - 1] + c[k]);
        for (int k = 0; k < K; k++) {
            const double lo = edge[k], hi = edge[k + 1];
            const double num = (std::isinf(lo) ? 0.0 : gauss_pdf(lo)) - (std::isinf(hi) ? 0.0 : gauss_pdf(hi));
            // mass of the cell from the side whose tail is smaller
            const double mass = lo >= 0 ? gauss_sf(lo) - gauss_sf(hi) : gauss_sf(-hi) - gauss_sf(-lo);
            c[k] = num / mass;
        }
    }
    for (int k = 0; k < K / 2; k++) {
        const double m = 0.5 * (c[K - 1 - k] - c[k]);
        c[k] = -m;
        c[K - 1 - k] = m;
    }
    for (int k = 0; k < K; k++)
        levels[k] = sigma * c[k];
    return true;
}

// ------------------------------------------------------------ rotation draws
size_t raw_per_set(int variant, int d)
{
    if (variant == VAR_PLANAR2D)
        return (size_t)(d + 1) / 2;
    if (variant == VAR_BLOCK8)
        return 64 * ((size_t)(d + 7) / 8);
    const size_t g = (size_t)(d + 3) / 4;
    return variant == VAR_FULL ? 8 * g : 4 * g;
}

size_t export_per_set(int variant, int d)
{
    if (variant == VAR_PLANAR2D)
        return 2 * ((size_t)(d + 1) / 2);
    if (variant == VAR_BLOCK8)
        return 64 * ((size_t)(d + 7) / 8);
    const size_t g = (size_t)(d + 3) / 4;
    return variant == VAR_FULL ? 8 * g : 4 * g;
}

namespace {
// Philox4x32-10 (Salmon et al., SC 2011): ten rounds of two 32x32->64-bit
// multiplications, with the Weyl key schedule between rounds.
void philox4x32_10(uint32_t ctr[4], uint32_t k0, uint32_t k1)
{
    for (int round = 0; round < 10; round++) {
        if (round > 0) {
            k0 += 0x9E3779B9u;
            k1 += 0xBB67AE85u;
        }
        const uint64_t p0 = (uint64_t)0xD2511F53u * ctr[0];
        const uint64_t p1 = (uint64_t)0xCD9E8D57u * ctr[2];
        const uint32_t n0 = (uint32_t)(p1 >> 32) ^ ctr[1] ^ k0;
        const uint32_t n1 = (uint32_t)p1;
        const uint32_t n2 = (uint32_t)(p0 >> 32) ^ ctr[3] ^ k1;
        const uint32_t n3 = (uint32_t)p0;
        ctr[0] = n0;
        ctr[1] = n1;
        ctr[2] = n2;
        ctr[3] = n3;
    }
}

void normal_pair(uint32_t a, uint32_t b, double *z)
{
    const double two_pi = 6.283185307179586476925;
    const double u1 = ((double)a + 0.5) * 0x1p-32;
    const double u2 = (double)b * 0x1p-32;
    const double r = std::sqrt(-2.0 * std::log(u1));
    z[0] = r * std::cos(two_pi * u2);
    z[1] = r * std::sin(two_pi * u2);
}
}  // namespace

void seeded_draws(int variant, int d, int n_sets, uint64_t seed, double *out)
{
    const uint32_t k0 = (uint32_t)seed, k1 = (uint32_t)(seed >> 32);
    size_t o = 0;
    if (variant == VAR_PLANAR2D) {
        const int g2 = (d + 1) / 2;
        for (int s = 0; s < n_sets; s++)
            for (int j = 0; j < g2; j++) {
                uint32_t c[4] = {(uint32_t)j, (uint32_t)s, 2u, 0u};
                philox4x32_10(c, k0, k1);
                out[o++] = 6.283185307179586476925 * ((double)c[0] * 0x1p-32);
            }
        return;
    }
    if (variant == VAR_BLOCK8) {
        // raw 8x8 matrix of block i, row-major: entries 4q .. 4q + 3 from
        // counter (i, set, 4, q)
        const int g8 = (d + 7) / 8;
        for (int s = 0; s < n_sets; s++)
            for (int i = 0; i < g8; i++)
                for (int q = 0; q < 16; q++) {
                    uint32_t c[4] = {(uint32_t)i, (uint32_t)s, 4u, (uint32_t)q};
                    philox4x32_10(c, k0, k1);
                    normal_pair(c[0], c[1], out + o);
                    normal_pair(c[2], c[3], out + o + 2);
                    o += 4;
                }
        return;
    }
    const int g = (d + 3) / 4;
    const int sides = variant == VAR_FULL ? 2 : 1;
    for (int s = 0; s < n_sets; s++)
        for (int i = 0; i < g; i++)
            for (int side = 0; side < sides; side++) {
                uint32_t c[4] = {(uint32_t)i, (uint32_t)s, (uint32_t)side, 0u};
                philox4x32_10(c, k0, k1);
                normal_pair(c[0], c[1], out + o);
                normal_pair(c[2], c[3], out + o + 2);
                o += 4;
            }
}

// --------------------------------------------------- normalisation and layout
namespace {
// Hamilton product, written out from ij = k, jk = i, ki = j (i^2 = j^2 = k^2 = -1).
void hamilton(const double p[4], const double q[4], double r[4])
{
    r[0] = p[0] * q[0] - p[1] * q[1] - p[2] * q[2] - p[3] * q[3];
    r[1] = p[0] * q[1] + p[1] * q[0] + p[2] * q[3] - p[3] * q[2];
    r[2] = p[0] * q[2] - p[1] * q[3] + p[2] * q[0] + p[3] * q[1];
    r[3] = p[0] * q[3] + p[1] * q[2] - p[2] * q[1] + p[3] * q[0];
}

bool unit4(const double *u, double q[4])
{
    const double n = std::sqrt(u[0] * u[0] + u[1] * u[1] + u[2] * u[2] + u[3] * u[3]);
    if (!(n > 0) || !std::isfinite(n))
        return false;
    for (int c = 0; c < 4; c++)
        q[c] = u[c] / n;
    return true;
}

// The rotation of an 8-D block from its raw draw G (row-major 8x8): the
// orthogonal factor Q of G = QR with a positive diagonal in R, by Householder
// reflections (Golub and Van Loan, Matrix Computations, Sec. 5.2.2): H_k
// zeroes column k of the working matrix below the diagonal, Q = H_0 ... H_6,
// then column k of Q is negated wherever R_kk < 0.  det Q is -1 to the power
// (reflections + negated columns); when it is -1, column 0 is negated once
// more, which puts Q in SO(8).  False when G's columns are dependent (an R_kk
// below 1e-12 of G's largest column norm, which rounding leaves in place of 0).
bool haar_so8(const double *G, double Q[64])
{
    double A[8][8], W[8][8], cmax = 0;
    for (int r = 0; r < 8; r++)
        for (int c = 0; c < 8; c++) {
            A[r][c] = G[8 * r + c];
            W[r][c] = r == c ? 1.0 : 0.0;
            if (!std::isfinite(A[r][c]))
                return false;
        }
    for (int c = 0; c < 8; c++) {
        double n = 0;
        for (int r = 0; r < 8; r++)
            n += A[r][c] * A[r][c];
        cmax = std::max(cmax, std::sqrt(n));
    }
    if (!(cmax > 0))
        return false;
    int flips = 0;
    for (int k = 0; k < 7; k++) {
        double nx = 0;
        for (int r = k; r < 8; r++)
            nx += A[r][k] * A[r][k];
        nx = std::sqrt(nx);
        if (!(nx > 0))
            return false;
        // v = x - alpha e_k with alpha = -sign(x_k) ||x|| (no cancellation)
        const double alpha = A[k][k] >= 0 ? -nx : nx;
        double v[8] = {0, 0, 0, 0, 0, 0, 0, 0};
        for (int r = k; r < 8; r++)
            v[r] = A[r][k];
        v[k] -= alpha;
        double vv = 0;
        for (int r = k; r < 8; r++)
            vv += v[r] * v[r];
        // A <- H A on columns k.., W <- W H (W accumulates Q)
        for (int c = k; c < 8; c++) {
            double t = 0;
            for (int r = k; r < 8; r++)
                t += v[r] * A[r][c];
            t *= 2.0 / vv;
            for (int r = k; r < 8; r++)
                A[r][c] -= t * v[r];
        }
        for (int r = 0; r < 8; r++) {
            double t = 0;
            for (int c = k; c < 8; c++)
                t += W[r][c] * v[c];
            t *= 2.0 / vv;
            for (int c = k; c < 8; c++)
                W[r][c] -= t * v[c];
        }
        flips++;   // det H_k = -1
    }
    for (int k = 0; k < 8; k++) {
        if (!(std::fabs(A[k][k]) > 1e-12 * cmax) || !std::isfinite(A[k][k]))
            return false;
        if (A[k][k] < 0) {
            for (int r = 0; r < 8; r++)
                W[r][k] = -W[r][k];
            flips++;
        }
    }
    if (flips & 1)
        for (int r = 0; r < 8; r++)
            W[r][0] = -W[r][0];
    for (int r = 0; r < 8; r++)
        for (int c = 0; c < 8; c++)
            Q[8 * r + c] = W[r][c];
    return true;
}
}  // namespace

void seeded_projection(int m, int d, uint64_t seed, double *out)
{
    const uint32_t k0 = (uint32_t)seed, k1 = (uint32_t)(seed >> 32);
    const int g4 = (d + 3) / 4;
    for (int i = 0; i < m; i++)
        for (int g = 0; g < g4; g++) {
            uint32_t c[4] = {(uint32_t)g, (uint32_t)i, 3u, 0u};
            philox4x32_10(c, k0, k1);
            double z[4];
            normal_pair(c[0], c[1], z);
            normal_pair(c[2], c[3], z + 2);
            for (int k = 0; k < 4 && 4 * g + k < d; k++)
                out[(size_t)i * d + 4 * g + k] = z[k];
        }
}

void rotate_rows_forward(int variant, int d, const float *unit_set, const double *in, int rows, double *out)
{
    for (int r = 0; r < rows; r++) {
        const double *v = in + (size_t)r * d;
        double *y = out + (size_t)r * d;
        if (variant == VAR_BLOCK8) {
            for (int i = 0; i < d / 8; i++)
                for (int a = 0; a < 8; a++) {
                    double acc = 0;
                    for (int c = 0; c < 8; c++)
                        acc += (double)unit_set[64 * i + 8 * a + c] * v[8 * i + c];
                    y[8 * i + a] = acc;
                }
            continue;
        }
        if (variant == VAR_PLANAR2D) {
            for (int j = 0; j < d / 2; j++) {
                const double c = unit_set[2 * j], sn = unit_set[2 * j + 1];
                y[2 * j] = c * v[2 * j] - sn * v[2 * j + 1];
                y[2 * j + 1] = sn * v[2 * j] + c * v[2 * j + 1];
            }
            continue;
        }
        for (int i = 0; i < d / 4; i++) {
            const float *q = unit_set + (variant == VAR_FULL ? 8 : 4) * i;
            const double qL[4] = {q[0], q[1], q[2], q[3]};
            double t[4];
            hamilton(qL, v + 4 * i, t);
            if (variant == VAR_FULL) {
                const double qRc[4] = {q[4], -q[5], -q[6], -q[7]};
                hamilton(t, qRc, y + 4 * i);
            } else {
                for (int k = 0; k < 4; k++)
                    y[4 * i + k] = t[k];
            }
        }
    }
}

bool build_rotation(int variant, int d, int n_sets, const double *raw, std::vector<float> &exported,
                    std::vector<float> &device_layout)
{
    // device layout: per set, slots_per_set slots of params_per_slot floats
    // (a lane of the tuned kernels owns two consecutive slots)
    const size_t per_set = (size_t)slots_per_set(variant, d) * params_per_slot(variant);
    const size_t rp = raw_per_set(variant, d);
    exported.assign((size_t)n_sets * export_per_set(variant, d), 0.f);
    device_layout.assign((size_t)n_sets * per_set, 0.f);
    for (int s = 0; s < n_sets; s++) {
        const double *rs = raw + s * rp;
        float *ex = exported.data() + s * export_per_set(variant, d);
        float *dv = device_layout.data() + (size_t)s * per_set;
        if (variant == VAR_PLANAR2D) {
            // slot l holds pairs 2l and 2l+1: (cos, sin) each
            const int g2 = (d + 1) / 2;
            for (int j = 0; j < g2; j++) {
                if (!std::isfinite(rs[j]))
                    return false;
                const double c = std::cos(rs[j]), sn = std::sin(rs[j]);
                ex[2 * j] = (float)c;
                ex[2 * j + 1] = (float)sn;
                dv[2 * j] = (float)c;
                dv[2 * j + 1] = (float)sn;
            }
            if (g2 & 1)
                dv[2 * g2] = 1.f;   // identity for the pair past the padded width
            continue;
        }
        if (variant == VAR_BLOCK8) {
            // exported and device layouts alike: Q of each block, row-major
            const int g8 = (d + 7) / 8;
            for (int i = 0; i < g8; i++) {
                double Q[64];
                if (!haar_so8(rs + 64 * i, Q))
                    return false;
                for (int k = 0; k < 64; k++) {
                    ex[64 * i + k] = (float)Q[k];
                    dv[64 * i + k] = (float)Q[k];
                }
            }
            continue;
        }
        const int g = (d + 3) / 4;
        for (int i = 0; i < g; i++) {
            double qL[4], qR[4] = {1, 0, 0, 0};
            if (!unit4(rs + (variant == VAR_FULL ? 8 : 4) * i, qL))
                return false;
            if (variant == VAR_FULL && !unit4(rs + 8 * i + 4, qR))
                return false;
            if (variant == VAR_FAST) {
                for (int c = 0; c < 4; c++) {
                    ex[4 * i + c] = (float)qL[c];
                    dv[4 * i + c] = (float)qL[c];
                }
                continue;
            }
            for (int c = 0; c < 4; c++) {
                ex[8 * i + c] = (float)qL[c];
                ex[8 * i + 4 + c] = (float)qR[c];
            }
            // M = matrix of v -> q_L v conj(q_R): column c is the image of e_c
            const double qRc[4] = {qR[0], -qR[1], -qR[2], -qR[3]};
            double M[4][4];
            for (int c = 0; c < 4; c++) {
                double e[4] = {0, 0, 0, 0}, t[4], col[4];
                e[c] = 1.0;
                hamilton(qL, e, t);
                hamilton(t, qRc, col);
                for (int r = 0; r < 4; r++)
                    M[r][c] = col[r];
            }
            for (int r = 0; r < 4; r++)
                for (int c = 0; c < 4; c++)
                    dv[16 * i + 4 * r + c] = (float)M[r][c];
        }
    }
    return true;
}

// ------------------------------------------------- matrix-core parameters
// For the quad-layout encoders: per chunk c (coordinates 8c .. 8c+7) and quad
// row i, row i of each 4x4 matrix the chunk's rotation applies, as fp16 hi =
// fp16(m) and lo = fp16(m - hi) (their sum is m to about 2^-22 relative):
// Full, Fast, 2-D: the matrices of slots 2c and 2c+1 (M = L(q_L) R(conj q_R),
// L(q_L), diag(R(theta_1), R(theta_2))); 8-D: the sub-blocks (0,0), (0,1),
// (1,0), (1,1) of the block's 8x8 Q.  Each row is 16 bytes: hi[4], lo[4].
namespace {
void put_row(const float m[4], uint16_t *out)
{
    for (int k = 0; k < 4; k++) {
        const _Float16 hi = (_Float16)m[k];
        const _Float16 lo = (_Float16)(m[k] - (float)hi);
        std::memcpy(out + k, &hi, 2);
        std::memcpy(out + 4 + k, &lo, 2);
    }
}

// the 4x4 matrix (row-major) a tuned kernel applies to slot j of a set
void slot_matrix(int variant, const float *set_layout, int j, float M[16])
{
    const float *P = set_layout + (size_t)j * params_per_slot(variant);
    if (variant == VAR_FULL) {
        for (int k = 0; k < 16; k++)
            M[k] = P[k];
    } else if (variant == VAR_FAST) {
        const float a = P[0], b = P[1], c = P[2], d = P[3];
        const float L[16] = {a, -b, -c, -d, b, a, -d, c, c, d, a, -b, d, -c, b, a};
        for (int k = 0; k < 16; k++)
            M[k] = L[k];
    } else {
        const float c1 = P[0], s1 = P[1], c2 = P[2], s2 = P[3];
        const float R[16] = {c1, -s1, 0, 0, s1, c1, 0, 0, 0, 0, c2, -s2, 0, 0, s2, c2};
        for (int k = 0; k < 16; k++)
            M[k] = R[k];
    }
}
}  // namespace

void build_mfma_params(int variant, int d, const float *set_layout, uint16_t *out)
{
    const int C = d / 8, pieces = variant == VAR_BLOCK8 ? 4 : 2;
    for (int c = 0; c < C; c++)
        for (int i = 0; i < 4; i++) {
            uint16_t *o = out + ((size_t)c * 4 + i) * pieces * 8;
            if (variant == VAR_BLOCK8) {
                const float *Q = set_layout + (size_t)c * 64;
                for (int s = 0; s < 2; s++)
                    for (int t = 0; t < 2; t++) {
                        const float row[4] = {Q[8 * (4 * s + i) + 4 * t], Q[8 * (4 * s + i) + 4 * t + 1],
                                              Q[8 * (4 * s + i) + 4 * t + 2], Q[8 * (4 * s + i) + 4 * t + 3]};
                        put_row(row, o + (2 * s + t) * 8);
                    }
            } else {
                for (int t = 0; t < 2; t++) {
                    float M[16];
                    slot_matrix(variant, set_layout, 2 * c + t, M);
                    put_row(M + 4 * i, o + t * 8);
                }
            }
        }
}

// ------------------------------------------------------- magnitude lookup table
bool build_magnitude_lut(int H, const double *tau, const double *lev, double *inv_h,
                         std::vector<LutEntry> &lut)
{
    double gap = tau[0];
    for (int i = 0; i + 1 < H - 1; i++)
        gap = std::min(gap, tau[i + 1] - tau[i]);
    if (!(gap > 0))
        return false;
    // cell width: below the smallest gap, and with every threshold at least
    // 2% of a cell away from a cell edge (rounding of the cell index then
    // never moves a value across a threshold)
    double h = 0;
    for (double f = 0.95; f > 0.5; f -= 0.005) {
        const double hh = gap * f;
        bool ok = true;
        for (int i = 0; i < H - 1 && ok; i++) {
            const double u = tau[i] / hh, frac = u - std::floor(u);
            ok = frac > 0.02 && frac < 0.98;
        }
        if (ok) {
            h = hh;
            break;
        }
    }
    if (!(h > 0))
        return false;
    const int cells = (int)std::floor(tau[H - 2] / h) + 2;
    if (cells > kLutMaxCells)
        return false;
    lut.assign(cells, LutEntry{});
    for (int c = 0; c < cells; c++) {
        const double lo_edge = c * h, hi_edge = (c + 1) * h;
        int m = 0;
        while (m < H - 1 && tau[m] < lo_edge)
            m++;
        LutEntry e;
        e.m = (uint32_t)m;
        e.lo = (float)lev[m];
        e.hi = (float)lev[std::min(m + 1, H - 1)];
        e.t = (m < H - 1 && tau[m] < hi_edge) ? (float)(tau[m] / h) : INFINITY;
        lut[c] = e;
    }
    *inv_h = 1.0 / h;
    return true;
}

}  // namespace isoq
