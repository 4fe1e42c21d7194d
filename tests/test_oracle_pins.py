"""Pins of the CPU oracle against facts that do not come from the oracle itself:
the defining relations of the quaternions (Sec. 4), the textbook matrix and
rotation formulas (Kuipers), Proposition 1, Table 1's counts, Max's 1960
Lloyd-Max tables, numpy/scipy routines, brute force and closed-form integrals
(Sec. 5.7).  CPU only."""
import json
import math
import os

import numpy as np
import pytest
from scipy import integrate, special, stats

import oracle
import workloads

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
ONE, I, J, K = np.eye(4)


def _rng(seed):
    return np.random.default_rng(seed)


def _unit(v):
    v = np.asarray(v, float)
    return v / np.linalg.norm(v)


# --------------------------------------------------------------------------- Sec. 4
def test_defining_relations():
    # i^2 = j^2 = k^2 = ijk = -1
    for e in (I, J, K):
        np.testing.assert_array_equal(oracle.qmul(e, e), -ONE)
    np.testing.assert_array_equal(oracle.qmul(oracle.qmul(I, J), K), -ONE)
    np.testing.assert_array_equal(oracle.qmul(I, oracle.qmul(J, K)), -ONE)
    # 1 is the identity on both sides
    p = _rng(0).standard_normal(4)
    np.testing.assert_array_equal(oracle.qmul(ONE, p), p)
    np.testing.assert_array_equal(oracle.qmul(p, ONE), p)


def test_algebra_laws():
    rng = _rng(1)
    for _ in range(50):
        p, q, r = rng.standard_normal((3, 4))
        # associativity, norm multiplicativity
        np.testing.assert_allclose(oracle.qmul(oracle.qmul(p, q), r),
                                   oracle.qmul(p, oracle.qmul(q, r)), atol=1e-13)
        np.testing.assert_allclose(np.linalg.norm(oracle.qmul(p, q)),
                                   np.linalg.norm(p) * np.linalg.norm(q), rtol=1e-13)
        # conj(pq) = conj(q) conj(p);  q conj(q) = |q|^2
        np.testing.assert_allclose(oracle.qconj(oracle.qmul(p, q)),
                                   oracle.qmul(oracle.qconj(q), oracle.qconj(p)), atol=1e-13)
        np.testing.assert_allclose(oracle.qmul(q, oracle.qconj(q)), np.dot(q, q) * ONE, atol=1e-13)
    # not commutative
    assert not np.allclose(oracle.qmul(I, J), oracle.qmul(J, I))


def _kuipers_left(p):
    a, b, c, d = p
    return np.array([[a, -b, -c, -d], [b, a, -d, c], [c, d, a, -b], [d, -c, b, a]])


def _kuipers_right(q):
    a, b, c, d = q
    return np.array([[a, -b, -c, -d], [b, a, d, -c], [c, -d, a, b], [d, c, -b, a]])


def test_product_matches_matrix_forms():
    """p q = L(p) q = R(q) p with the textbook left/right multiplication matrices."""
    rng = _rng(2)
    for _ in range(50):
        p, q = rng.standard_normal((2, 4))
        pq = oracle.qmul(p, q)
        np.testing.assert_allclose(pq, _kuipers_left(p) @ q, atol=1e-14)
        np.testing.assert_allclose(pq, _kuipers_right(q) @ p, atol=1e-14)


# ------------------------------------------------------------------ Proposition 1
def _matrix_of(f):
    return np.stack([f(e) for e in (ONE, I, J, K)], axis=1)


def test_proposition1_orthogonal_inverse_double_cover():
    rng = _rng(3)
    for _ in range(30):
        qL = oracle.qnormalize(rng.standard_normal(4))
        qR = oracle.qnormalize(rng.standard_normal(4))
        M = _matrix_of(lambda v: oracle.full_forward(qL, qR, v))
        np.testing.assert_allclose(M.T @ M, np.eye(4), atol=1e-14)
        assert abs(np.linalg.det(M) - 1.0) < 1e-13          # in SO(4)
        Mi = _matrix_of(lambda v: oracle.full_inverse(qL, qR, v))
        np.testing.assert_allclose(Mi @ M, np.eye(4), atol=1e-14)
        np.testing.assert_allclose(Mi, M.T, atol=1e-14)
        Mneg = _matrix_of(lambda v: oracle.full_forward(-qL, -qR, v))
        np.testing.assert_allclose(Mneg, M, atol=1e-15)
        v = rng.standard_normal(4)
        np.testing.assert_allclose(np.linalg.norm(oracle.full_forward(qL, qR, v)),
                                   np.linalg.norm(v), rtol=1e-14)
        # Fast: left isoclinic factor only
        F = _matrix_of(lambda v: oracle.fast_forward(qL, v))
        np.testing.assert_allclose(F.T @ F, np.eye(4), atol=1e-14)
        Fi = _matrix_of(lambda v: oracle.fast_inverse(qL, v))
        np.testing.assert_allclose(Fi @ F, np.eye(4), atol=1e-14)


def test_full_with_unit_right_factor_is_fast():
    rng = _rng(4)
    for _ in range(30):
        qL = oracle.qnormalize(rng.standard_normal(4))
        v = rng.standard_normal(4)
        np.testing.assert_array_equal(oracle.full_forward(qL, ONE, v), oracle.fast_forward(qL, v))
        np.testing.assert_array_equal(oracle.full_inverse(qL, ONE, v), oracle.fast_inverse(qL, v))


def test_equal_factors_rotate_imaginary_part_like_rodrigues():
    """q v conj(q) fixes the real part and rotates (b, c, d) about the axis of q
    by angle 2 acos(a) (the classical quaternion rotation, Kuipers)."""
    rng = _rng(5)
    for _ in range(30):
        q = oracle.qnormalize(rng.standard_normal(4))
        v = rng.standard_normal(4)
        out = oracle.full_forward(q, q, v)
        assert abs(out[0] - v[0]) < 1e-14
        ang = 2.0 * math.acos(np.clip(q[0], -1, 1))
        k = _unit(q[1:])
        w = v[1:]
        rod = (w * math.cos(ang) + np.cross(k, w) * math.sin(ang)
               + k * np.dot(k, w) * (1 - math.cos(ang)))
        np.testing.assert_allclose(out[1:], rod, atol=1e-13)


def test_planar_rotation_is_complex_multiplication():
    rng = _rng(6)
    for _ in range(30):
        th = rng.uniform(0, 2 * np.pi)
        u = rng.standard_normal(2)
        z = complex(u[0], u[1]) * np.exp(1j * th)
        np.testing.assert_allclose(oracle.planar_forward(th, u), [z.real, z.imag], atol=1e-14)
        np.testing.assert_allclose(oracle.planar_inverse(th, oracle.planar_forward(th, u)), u,
                                   atol=1e-14)


# ------------------------------------------------------------------- Table 1 counts
def test_table1_counts():
    g = json.load(open(os.path.join(GOLDEN, "table1_complexity.json")))
    d = g["d"]
    for name in ("full", "fast", "2d"):
        rot = workloads.rotation_draws(name, d, 1, seed=1)
        x = _unit(_rng(7).standard_normal(d))
        oracle.mul_count_reset()
        oracle.encode(name, d, rot, x)
        assert oracle.mul_count() == g[name]["fma"], name
        assert oracle.table1_params(name, d) == g[name]["params"], name
        assert oracle.num_blocks(name, d) == g[name]["blocks"], name
    gen = g["general"]
    for d in (4, 8, 64, 96, 256, 512):
        g4, g2 = -(-d // 4), -(-d // 2)
        for name, gg, per in (("full", g4, "g4"), ("fast", g4, "g4"), ("2d", g2, "g2")):
            rot = workloads.rotation_draws(name, d, 1, seed=2)
            oracle.mul_count_reset()
            oracle.encode(name, d, rot, np.ones(d) / np.sqrt(d))
            assert oracle.mul_count() == gen[name]["fma_per_" + per] * gg
            assert oracle.table1_params(name, d) == gen[name]["params_per_" + per] * gg


# --------------------------------------------------------------------- codebook
def test_codebook_matches_max_table():
    g = json.load(open(os.path.join(GOLDEN, "lloyd_max_gaussian.json")))
    for b in (1, 2, 3, 4):
        pos = np.array(g["levels_positive"][str(b)])
        conv = oracle.lloyd_max_gaussian(b, 1.0, iters=5000)
        K = 1 << b
        np.testing.assert_allclose(conv[K // 2:], pos, atol=6e-4, rtol=6e-4)
        np.testing.assert_array_equal(conv[:K // 2], -conv[K // 2:][::-1])
        # distortion of the converged codebook, by numerical integration
        t = np.concatenate([[-np.inf], oracle.thresholds(b, conv), [np.inf]])
        D = sum(integrate.quad(lambda x, c=conv[k]: (x - c) ** 2 * stats.norm.pdf(x),
                               t[k], t[k + 1])[0] for k in range(K))
        assert abs(D - g["distortion"][str(b)]) <= 1e-3 * g["distortion"][str(b)] + 5e-6
        # 200 iterations (the workload setting) is within 1e-3 of the fixed point
        c200 = oracle.lloyd_max_gaussian(b, 1.0, iters=200)
        np.testing.assert_allclose(c200, conv, atol=1e-3)


def test_codebook_centroid_condition_by_quadrature():
    """Converged levels are the conditional means of their cells (computed by
    scipy quadrature, not the closed form the oracle uses)."""
    for b in (2, 3):
        for sigma in (1.0, 1 / np.sqrt(128)):
            c = oracle.lloyd_max_gaussian(b, sigma, iters=200)
            t = np.concatenate([[-np.inf], oracle.thresholds(b, c), [np.inf]])
            for k in range(len(c)):
                m = integrate.quad(lambda x: x * stats.norm.pdf(x, scale=sigma), t[k], t[k + 1])[0]
                p = integrate.quad(lambda x: stats.norm.pdf(x, scale=sigma), t[k], t[k + 1])[0]
                assert abs(m / p - c[k]) < 1e-8 * max(1.0, abs(c[k]) / sigma) * sigma * 10


def test_thresholds_are_midpoints_and_symmetric():
    for b in (1, 2, 3, 4):
        c = oracle.codebook(b, 128)
        t = oracle.thresholds(b, c)
        np.testing.assert_allclose(t, 0.5 * (c[:-1] + c[1:]), rtol=0, atol=0)
        assert t[len(t) // 2] == 0.0


# -------------------------------------------------------------------- quantizer
def _identity_draws(variant, d):
    v = workloads.variant_id(variant)
    if v == workloads.PLANAR2D:
        return np.zeros((d + 1) // 2)
    per = 8 if v == workloads.FULL else 4
    g = (d + 3) // 4
    r = np.zeros((g, per))
    r[:, 0] = 1.0
    if per == 8:
        r[:, 4] = 1.0
    return r.reshape(-1)


@pytest.mark.parametrize("variant", ["full", "fast", "2d"])
@pytest.mark.parametrize("bits", [2, 3, 4])
def test_identity_rotation_is_plain_bucketize(variant, bits):
    d = 64
    x = workloads.unit_gaussian_rows(300, d, seed=11, dtype=np.float64)
    c = oracle.codebook(bits, d)
    idx, rho, xh = oracle.stage1(variant, d, bits, _identity_draws(variant, d), c, x)
    xbar = x / np.linalg.norm(x, axis=1, keepdims=True)
    t = oracle.thresholds(bits, c)
    np.testing.assert_array_equal(idx, np.searchsorted(t, xbar, side="left"))
    np.testing.assert_array_equal(idx, np.argmin(np.abs(xbar[..., None] - c), axis=-1))
    np.testing.assert_allclose(rho, np.linalg.norm(x, axis=1), rtol=1e-15)
    np.testing.assert_allclose(xh, rho[:, None] * c[idx], rtol=1e-14, atol=1e-16)


def _brute_force_indices(variant, d, bits, rot, c, xbar):
    """argmin over the whole product codebook {T^-1 c_idx} in the original space."""
    K = 1 << bits
    pw = oracle.padded_width(variant, d)
    grids = np.array(np.meshgrid(*[np.arange(K)] * pw, indexing="ij")).reshape(pw, -1).T
    # the decoder is linear: its matrix from the basis, then every codeword at once
    dec = np.stack([oracle.decode(variant, d, rot, e) for e in np.eye(pw)], axis=1)
    words = c[grids] @ dec.T
    best = np.argmin(((xbar[None, :] - words) ** 2).sum(1))
    return grids[best]


@pytest.mark.parametrize("variant,d,bits", [("full", 4, 2), ("full", 4, 3), ("fast", 4, 3),
                                            ("2d", 4, 3), ("full", 8, 2), ("fast", 8, 2),
                                            ("2d", 2, 4)])
def test_brute_force_product_codebook(variant, d, bits):
    """By orthogonality (Prop. 1) the per-coordinate nearest levels in the rotated
    basis are the nearest codeword of the product codebook in the input space."""
    rng = _rng(12)
    rot = workloads.rotation_draws(variant, d, 1, seed=3)
    c = oracle.codebook(bits, d)
    n = 40 if d == 8 else 120
    x = rng.standard_normal((n, d))
    idx, rho, xh = oracle.stage1(variant, d, bits, rot, c, x)
    for r in range(n):
        xbar = x[r] / np.linalg.norm(x[r])
        np.testing.assert_array_equal(idx[r], _brute_force_indices(variant, d, bits, rot, c, xbar))


# -------------------------------------------------------------------- MSE theory
def _sphere_mse(d, bits, c):
    """E[(z - Q(z))^2] for one coordinate of a uniform point on S^{d-1}:
    density f_d(z) = (1 - z^2)^((d-3)/2) / B(1/2, (d-1)/2) (Sec. 5.7)."""
    t = np.concatenate([[-1.0], oracle.thresholds(bits, c), [1.0]])
    norm = special.beta(0.5, (d - 1) / 2.0)
    f = lambda z: (1 - z * z) ** ((d - 3) / 2.0) / norm
    return sum(integrate.quad(lambda z, ck=c[k]: (z - ck) ** 2 * f(z), t[k], t[k + 1],
                              epsabs=1e-14)[0] for k in range(len(c)))


@pytest.mark.parametrize("variant", ["full", "fast", "2d"])
def test_mse_matches_sphere_integral(variant):
    """Unit-norm Gaussian rows are uniform on the sphere and every block rotation
    is orthogonal, so each rotated coordinate has the marginal f_d; the
    per-coordinate MSE is then a 1-D integral, the same for all variants."""
    d, bits, n = 128, 3, 6000
    x = workloads.unit_gaussian_rows(n, d, seed=13, dtype=np.float64)
    rot = workloads.rotation_draws(variant, d, 1, seed=1)
    c = oracle.codebook(bits, d)
    _, _, xh = oracle.stage1(variant, d, bits, rot, c, x, want_idx=False)
    mse = np.mean((x - xh) ** 2)
    ref = _sphere_mse(d, bits, c)
    assert abs(mse / ref - 1) < 0.015, (mse, ref)


def test_mse_large_d_approaches_gaussian_distortion():
    """For large d the marginal tends to N(0, 1/d), so d * MSE -> Max's D_b."""
    g = json.load(open(os.path.join(GOLDEN, "lloyd_max_gaussian.json")))
    d, n = 512, 1500
    x = workloads.unit_gaussian_rows(n, d, seed=14, dtype=np.float64)
    for bits in (2, 3, 4):
        c = oracle.codebook(bits, d)
        rot = workloads.rotation_draws("full", d, 1, seed=1)
        _, _, xh = oracle.stage1("full", d, bits, rot, c, x, want_idx=False)
        dm = d * np.mean((x - xh) ** 2)
        assert abs(dm / g["distortion"][str(bits)] - 1) < 0.03, (bits, dm)


# ------------------------------------------------------------ Sec. 5.7 marginals
def test_haar_block_marginals():
    """A fixed unit block rotated by a Haar-random factor: E[y_j^2] = 1/k, with
    the f_4 law (2/pi) sqrt(1 - z^2) for quaternion factors and the arcsine law
    for the planar case."""
    n = 20000
    v = _unit([0.3, -0.5, 0.7, 0.2])
    seeds = np.arange(n)
    uL = workloads.philox_gaussian4(seeds, 0, 0, 21)
    uR = workloads.philox_gaussian4(seeds, 0, 1, 21)
    ys_fast = np.array([oracle.fast_forward(oracle.qnormalize(a), v) for a in uL])
    ys_full = np.array([oracle.full_forward(oracle.qnormalize(a), oracle.qnormalize(b), v)
                        for a, b in zip(uL, uR)])
    cdf4 = lambda z: 0.5 + (z * np.sqrt(1 - z * z) + np.arcsin(z)) / np.pi
    for ys in (ys_fast, ys_full):
        np.testing.assert_allclose((ys ** 2).mean(0), 0.25, atol=0.01)
        for j in range(4):
            assert stats.kstest(ys[:, j], cdf4).pvalue > 1e-3
    th = workloads.rotation_draws("2d", 2 * n, 1, seed=22)
    u = _unit([0.6, -0.8])
    y2 = np.array([oracle.planar_forward(t, u) for t in th[:n]])
    np.testing.assert_allclose((y2 ** 2).mean(0), 0.5, atol=0.01)
    assert stats.kstest(y2[:, 0], lambda z: 0.5 + np.arcsin(z) / np.pi).pvalue > 1e-3


# --------------------------------------------------------------- pipeline details
def test_zero_vector():
    for variant in ("full", "fast", "2d"):
        for bits in (2, 3, 4):
            c = oracle.codebook(bits, 16)
            rot = workloads.rotation_draws(variant, 16, 1, seed=1)
            idx, rho, xh = oracle.stage1(variant, 16, bits, rot, c, np.zeros((1, 16)))
            assert rho[0] == 0.0
            assert np.all(idx == (1 << bits) // 2 - 1)
            assert np.all(xh == 0.0)


def test_scale_invariance_of_indices():
    """Norm and direction are split (Sec. 3): scaling a nonzero row by s leaves
    the indices unchanged and scales the reconstruction by s."""
    d, bits = 32, 3
    x = workloads.unit_gaussian_rows(40, d, seed=23, dtype=np.float64)
    for variant in ("full", "fast", "2d"):
        rot = workloads.rotation_draws(variant, d, 1, seed=8)
        c = oracle.codebook(bits, d)
        i0, r0, h0 = oracle.stage1(variant, d, bits, rot, c, x)
        for s in (1e-6, 1e-3, 1e3):
            i1, r1, h1 = oracle.stage1(variant, d, bits, rot, c, s * x)
            np.testing.assert_array_equal(i1, i0)
            np.testing.assert_allclose(r1, s * r0, rtol=1e-14)
            np.testing.assert_allclose(h1, s * h0, rtol=1e-12, atol=1e-14 * s)


def test_encoder_is_block_diagonal_kuipers():
    """The encoder applies, block by block on contiguous coordinates 4i..4i+3
    (coordinate 4i real), the matrix L(q_L) R(conj q_R) built from the textbook
    forms; Fast uses L(q_L); 2-D uses the rotation matrix on pairs."""
    d = 16
    rng = _rng(15)
    x = _unit(rng.standard_normal(d))
    rot = workloads.rotation_draws("full", d, 1, seed=4).reshape(-1, 8)
    blocks = []
    for u in rot:
        qL, qR = _unit(u[:4]), _unit(u[4:])
        blocks.append(_kuipers_left(qL) @ _kuipers_right(qR * [1, -1, -1, -1]))
    from scipy.linalg import block_diag
    np.testing.assert_allclose(oracle.encode("full", d, rot.reshape(-1), x), block_diag(*blocks) @ x,
                               atol=1e-14)
    rotf = workloads.rotation_draws("fast", d, 1, seed=4).reshape(-1, 4)
    Bf = block_diag(*[_kuipers_left(_unit(u)) for u in rotf])
    np.testing.assert_allclose(oracle.encode("fast", d, rotf.reshape(-1), x), Bf @ x, atol=1e-14)
    th = workloads.rotation_draws("2d", d, 1, seed=4)
    B2 = block_diag(*[[[np.cos(t), -np.sin(t)], [np.sin(t), np.cos(t)]] for t in th])
    np.testing.assert_allclose(oracle.encode("2d", d, th, x), B2 @ x, atol=1e-14)
    # decoder is the transpose
    y = rng.standard_normal(d)
    np.testing.assert_allclose(oracle.decode("full", d, rot.reshape(-1), y), block_diag(*blocks).T @ y,
                               atol=1e-14)


def test_zero_padding_when_d_not_multiple_of_four():
    """d = 6: the last block is zero padded and the padding dropped after the
    inverse (Sec. 5.1, Algorithm 1); equals the d = 8 path on the padded input
    with the padded coordinates' outputs discarded."""
    d, bits = 6, 3
    rng = _rng(16)
    x = rng.standard_normal((50, d))
    rot = workloads.rotation_draws("full", 8, 1, seed=5)
    c = oracle.codebook(bits, d)
    idx, rho, xh = oracle.stage1("full", d, bits, rot, c, x)
    assert idx.shape == (50, 8)
    for r in range(50):
        xb = np.zeros(8)
        xb[:d] = x[r] / np.linalg.norm(x[r])
        y = oracle.encode("full", 8, rot, xb)
        np.testing.assert_array_equal(idx[r], np.searchsorted(oracle.thresholds(bits, c), y))
        rec = oracle.decode("full", 8, rot, c[idx[r]])
        np.testing.assert_allclose(xh[r], rho[r] * rec[:d], rtol=1e-15, atol=1e-17)


@pytest.mark.parametrize("variant,d,pw", [("2d", 5, 6), ("2d", 9, 10), ("fast", 7, 8), ("fast", 1, 4)])
def test_zero_padding_other_variants(variant, d, pw):
    """Odd widths in the 2-D case pad the last pair, widths below a multiple
    of 4 pad the last quaternion block (Sec. 5.1, Algorithm 1): the result is
    the pw-wide path on the zero-padded direction with the padded outputs
    dropped, and the record holds all pw rotated coordinates."""
    bits = 3
    rng = _rng(18)
    x = rng.standard_normal((40, d))
    rot = workloads.rotation_draws(variant, pw, 1, seed=7)
    assert len(rot) == workloads.raw_params_per_set(variant, d)
    c = oracle.codebook(bits, d)
    idx, rho, xh = oracle.stage1(variant, d, bits, rot, c, x)
    assert idx.shape == (40, pw) and oracle.padded_width(variant, d) == pw
    thr = oracle.thresholds(bits, c)
    for r in range(40):
        xb = np.zeros(pw)
        xb[:d] = x[r] / np.linalg.norm(x[r])
        y = oracle.encode(variant, pw, rot, xb)
        np.testing.assert_array_equal(idx[r], np.searchsorted(thr, y))
        rec = oracle.decode(variant, pw, rot, c[idx[r]])
        np.testing.assert_allclose(xh[r], rho[r] * rec[:d], rtol=1e-15, atol=1e-17)


def test_multiple_parameter_sets():
    d, bits, n_sets, rps = 16, 3, 3, 2
    rng = _rng(17)
    x = rng.standard_normal((20, d))
    rot = workloads.rotation_draws("fast", d, n_sets, seed=6)
    per = workloads.raw_params_per_set("fast", d)
    c = oracle.codebook(bits, d)
    idx, rho, xh = oracle.stage1("fast", d, bits, rot, c, x, n_sets=n_sets, rows_per_set=rps)
    for r in range(20):
        s = (r // rps) % n_sets
        i1, r1, h1 = oracle.stage1("fast", d, bits, rot[s * per:(s + 1) * per], c, x[r:r + 1])
        np.testing.assert_array_equal(idx[r], i1[0])
        np.testing.assert_array_equal(xh[r], h1[0])
    sel = np.array([19, 0, 7])
    i2, r2, h2 = oracle.stage1("fast", d, bits, rot, c, x, n_sets=n_sets, rows_per_set=rps, rows=sel)
    np.testing.assert_array_equal(i2, idx[sel])
    np.testing.assert_array_equal(h2, xh[sel])


def test_dequantize_inverts_stage1_decoder():
    d, bits = 32, 3
    for variant in ("full", "fast", "2d"):
        x = workloads.unit_gaussian_rows(30, d, seed=18, dtype=np.float32)
        rot = workloads.rotation_draws(variant, d, 1, seed=7)
        c = oracle.codebook(bits, d)
        idx, rho, xh = oracle.stage1(variant, d, bits, rot, c, x)
        np.testing.assert_array_equal(oracle.dequantize(variant, d, bits, rot, c, idx, rho), xh)


# ---------------------------------------------------------------------- packing
def test_pack_matches_little_endian_integer():
    """LSB-first record: the record read as a little-endian integer equals
    sum_j idx_j << (j * bits)."""
    rng = _rng(19)
    for bits in (1, 2, 3, 4, 5):
        for m in (1, 7, 8, 128, 131):
            idx = rng.integers(0, 1 << bits, size=(5, m), dtype=np.uint8)
            packed = oracle.pack(idx, bits)
            assert packed.shape == (5, (m * bits + 7) // 8)
            for r in range(5):
                val = sum(int(v) << (j * bits) for j, v in enumerate(idx[r]))
                assert bytes(packed[r]) == val.to_bytes(packed.shape[1], "little")
            np.testing.assert_array_equal(oracle.unpack(packed, m, bits), idx)


def test_pack_hand_example():
    # indices 1..7,0 at 3 bits, worked by hand: set bits are 0,4,6,7 (byte 0),
    # 11,12,14 (byte 1) and 16..20 (byte 2) -> bytes D1 58 1F
    packed = oracle.pack(np.array([[1, 2, 3, 4, 5, 6, 7, 0]], np.uint8), 3)
    assert list(packed[0]) == [0xD1, 0x58, 0x1F]
