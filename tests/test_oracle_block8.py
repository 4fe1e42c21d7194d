"""Pins of the oracle's 8-D grouped blocks (the block-size axis of Table 3; Sec.
5.7 gives the law of a Haar block rotation for any block size k, here k = 8)
against facts that do not come from the oracle: numpy's QR and determinant,
orthogonal inputs that the orthonormalisation must leave alone, the quaternion
path (Full) embedded as two 4x4 blocks, the Beta law of a uniform point on
S^7, the covariance identity of Sec. 5.7, brute force over the product
codebook and the sphere-marginal MSE integral.  CPU only."""
import numpy as np
import pytest
from scipy import integrate, special, stats

import oracle
import workloads


def _rng(seed):
    return np.random.default_rng(seed)


def _numpy_haar_q(G):
    """Q of G = QR with diag R > 0 (numpy's Householder QR, signs fixed), then
    column 0 negated when det Q = -1."""
    Q, R = np.linalg.qr(G)
    Q = Q * np.sign(np.diag(R))[None, :]
    if np.linalg.det(Q) < 0:
        Q[:, 0] = -Q[:, 0]
    return Q


def _L(q):
    a, b, c, d = q
    return np.array([[a, -b, -c, -d], [b, a, -d, c], [c, d, a, -b], [d, -c, b, a]])


def _R(q):
    a, b, c, d = q
    return np.array([[a, -b, -c, -d], [b, a, d, -c], [c, -d, a, b], [d, c, -b, a]])


def test_det8_matches_numpy():
    rng = _rng(1)
    for _ in range(50):
        M = rng.standard_normal((8, 8))
        assert abs(oracle.det8(M) - np.linalg.det(M)) <= 1e-12 * max(1.0, abs(np.linalg.det(M)))
    P = np.eye(8)[[1, 0, 2, 3, 4, 5, 6, 7]]      # one transposition: det -1
    assert oracle.det8(P) == -1.0
    assert oracle.det8(np.zeros((8, 8))) == 0.0


def test_orthonormalize_matches_numpy_qr_and_is_in_so8():
    G = workloads.rotation_draws("8d", 8 * 40, 1, seed=2).reshape(40, 8, 8)
    neg = 0
    for g in G:
        Q = oracle.orthonormalize8(g)
        np.testing.assert_allclose(Q, _numpy_haar_q(g), atol=1e-13)
        np.testing.assert_allclose(Q.T @ Q, np.eye(8), atol=1e-14)
        assert abs(np.linalg.det(Q) - 1.0) < 1e-13
        Qr, Rr = np.linalg.qr(g)
        neg += np.linalg.det(Qr * np.sign(np.diag(Rr))[None, :]) < 0
    # about half the draws land on the det -1 coset, so the fix is exercised
    assert 5 <= neg <= 35


def test_orthonormalize_leaves_a_rotation_alone():
    """A matrix already in SO(8) is its own Q (R = I)."""
    rng = _rng(3)
    for _ in range(20):
        Q0 = stats.special_ortho_group.rvs(8, random_state=rng)
        np.testing.assert_allclose(oracle.orthonormalize8(Q0), Q0, atol=1e-14)
    np.testing.assert_array_equal(oracle.orthonormalize8(np.eye(8)), np.eye(8))


def test_dependent_columns_are_rejected():
    with pytest.raises(ValueError):
        oracle.orthonormalize8(np.ones((8, 8)))
    G = workloads.rotation_draws("8d", 8, 1, seed=30).reshape(8, 8)
    G[:, 5] = 2.0 * G[:, 1] - G[:, 2]
    with pytest.raises(ValueError):
        oracle.orthonormalize8(G)


def test_block_forward_inverse_are_q_and_its_transpose():
    G = workloads.rotation_draws("8d", 8, 1, seed=4).reshape(8, 8)
    Q = _numpy_haar_q(G)
    v = _rng(5).standard_normal(8)
    y = oracle.block8_forward(G, v)
    np.testing.assert_allclose(y, Q @ v, atol=1e-14)
    np.testing.assert_allclose(oracle.block8_inverse(G, y), v, atol=1e-14)
    np.testing.assert_allclose(np.linalg.norm(y), np.linalg.norm(v), rtol=1e-15)


def test_embedded_quaternion_blocks_give_the_full_path():
    """With G = diag(M_1, M_2), M = L(q_L) R(conj q_R) from the textbook
    left/right multiplication matrices, G is already in SO(8), so the 8-D path
    is IsoQuant-Full on the same quaternions."""
    d, bits, n = 32, 3, 300
    raw_full = workloads.rotation_draws("full", d, 1, seed=6).reshape(d // 4, 8)
    blocks = []
    for i in range(d // 8):
        Ms = []
        for u in raw_full[2 * i: 2 * i + 2]:
            qL, qR = u[:4] / np.linalg.norm(u[:4]), u[4:] / np.linalg.norm(u[4:])
            Ms.append(_L(qL) @ _R(qR * np.array([1, -1, -1, -1])))
        G = np.zeros((8, 8))
        G[:4, :4], G[4:, 4:] = Ms
        blocks.append(G)
    rot8 = np.stack(blocks).reshape(-1)
    c = oracle.codebook(bits, d)
    x = workloads.unit_gaussian_rows(n, d, seed=7, dtype=np.float64)
    i8, r8, h8, y8 = oracle.stage1("8d", d, bits, rot8, c, x, want_ytil=True)
    i4, r4, h4, y4 = oracle.stage1("full", d, bits, raw_full.reshape(-1), c, x, want_ytil=True)
    np.testing.assert_allclose(y8, y4, atol=1e-14)
    near = np.abs(y4[..., None] - oracle.thresholds(bits, c)).min(-1) <= 1e-12
    assert np.all((i8 == i4) | near)
    ok = ~near.any(1)
    np.testing.assert_allclose(h8[ok], h4[ok], atol=1e-14)
    np.testing.assert_array_equal(r8, r4)


def test_haar_marginal_k8():
    """Sec. 5.7 with k = 8: a fixed unit block rotated by R ~ Haar(SO(8)) is
    uniform on S^7, so each coordinate z has density prop. to (1 - z^2)^(5/2),
    i.e. (z + 1) / 2 ~ Beta(7/2, 7/2), and E[y_j^2] = r^2 / 8."""
    n = 6000
    G = workloads.rotation_draws("8d", 8 * n, 1, seed=8).reshape(n, 8, 8)
    v = np.array([0.3, -0.5, 0.7, 0.2, 0.1, -0.25, 0.4, 0.05])
    r = np.linalg.norm(v)
    ys = np.array([oracle.block8_forward(g, v) for g in G]) / r
    np.testing.assert_allclose((ys ** 2).mean(0), 1.0 / 8.0, atol=0.01)
    np.testing.assert_allclose(ys.mean(0), 0.0, atol=0.015)
    for j in range(8):
        assert stats.kstest((ys[:, j] + 1) / 2, stats.beta(3.5, 3.5).cdf).pvalue > 1e-3
    # the same law written as the normalised density of Sec. 5.7
    f8 = lambda z: (1 - z * z) ** 2.5 / special.beta(0.5, 3.5)
    assert abs(integrate.quad(f8, -1, 1, epsabs=1e-13)[0] - 1.0) < 1e-10
    cdf = lambda z: np.array([integrate.quad(f8, -1, t)[0] for t in np.atleast_1d(z)])
    assert stats.kstest(ys[:2000, 0], cdf).pvalue > 1e-3


def test_block_covariance_becomes_isotropic():
    """Sec. 5.7: E_R[R Sigma R^T] = tr(Sigma) / k I for R ~ Haar(SO(k))."""
    n = 6000
    G = workloads.rotation_draws("8d", 8 * n, 1, seed=9).reshape(n, 8, 8)
    A = _rng(10).standard_normal((8, 8))
    Sigma = A @ A.T / 8
    acc = np.zeros((8, 8))
    for g in G:
        Q = oracle.orthonormalize8(g)
        acc += Q @ Sigma @ Q.T
    acc /= n
    np.testing.assert_allclose(acc, np.trace(Sigma) / 8 * np.eye(8), atol=0.06 * np.trace(Sigma) / 8)


def test_brute_force_product_codebook_d8():
    """By orthogonality the per-coordinate nearest levels in the rotated basis
    are the nearest of the 4^8 codewords Q^T c_idx in the input space."""
    d, bits, n = 8, 2, 30
    rot = workloads.rotation_draws("8d", d, 1, seed=11)
    Q = _numpy_haar_q(rot.reshape(8, 8))
    c = oracle.codebook(bits, d)
    x = _rng(12).standard_normal((n, d))
    idx, rho, xh = oracle.stage1("8d", d, bits, rot, c, x)
    grids = np.array(np.meshgrid(*[np.arange(4)] * 8, indexing="ij")).reshape(8, -1).T
    words = c[grids] @ Q          # rows: (Q^T c_idx)^T
    for r in range(n):
        xbar = x[r] / np.linalg.norm(x[r])
        best = grids[np.argmin(((xbar[None, :] - words) ** 2).sum(1))]
        np.testing.assert_array_equal(idx[r], best)
        np.testing.assert_allclose(xh[r], rho[r] * c[best] @ Q, atol=1e-15)


def test_identity_blocks_are_plain_bucketize():
    d, bits = 64, 3
    x = workloads.unit_gaussian_rows(200, d, seed=13, dtype=np.float64)
    c = oracle.codebook(bits, d)
    rot = np.tile(np.eye(8).reshape(-1), d // 8)
    idx, rho, xh = oracle.stage1("8d", d, bits, rot, c, x)
    xbar = x / np.linalg.norm(x, axis=1, keepdims=True)
    np.testing.assert_array_equal(idx, np.searchsorted(oracle.thresholds(bits, c), xbar, side="left"))
    np.testing.assert_allclose(xh, rho[:, None] * c[idx], rtol=1e-14, atol=1e-16)


def test_rotation_counts():
    """64 multiplications per block and direction: 8 d per vector, 1,024 at
    d = 128 (the same forward count as IsoQuant-Full in Table 1)."""
    d = 128
    rot = workloads.rotation_draws("8d", d, 1, seed=1)
    assert len(rot) == oracle.raw_params_per_set("8d", d) == 64 * 16
    assert oracle.num_blocks("8d", d) == 16 and oracle.padded_width("8d", d) == 128
    oracle.mul_count_reset()
    y = oracle.encode("8d", d, rot, _rng(14).standard_normal(d))
    assert oracle.mul_count() == 1024
    oracle.mul_count_reset()
    oracle.decode("8d", d, rot, y)
    assert oracle.mul_count() == 1024


def _sphere_mse(d, bits, c):
    t = np.concatenate([[-1.0], oracle.thresholds(bits, c), [1.0]])
    norm = special.beta(0.5, (d - 1) / 2.0)
    f = lambda z: (1 - z * z) ** ((d - 3) / 2.0) / norm
    return sum(integrate.quad(lambda z, ck=c[k]: (z - ck) ** 2 * f(z), t[k], t[k + 1], epsabs=1e-14)[0]
               for k in range(len(c)))


def test_mse_matches_sphere_integral():
    """Unit-norm Gaussian rows are uniform on S^(d-1) and the block rotation is
    orthogonal, so every rotated coordinate has the marginal f_d of Sec. 5.7:
    the per-coordinate MSE equals the 1-D integral the other variants meet."""
    d, bits, n = 128, 3, 6000
    x = workloads.unit_gaussian_rows(n, d, seed=15, dtype=np.float64)
    rot = workloads.rotation_draws("8d", d, 1, seed=1)
    c = oracle.codebook(bits, d)
    _, _, xh = oracle.stage1("8d", d, bits, rot, c, x, want_idx=False)
    mse = np.mean((x - xh) ** 2)
    ref = _sphere_mse(d, bits, c)
    assert abs(mse / ref - 1) < 0.015, (mse, ref)


@pytest.mark.parametrize("d,pw", [(13, 16), (5, 8), (1, 8), (70, 72)])
def test_zero_padding(d, pw):
    """Widths that are not a multiple of 8 pad the last block with zeros (Sec.
    4.1, Algorithm 1): the result is the pw-wide path on the zero-padded
    direction with the padded outputs dropped; all pw indices are kept."""
    bits = 3
    x = _rng(16).standard_normal((30, d))
    rot = workloads.rotation_draws("8d", pw, 1, seed=17)
    assert len(rot) == workloads.raw_params_per_set("8d", d) == oracle.raw_params_per_set("8d", d)
    c = oracle.codebook(bits, d)
    idx, rho, xh = oracle.stage1("8d", d, bits, rot, c, x)
    assert idx.shape == (30, pw) and oracle.padded_width("8d", d) == pw
    thr = oracle.thresholds(bits, c)
    for r in range(30):
        xb = np.zeros(pw)
        xb[:d] = x[r] / np.linalg.norm(x[r])
        y = oracle.encode("8d", pw, rot, xb)
        np.testing.assert_array_equal(idx[r], np.searchsorted(thr, y))
        rec = oracle.decode("8d", pw, rot, c[idx[r]])
        np.testing.assert_allclose(xh[r], rho[r] * rec[:d], rtol=1e-15, atol=1e-17)


def test_zero_row_scale_invariance_and_sets():
    d, bits = 32, 3
    c = oracle.codebook(bits, d)
    rot = workloads.rotation_draws("8d", d, 3, seed=18)
    idx, rho, xh = oracle.stage1("8d", d, bits, rot[: 64 * 4], c, np.zeros((1, d)))
    assert rho[0] == 0 and np.all(idx == 3) and np.all(xh == 0)
    x = workloads.unit_gaussian_rows(24, d, seed=19, dtype=np.float64)
    i0, r0, h0 = oracle.stage1("8d", d, bits, rot, c, x, n_sets=3, rows_per_set=2)
    i1, r1, h1 = oracle.stage1("8d", d, bits, rot, c, 1e3 * x, n_sets=3, rows_per_set=2)
    np.testing.assert_array_equal(i0, i1)
    np.testing.assert_allclose(h1, 1e3 * h0, rtol=1e-12, atol=1e-12)
    per = 64 * 4
    for r in range(24):
        s = (r // 2) % 3
        ir, _, hr = oracle.stage1("8d", d, bits, rot[s * per:(s + 1) * per], c, x[r:r + 1])
        np.testing.assert_array_equal(i0[r], ir[0])
        np.testing.assert_allclose(h0[r], hr[0], rtol=0, atol=0)
