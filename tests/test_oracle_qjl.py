"""Pins of the oracle's stage-2 residual sketch (oracle.qjl_encode,
oracle.qjl_inner_product; Sec. 8: the residual r = x - x_hat is projected by a
quantized Johnson-Lindenstrauss transform and corrects inner products).

- Unbiasedness over the Gaussian projection: the mean of the two-stage
  estimate over many independent S equals <q, x> (Monte Carlo, within 4
  standard errors), and its variance obeys the QJL bound
  pi / (2 m) * ||q||^2 * ||r||^2.  A dropped sqrt(pi/2), a flipped sign
  convention or a wrong residual biases the mean.
- S = I (m = d): the estimate is <q, x_hat> + sqrt(pi/2)/d ||r|| sum_i q_i s_i
  with s_i the sign of r_i (ties negative), written out.
- Scale equivariance: x -> c x (c > 0) keeps the bits and scales the estimate.
- The projection of the residual equals the projection of the rotated-domain
  quantization error mapped back by T^{-1}: S r = S T^{-1}(rho (y~ - c[idx])),
  Prop. 1 applied to the residual (the route the HIP kernel takes).
"""
import numpy as np
import pytest

import oracle
import workloads


def _setup(variant, d, bits, seed=3):
    rot = workloads.rotation_draws(variant, d, 1, seed=seed)
    levels = oracle.codebook(bits, d)
    return rot, levels


@pytest.mark.parametrize("variant", ["full", "fast", "2d"])
def test_unbiased_with_qjl_variance_bound(variant):
    d, bits, m, draws = 16, 2, 16, 4000
    rot, levels = _setup(variant, d, bits)
    rng = np.random.default_rng(5)
    x = rng.standard_normal((1, d))
    q = rng.standard_normal(d)
    _, _, xh = oracle.stage1(variant, d, bits, rot, levels, x)
    r = x[0] - xh[0]
    # a random query, and one aligned with the residual (stage 1 alone is then
    # biased by exactly ||q|| ||r||)
    qs = np.stack([q, r / np.linalg.norm(r) * np.linalg.norm(q)])
    est = np.empty((draws, 2))
    for k in range(draws):
        S = rng.standard_normal((m, d))
        z, gamma, _, _, _, xh2 = oracle.qjl_encode(variant, d, bits, rot, levels, S, x)
        est[k] = oracle.qjl_inner_product(qs, xh2, z, gamma, S)[:, 0]
    for g in range(2):
        truth = float(qs[g] @ x[0])
        se = est[:, g].std() / np.sqrt(draws)
        assert abs(est[:, g].mean() - truth) < 4 * se, (g, est[:, g].mean(), truth, se)
        bound = np.pi / (2 * m) * (qs[g] @ qs[g]) * (r @ r)
        assert est[:, g].var() <= 1.1 * bound, (g, est[:, g].var(), bound)
    se = est[:, 1].std() / np.sqrt(draws)
    base = float(qs[1] @ xh[0])
    assert abs(base - float(qs[1] @ x[0])) > 8 * se


def test_identity_projection_closed_form():
    variant, d, bits = "fast", 32, 3
    rot, levels = _setup(variant, d, bits)
    x = workloads.unit_gaussian_rows(20, d, seed=8, dtype=np.float64)
    q = np.random.default_rng(9).standard_normal(d)
    z, gamma, p, idx, rho, xh = oracle.qjl_encode(variant, d, bits, rot, levels, np.eye(d), x)
    r = x - xh
    np.testing.assert_array_equal(z, (r > 0).astype(np.uint8))
    np.testing.assert_allclose(gamma, np.linalg.norm(r, axis=1), rtol=1e-15)
    s = np.where(r > 0, 1.0, -1.0)
    ref = xh @ q + np.sqrt(np.pi / 2) / d * gamma * (s @ q)
    np.testing.assert_allclose(oracle.qjl_inner_product(q, xh, z, gamma, np.eye(d)), ref, rtol=1e-13)


def test_scale_equivariance():
    variant, d, bits, m = "full", 64, 3, 64
    rot, levels = _setup(variant, d, bits)
    S = workloads.qjl_matrix(m, d, seed=2)
    x = workloads.unit_gaussian_rows(30, d, seed=4, dtype=np.float64)
    q = np.random.default_rng(1).standard_normal(d)
    z1, g1, _, _, _, xh1 = oracle.qjl_encode(variant, d, bits, rot, levels, S, x)
    z2, g2, _, _, _, xh2 = oracle.qjl_encode(variant, d, bits, rot, levels, S, 8.0 * x)
    np.testing.assert_array_equal(z1, z2)
    np.testing.assert_allclose(g2, 8.0 * g1, rtol=1e-13)
    np.testing.assert_allclose(oracle.qjl_inner_product(q, xh2, z2, g2, S),
                               8.0 * oracle.qjl_inner_product(q, xh1, z1, g1, S), rtol=1e-12)


@pytest.mark.parametrize("variant", ["full", "fast", "2d"])
def test_residual_projection_through_rotated_error(variant):
    d, bits, m = 128, 3, 128
    rot, levels = _setup(variant, d, bits)
    S = workloads.qjl_matrix(m, d, seed=6)
    x = workloads.unit_gaussian_rows(40, d, seed=12, dtype=np.float64) * 3.0
    _, gamma, p, idx, rho, xh = oracle.qjl_encode(variant, d, bits, rot, levels, S, x)
    _, _, _, yt = oracle.stage1(variant, d, bits, rot, levels, x, want_ytil=True)
    e = yt - levels[idx]                                   # rotated-domain error of x / rho
    r_back = np.stack([oracle.decode(variant, d, rot, ei) for ei in e]) * rho[:, None]
    np.testing.assert_allclose(r_back @ S.T, p, rtol=1e-9, atol=1e-12)
    np.testing.assert_allclose(np.linalg.norm(e, axis=1) * rho, gamma, rtol=1e-12)


def test_qjl_matrix_is_standard_gaussian():
    from scipy import stats
    S = workloads.qjl_matrix(256, 128, seed=1)
    assert S.shape == (256, 128)
    assert stats.kstest(S.reshape(-1), "norm").pvalue > 1e-3
    assert not np.array_equal(S, workloads.qjl_matrix(256, 128, seed=2))
