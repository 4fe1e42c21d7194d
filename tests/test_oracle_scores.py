"""Pins of the oracle's attention logits against quantized keys
(oracle.attention_scores: scale * <q, dequantized key>, by definition).

- With identity rotations the logit is the textbook codebook dot product
  scale * rho * sum_j q_j c[idx_j].
- Proposition 1 (T orthogonal): the logit equals scale * rho * <T q, c[idx]>,
  computed here through the oracle's forward rotation, a route independent of
  the inverse rotation inside dequantize; a transposed or conjugated factor in
  either route breaks the equality.
- d = 4: the logit equals scale * rho * <q, M^T c[idx]> with M the explicit
  4 x 4 matrix of the sandwich, built column by column from the basis.
"""
import numpy as np
import pytest

import oracle
import workloads
from test_oracle_pins import _identity_draws


def _keys(rng, n, d, bits):
    K = 1 << bits
    idx = rng.integers(0, K, (n, d)).astype(np.uint8)
    rho = rng.uniform(0.1, 3.0, n)
    return idx, rho


@pytest.mark.parametrize("variant", ["full", "fast", "2d"])
@pytest.mark.parametrize("bits", [2, 3, 4])
def test_identity_rotation_is_codebook_dot(variant, bits):
    d = 64
    rng = np.random.default_rng(1)
    c = oracle.codebook(bits, d)
    idx, rho = _keys(rng, 50, d, bits)
    q = rng.standard_normal((3, d))
    s = oracle.attention_scores(variant, d, bits, _identity_draws(variant, d), c, q, idx, rho, 0.125)
    ref = 0.125 * np.einsum("gd,nd->gn", q, c[idx]) * rho[None, :]
    np.testing.assert_allclose(s, ref, rtol=1e-13, atol=1e-15)


@pytest.mark.parametrize("variant", ["full", "fast", "2d"])
@pytest.mark.parametrize("d,bits", [(128, 3), (256, 2), (64, 4)])
def test_rotated_query_form_proposition1(variant, d, bits):
    rng = np.random.default_rng(2)
    n_sets = 3
    rot = workloads.rotation_draws(variant, d, n_sets, seed=5)
    c = oracle.codebook(bits, d)
    idx, rho = _keys(rng, 40, d, bits)
    q = rng.standard_normal((2, d))
    per = oracle.raw_params_per_set(variant, d)
    for set_index in range(n_sets):
        s = oracle.attention_scores(variant, d, bits, rot, c, q, idx, rho, 0.5, set_index=set_index)
        rot_s = rot[set_index * per:(set_index + 1) * per]
        qt = np.stack([oracle.encode(variant, d, rot_s, qg) for qg in q])
        ref = 0.5 * (qt @ c[idx].T) * rho[None, :]
        np.testing.assert_allclose(s, ref, rtol=1e-12, atol=1e-13)
    # a different set gives different logits (the set index is honoured)
    s0 = oracle.attention_scores(variant, d, bits, rot, c, q, idx, rho, 0.5, set_index=0)
    s1 = oracle.attention_scores(variant, d, bits, rot, c, q, idx, rho, 0.5, set_index=1)
    assert np.abs(s0 - s1).max() > 1e-3


@pytest.mark.parametrize("variant", ["full", "fast"])
def test_d4_logit_through_explicit_matrix(variant):
    """One quaternion block: dequantized key = rho * M^T c[idx] with M the
    sandwich's 4 x 4 matrix built from the standard basis."""
    d, bits = 4, 3
    rng = np.random.default_rng(3)
    rot = workloads.rotation_draws(variant, d, 1, seed=9)
    c = oracle.codebook(bits, d)
    M = np.stack([oracle.encode(variant, d, rot, e) for e in np.eye(4)], axis=1)
    np.testing.assert_allclose(M.T @ M, np.eye(4), atol=1e-14)
    idx, rho = _keys(rng, 30, d, bits)
    q = rng.standard_normal(d)
    s = oracle.attention_scores(variant, d, bits, rot, c, q, idx, rho, 1.0)
    ref = np.array([r * q @ (M.T @ c[i]) for i, r in zip(idx, rho)])
    np.testing.assert_allclose(s, ref, rtol=1e-13, atol=1e-15)
