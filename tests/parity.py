"""Comparison of the HIP path against the oracle (shared by the GPU tests).

Rule (per coordinate): the GPU index must equal the oracle's, except where the
oracle's rotated normalised coordinate lies within BAND of a decision
threshold; there the GPU may take either neighbouring cell.  Reconstructions
are compared per row by relative L2 error: fp32 rows within 1e-5, fp16 rows
within 2e-3.  A row with a near-threshold coordinate must match one of the
oracle's own reconstructions over the admissible cells of those coordinates
(the alternatives come from the oracle's values and thresholds, never from
the GPU's output).
"""
import itertools

import numpy as np

import oracle

BAND = 1e-6
TOL = {np.dtype(np.float32): 1e-5, np.dtype(np.float16): 2e-3}
MIN_AGREEMENT = 0.9999


def _admissible(yt, thr, idx_o):
    """Per coordinate: (near?, low cell, high cell) around the closest threshold."""
    dist = np.abs(yt[..., None] - thr)
    k = dist.argmin(-1)
    near = dist.min(-1) <= BAND
    return near, k, k + 1


def rel_err(a, b):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    num = np.linalg.norm(a - b, axis=-1)
    den = np.linalg.norm(b, axis=-1)
    return np.where(den > 0, num / np.where(den > 0, den, 1), num)


class Oracle:
    """Oracle results for selected rows of one workload."""

    def __init__(self, variant, d, bits, rot, levels, x, n_sets=1, rows_per_set=1, rows=None,
                 selected=False):
        self.variant, self.d, self.bits = variant, d, bits
        self.rot, self.levels = rot, levels
        self.n_sets, self.rps = n_sets, rows_per_set
        self.rows = None if rows is None else np.asarray(rows, np.int64)
        self.idx, self.rho, self.xh, self.yt = oracle.stage1(
            variant, d, bits, rot, levels, x, n_sets=n_sets, rows_per_set=rows_per_set,
            rows=self.rows, want_ytil=True, selected=selected)
        self.thr = oracle.thresholds(bits, levels)
        self.near, self.k_lo, self.k_hi = _admissible(self.yt, self.thr, self.idx)

    def row_numbers(self):
        return np.arange(len(self.rho)) if self.rows is None else self.rows

    def check_indices(self, idx_gpu):
        """idx_gpu: [m, d] unpacked GPU indices for the same rows."""
        idx_gpu = np.asarray(idx_gpu)
        same = idx_gpu == self.idx
        far_bad = ~same & ~self.near
        assert not far_bad.any(), (
            f"{int(far_bad.sum())} index mismatches away from a threshold, first at "
            f"{np.argwhere(far_bad)[:5].tolist()}")
        near_ok = (idx_gpu == self.k_lo) | (idx_gpu == self.k_hi)
        assert np.all(near_ok | same), "near-threshold index outside the two admissible cells"
        agree = same.mean()
        assert agree >= MIN_AGREEMENT, agree
        return agree

    def check_norms(self, rho_gpu):
        rho_gpu = np.asarray(rho_gpu, np.float64)
        err = np.abs(rho_gpu - self.rho)
        assert np.all(err <= 1e-6 * self.rho + 1e-30), err.max()

    def _candidates(self, r):
        """Oracle reconstructions of row r over the admissible cells of its
        near-threshold coordinates."""
        js = np.flatnonzero(self.near[r])
        if len(js) > 6:
            raise AssertionError(f"row {r}: {len(js)} near-threshold coordinates")
        out = []
        for choice in itertools.product(*[(self.k_lo[r, j], self.k_hi[r, j]) for j in js]):
            idx = self.idx[r].copy()
            idx[js] = choice
            row_no = self.row_numbers()[r]
            # dequantize with the row's true set: build a one-row call at that row number
            s = 0 if self.n_sets <= 1 else (row_no // self.rps) % self.n_sets
            per = oracle.raw_params_per_set(self.variant, self.d)
            rot_s = np.asarray(self.rot).reshape(-1)[s * per:(s + 1) * per]
            out.append(oracle.dequantize(self.variant, self.d, self.bits, rot_s, self.levels,
                                         idx[None], self.rho[r:r + 1])[0])
        return out

    def check_xhat(self, xh_gpu, dtype):
        """Per-row relative error against the oracle (with near-threshold rows
        matched against their admissible alternatives)."""
        tol = TOL[np.dtype(dtype)]
        xh_gpu = np.asarray(xh_gpu, np.float64)
        err = rel_err(xh_gpu, self.xh)
        has_near = self.near.any(-1)
        bad = (err > tol) & ~has_near
        assert not bad.any(), f"{int(bad.sum())} rows beyond {tol}; worst {err[bad].max()}"
        for r in np.flatnonzero(has_near & (err > tol)):
            errs = [rel_err(xh_gpu[r], c) for c in self._candidates(r)]
            assert min(errs) <= tol, (r, errs)
        return float(err[~has_near].max()) if (~has_near).any() else 0.0
