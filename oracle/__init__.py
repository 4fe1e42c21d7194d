"""Python access to the IsoQuant stage-1 oracle (``isoq_oracle.c``).

TEST INFRASTRUCTURE ONLY: the test suite, the smoke check and the benchmark's
CPU-baseline leg may use this package; the product path never does.  The
oracle shares no code with the HIP library.  This wrapper only marshals
arguments (numpy arrays in, numpy arrays out) and widens inputs to float64,
which is exact for fp16 and fp32 values.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "isoq_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

FULL, FAST, PLANAR2D, BLOCK8 = 0, 1, 2, 3
VARIANTS = {"full": FULL, "fast": FAST, "2d": PLANAR2D, "8d": BLOCK8}


def build() -> str:
    """Compile the oracle with gcc (IEEE double, no FMA contraction)."""
    tmp = _LIB + ".tmp"
    cmd = ["gcc", "-O2", "-std=gnu11", "-ffp-contract=off", "-fno-fast-math",
           "-fPIC", "-shared", _SRC, "-o", tmp, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, _LIB)
    return _LIB


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
            build()
        L = ctypes.CDLL(_LIB)
        dp = ctypes.POINTER(ctypes.c_double)
        u8p = ctypes.POINTER(ctypes.c_uint8)
        i64 = ctypes.c_int64
        L.orc_qmul.argtypes = [dp, dp, dp]
        L.orc_qconj.argtypes = [dp, dp]
        L.orc_qnormalize.argtypes = [dp, dp]
        L.orc_full_forward.argtypes = [dp, dp, dp, dp]
        L.orc_full_inverse.argtypes = [dp, dp, dp, dp]
        L.orc_fast_forward.argtypes = [dp, dp, dp]
        L.orc_fast_inverse.argtypes = [dp, dp, dp]
        L.orc_planar_forward.argtypes = [ctypes.c_double, dp, dp]
        L.orc_planar_inverse.argtypes = [ctypes.c_double, dp, dp]
        L.orc_det8.argtypes = [dp]
        L.orc_det8.restype = ctypes.c_double
        L.orc_orthonormalize8.argtypes = [dp, dp]
        L.orc_orthonormalize8.restype = ctypes.c_int
        L.orc_block8_forward.argtypes = [dp, dp, dp]
        L.orc_block8_inverse.argtypes = [dp, dp, dp]
        L.orc_thresholds.argtypes = [ctypes.c_int, dp, dp]
        L.orc_lloyd_max_gaussian.argtypes = [ctypes.c_int, ctypes.c_double, ctypes.c_int, dp]
        L.orc_lloyd_max_gaussian.restype = ctypes.c_int
        L.orc_num_blocks.argtypes = [ctypes.c_int, ctypes.c_int]
        L.orc_raw_params_per_set.argtypes = [ctypes.c_int, ctypes.c_int]
        L.orc_table1_params.argtypes = [ctypes.c_int, ctypes.c_int]
        L.orc_encode.argtypes = [ctypes.c_int, ctypes.c_int, dp, dp, dp]
        L.orc_decode.argtypes = [ctypes.c_int, ctypes.c_int, dp, dp, dp]
        L.orc_stage1.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int, i64,
                                 dp, dp, dp, i64, i64, u8p, dp, dp, dp]
        L.orc_stage1.restype = ctypes.c_int
        L.orc_stage1_rows.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int, i64,
                                      dp, dp, ctypes.POINTER(ctypes.c_int64), i64, dp, u8p, dp, dp,
                                      dp]
        L.orc_stage1_rows.restype = ctypes.c_int
        L.orc_dequantize.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int, i64,
                                     dp, dp, u8p, dp, i64, i64, dp]
        L.orc_dequantize.restype = ctypes.c_int
        L.orc_record_bytes.argtypes = [ctypes.c_int, ctypes.c_int]
        L.orc_record_bytes.restype = i64
        L.orc_pack.argtypes = [u8p, i64, ctypes.c_int, ctypes.c_int, u8p]
        L.orc_unpack.argtypes = [u8p, i64, ctypes.c_int, ctypes.c_int, u8p]
        L.orc_mul_count.restype = ctypes.c_uint64
        _lib = L
    return _lib


def _d(a):
    return np.ascontiguousarray(a, dtype=np.float64)


def _p(a, t=ctypes.c_double):
    return a.ctypes.data_as(ctypes.POINTER(t))


def _variant(v) -> int:
    return VARIANTS[v] if isinstance(v, str) else int(v)


# --- quaternion algebra (Sec. 4) ---------------------------------------------
def qmul(p, q):
    p, q, out = _d(p), _d(q), np.zeros(4)
    lib().orc_qmul(_p(p), _p(q), _p(out))
    return out


def qconj(q):
    q, out = _d(q), np.zeros(4)
    lib().orc_qconj(_p(q), _p(out))
    return out


def qnormalize(u):
    u, out = _d(u), np.zeros(4)
    lib().orc_qnormalize(_p(u), _p(out))
    return out


def full_forward(qL, qR, v):
    qL, qR, v, out = _d(qL), _d(qR), _d(v), np.zeros(4)
    lib().orc_full_forward(_p(qL), _p(qR), _p(v), _p(out))
    return out


def full_inverse(qL, qR, v):
    qL, qR, v, out = _d(qL), _d(qR), _d(v), np.zeros(4)
    lib().orc_full_inverse(_p(qL), _p(qR), _p(v), _p(out))
    return out


def fast_forward(qL, v):
    qL, v, out = _d(qL), _d(v), np.zeros(4)
    lib().orc_fast_forward(_p(qL), _p(v), _p(out))
    return out


def fast_inverse(qL, v):
    qL, v, out = _d(qL), _d(v), np.zeros(4)
    lib().orc_fast_inverse(_p(qL), _p(v), _p(out))
    return out


def planar_forward(theta, u):
    u, out = _d(u), np.zeros(2)
    lib().orc_planar_forward(float(theta), _p(u), _p(out))
    return out


def planar_inverse(theta, u):
    u, out = _d(u), np.zeros(2)
    lib().orc_planar_inverse(float(theta), _p(u), _p(out))
    return out


# --- 8-D grouped blocks (Table 3; Sec. 5.7 with k = 8) ---------------------------
def det8(M):
    """Determinant of an 8x8 matrix (Gaussian elimination, partial pivoting)."""
    M = _d(np.asarray(M).reshape(8, 8))
    return float(lib().orc_det8(_p(M)))


def orthonormalize8(G):
    """The block rotation of a raw 8x8 draw G: Gram-Schmidt Q of G's columns
    (G = QR, diag R > 0), with column 0 negated when det Q = -1.  [8, 8]."""
    G = _d(np.asarray(G).reshape(8, 8))
    Q = np.zeros((8, 8))
    if lib().orc_orthonormalize8(_p(G), _p(Q)) != 0:
        raise ValueError("linearly dependent columns")
    return Q


def block8_forward(G, v):
    G, v, out = _d(np.asarray(G).reshape(8, 8)), _d(v), np.zeros(8)
    lib().orc_block8_forward(_p(G), _p(v), _p(out))
    return out


def block8_inverse(G, y):
    G, y, out = _d(np.asarray(G).reshape(8, 8)), _d(y), np.zeros(8)
    lib().orc_block8_inverse(_p(G), _p(y), _p(out))
    return out


# --- codebook ------------------------------------------------------------------
def lloyd_max_gaussian(bits: int, sigma: float, iters: int = 200) -> np.ndarray:
    out = np.zeros(1 << bits)
    rc = lib().orc_lloyd_max_gaussian(int(bits), float(sigma), int(iters), _p(out))
    if rc != 0:
        raise ValueError("bad codebook arguments")
    return out


def codebook(bits: int, d: int, iters: int = 200) -> np.ndarray:
    """Lloyd-Max levels for N(0, 1/d) (the reading used for every workload)."""
    return lloyd_max_gaussian(bits, 1.0 / np.sqrt(d), iters)


def thresholds(bits: int, levels) -> np.ndarray:
    levels = _d(levels)
    out = np.zeros((1 << bits) - 1)
    lib().orc_thresholds(int(bits), _p(levels), _p(out))
    return out


# --- geometry / counts -----------------------------------------------------------
def num_blocks(variant, d: int) -> int:
    return lib().orc_num_blocks(_variant(variant), int(d))


def raw_params_per_set(variant, d: int) -> int:
    return lib().orc_raw_params_per_set(_variant(variant), int(d))


def table1_params(variant, d: int) -> int:
    return lib().orc_table1_params(_variant(variant), int(d))


def block_width(variant) -> int:
    v = _variant(variant)
    return 2 if v == PLANAR2D else 8 if v == BLOCK8 else 4


def padded_width(variant, d: int) -> int:
    return num_blocks(variant, d) * block_width(variant)


def mul_count_reset():
    lib().orc_mul_count_reset()


def mul_count() -> int:
    return int(lib().orc_mul_count())


def encode(variant, d, rot, xbar):
    v = _variant(variant)
    rot, xbar = _d(rot), _d(xbar)
    out = np.zeros(padded_width(v, d))
    lib().orc_encode(v, int(d), _p(rot), _p(xbar), _p(out))
    return out


def decode(variant, d, rot, yhat):
    v = _variant(variant)
    rot, yhat = _d(rot), _d(yhat)
    out = np.zeros(int(d))
    lib().orc_decode(v, int(d), _p(rot), _p(yhat), _p(out))
    return out


# --- Algorithm 1 -------------------------------------------------------------------
def stage1(variant, d: int, bits: int, rot, levels, x, n_sets: int = 1, rows_per_set: int = 1,
           rows=None, want_idx=True, want_xhat=True, want_ytil=False, selected=False):
    """Run Algorithm 1 on rows of ``x`` ([n, d], any float dtype).

    ``rows`` optionally selects a subset (array of row numbers); the set of a
    row is computed from its global row number.  With ``selected``, ``x`` holds
    just those rows, in that order.  Returns (idx, rho, xhat) for the selected
    rows, plus ytil (rotated normalised coordinates before Q) when
    ``want_ytil``; idx and ytil have ``padded_width`` columns.
    """
    v = _variant(variant)
    rot = _d(rot)
    levels = _d(levels)
    x = np.asarray(x)
    pw = padded_width(v, d)
    L = lib()
    if rows is None:
        xs = _d(x.reshape(-1, d))
    else:
        rows = np.ascontiguousarray(rows, dtype=np.int64)
        xs = _d(x.reshape(-1, d)) if selected else _d(x.reshape(-1, d)[rows])
        if xs.shape[0] != len(rows):
            raise ValueError("selected rows and row numbers differ in count")
    m = xs.shape[0]
    idx = np.zeros((m, pw), np.uint8) if want_idx else None
    rho = np.zeros(m)
    xh = np.zeros((m, d)) if want_xhat else None
    yt = np.zeros((m, pw)) if want_ytil else None
    opt = lambda a, t=ctypes.c_double: _p(a, t) if a is not None else None
    if rows is None:
        rc = L.orc_stage1(v, d, bits, n_sets, rows_per_set, _p(rot), _p(levels), _p(xs), 0, m,
                          opt(idx, ctypes.c_uint8), _p(rho), opt(xh), opt(yt))
    else:
        rc = L.orc_stage1_rows(v, d, bits, n_sets, rows_per_set, _p(rot), _p(levels),
                               _p(rows, ctypes.c_int64), m, _p(xs), opt(idx, ctypes.c_uint8),
                               _p(rho), opt(xh), opt(yt))
    if rc != 0:
        raise ValueError("the oracle rejected its arguments")
    return (idx, rho, xh, yt) if want_ytil else (idx, rho, xh)


def stage1_range(variant, d, bits, rot, levels, xd, row_begin, row_end, n_sets=1, rows_per_set=1,
                 idx=None, rho=None, xh=None):
    """Low-level entry used by the CPU baseline: rows [row_begin, row_end) of a
    float64 [n, d] array, writing into preallocated outputs (ctypes releases
    the GIL, so several Python threads can split the rows)."""
    v = _variant(variant)
    return lib().orc_stage1(v, d, bits, n_sets, rows_per_set, _p(rot), _p(levels), _p(xd),
                            int(row_begin), int(row_end),
                            _p(idx, ctypes.c_uint8) if idx is not None else None,
                            _p(rho), _p(xh) if xh is not None else None, None)


def dequantize(variant, d: int, bits: int, rot, levels, idx, rho, n_sets: int = 1,
               rows_per_set: int = 1):
    v = _variant(variant)
    rot, levels, rho = _d(rot), _d(levels), _d(rho)
    idx = np.ascontiguousarray(idx, dtype=np.uint8)
    n = rho.shape[0]
    xh = np.zeros((n, d))
    rc = lib().orc_dequantize(v, d, bits, n_sets, rows_per_set, _p(rot), _p(levels),
                              _p(idx, ctypes.c_uint8), _p(rho), 0, n, _p(xh))
    if rc != 0:
        raise ValueError("orc_dequantize rejected its arguments")
    return xh


# --- attention logits against quantized keys --------------------------------------
def attention_scores(variant, d: int, bits: int, rot, levels, q, idx, rho, scale: float = 1.0,
                     set_index: int = 0):
    """Attention logits of queries against quantized keys, by definition:
    s[g, t] = scale * <q_g, xhat_t>, where xhat_t = rho_t * T^{-1}(c[idx_t]) is
    the oracle's dequantization (Algorithm 1, last steps) of key t with the
    rotation set ``set_index``.  q: [G, d] (or [d]); idx: unpacked [n, padded]
    indices; rho: [n].  Returns float64 [G, n] (or [n])."""
    v = _variant(variant)
    per = raw_params_per_set(v, d)
    rot_s = _d(rot).reshape(-1)[set_index * per:(set_index + 1) * per]
    xh = dequantize(v, d, bits, rot_s, levels, idx, rho)
    qd = _d(q)
    return scale * (qd @ xh.T)


# --- stage 2: QJL residual sketch (Sec. 8) ------------------------------------------
def qjl_encode(variant, d: int, bits: int, rot, levels, S, x, n_sets: int = 1, rows_per_set: int = 1):
    """Stage-2 sketch of the stage-1 residual, by definition (Sec. 8 keeps
    TurboQuant's residual correction: r = x - x_hat, projected by a quantized
    Johnson-Lindenstrauss transform): with S [m, d] Gaussian,
        z_i = [ (S r)_i > 0 ],  gamma = ||r||.
    Returns (z [n, m] uint8 in {0, 1}, gamma [n], p = S r [n, m], idx, rho,
    x_hat) in float64."""
    idx, rho, xh = stage1(variant, d, bits, rot, levels, x, n_sets=n_sets, rows_per_set=rows_per_set)
    r = _d(x).reshape(-1, d) - xh
    p = r @ _d(S).T
    z = (p > 0).astype(np.uint8)
    return z, np.linalg.norm(r, axis=1), p, idx, rho, xh


def qjl_inner_product(q, xhat, z, gamma, S):
    """Two-stage inner-product estimate of <q, x> (TurboQuant's product
    estimator, QJL on the residual): <q, x_hat> + sqrt(pi/2)/m * gamma *
    <S q, 2 z - 1>.  q: [d] or [G, d]; xhat [n, d]; z [n, m]; gamma [n].
    Returns [n] or [G, n]."""
    S = _d(S)
    m = S.shape[0]
    qd = _d(q)
    sq = qd @ S.T                                    # [.., m]
    signs = 2.0 * np.asarray(z, np.float64) - 1.0    # [n, m]
    return qd @ _d(xhat).T + np.sqrt(np.pi / 2.0) / m * (sq @ signs.T) * _d(gamma)


# --- packing -------------------------------------------------------------------------
def record_bytes(m: int, bits: int) -> int:
    return int(lib().orc_record_bytes(int(m), int(bits)))


def pack(idx, bits: int) -> np.ndarray:
    idx = np.ascontiguousarray(idx, dtype=np.uint8)
    n, m = idx.shape
    out = np.zeros((n, record_bytes(m, bits)), np.uint8)
    lib().orc_pack(_p(idx, ctypes.c_uint8), n, m, bits, _p(out, ctypes.c_uint8))
    return out


def unpack(packed, m: int, bits: int) -> np.ndarray:
    packed = np.ascontiguousarray(packed, dtype=np.uint8)
    n = packed.shape[0]
    out = np.zeros((n, m), np.uint8)
    lib().orc_unpack(_p(packed, ctypes.c_uint8), n, m, bits, _p(out, ctypes.c_uint8))
    return out
