"""Seeded synthetic inputs shared by the tests, the smoke check and the benchmark.

This module holds random draws and input recipes only, none of the method's
arithmetic: it produces raw (unnormalised) quaternion draws u ~ N(0, I_4),
raw planar angles theta ~ U[0, 2 pi), raw 8x8 Gaussian matrices for 8-D
blocks (not orthonormalised), and unit-norm Gaussian input rows.  Both
the oracle and the HIP library normalise and use the draws on their own.

Rotation draws use Philox4x32-10 (Salmon, Moraes, Dror and Shaw, "Parallel
random numbers: as easy as 1, 2, 3", SC 2011) as a counter-based generator and
the Box-Muller transform, with this counter layout (the HIP library's seeded
initialisation implements the same definition independently):

    key     = (seed mod 2^32, seed div 2^32)
    counter = (block, set, stream, 0), stream 0 = u_L, 1 = u_R, 2 = angle
              (and (column group, row, 3, 0) for the stage-2 projection,
              (block, set, 4, q) for entries 4q .. 4q + 3 of the raw
              row-major 8x8 matrix of an 8-D block, q = 0 .. 15)
    u       = (z0, z1, z2, z3) with (z0, z1) = BM(w0, w1), (z2, z3) = BM(w2, w3)
    BM(a, b) = sqrt(-2 ln U1) * (cos 2 pi U2, sin 2 pi U2),
               U1 = (a + 0.5) / 2^32, U2 = b / 2^32
    theta   = 2 pi * w0 / 2^32

Input rows use numpy's PCG64 stream: i.i.d. N(0, 1) rows scaled to unit norm
(the paper's synthetic normalised vectors), then rounded to the I/O dtype.
"""
from __future__ import annotations

import numpy as np

PHILOX_M0 = 0xD2511F53
PHILOX_M1 = 0xCD9E8D57
PHILOX_W0 = 0x9E3779B9
PHILOX_W1 = 0xBB67AE85
_MASK32 = np.uint64(0xFFFFFFFF)

FULL, FAST, PLANAR2D, BLOCK8 = 0, 1, 2, 3
_VARIANTS = {"full": FULL, "fast": FAST, "2d": PLANAR2D, "8d": BLOCK8}


def variant_id(v) -> int:
    return _VARIANTS[v] if isinstance(v, str) else int(v)


def philox4x32_10(counter, key):
    """Philox4x32 with 10 rounds, vectorised.  counter: [..., 4], key: [..., 2]
    (uint32-valued integer arrays).  Returns uint32 array [..., 4]."""
    c = np.asarray(counter, dtype=np.uint64) & _MASK32
    k = np.asarray(key, dtype=np.uint64) & _MASK32
    c0, c1, c2, c3 = c[..., 0], c[..., 1], c[..., 2], c[..., 3]
    k0 = np.broadcast_to(k[..., 0], c0.shape).copy()
    k1 = np.broadcast_to(k[..., 1], c0.shape).copy()
    for r in range(10):
        if r:
            k0 = (k0 + np.uint64(PHILOX_W0)) & _MASK32
            k1 = (k1 + np.uint64(PHILOX_W1)) & _MASK32
        p0 = np.uint64(PHILOX_M0) * c0
        p1 = np.uint64(PHILOX_M1) * c2
        hi0, lo0 = p0 >> np.uint64(32), p0 & _MASK32
        hi1, lo1 = p1 >> np.uint64(32), p1 & _MASK32
        c0, c1, c2, c3 = (hi1 ^ c1 ^ k0), lo1, (hi0 ^ c3 ^ k1), lo0
    return np.stack([c0, c1, c2, c3], axis=-1).astype(np.uint32)


def _key(seed: int):
    seed = int(seed) & 0xFFFFFFFFFFFFFFFF
    return np.array([seed & 0xFFFFFFFF, seed >> 32], dtype=np.uint64)


def _box_muller(a, b):
    u1 = (a.astype(np.float64) + 0.5) * 2.0 ** -32
    u2 = b.astype(np.float64) * 2.0 ** -32
    r = np.sqrt(-2.0 * np.log(u1))
    return r * np.cos(2.0 * np.pi * u2), r * np.sin(2.0 * np.pi * u2)


def philox_gaussian4(blocks, sets, stream, seed, word3=0):
    """Four N(0,1) draws per counter (block, set, stream, word3): array [..., 4]
    float64."""
    blocks, sets, word3 = np.broadcast_arrays(np.asarray(blocks, np.uint64), np.asarray(sets, np.uint64),
                                              np.asarray(word3, np.uint64))
    ctr = np.stack([blocks, sets, np.full_like(blocks, stream), word3], axis=-1)
    w = philox4x32_10(ctr, _key(seed))
    z0, z1 = _box_muller(w[..., 0], w[..., 1])
    z2, z3 = _box_muller(w[..., 2], w[..., 3])
    return np.stack([z0, z1, z2, z3], axis=-1)


def raw_params_per_set(variant, d: int) -> int:
    v = variant_id(variant)
    if v == PLANAR2D:
        return (d + 1) // 2
    if v == BLOCK8:
        return 64 * ((d + 7) // 8)
    g = (d + 3) // 4
    return 8 * g if v == FULL else 4 * g


def rotation_draws(variant, d: int, n_sets: int = 1, seed: int = 1) -> np.ndarray:
    """Raw rotation draws, flat float64 array [n_sets * raw_params_per_set].

    Full: per set, per block i: (u_L[0..3], u_R[0..3]); Fast: u_L[0..3];
    2-D: one angle theta per coordinate pair; 8-D: per set, per block of 8
    coordinates, a raw 8x8 N(0, 1) matrix, row-major.
    """
    v = variant_id(variant)
    if v == BLOCK8:
        g8 = (d + 7) // 8
        s, b, q = np.meshgrid(np.arange(n_sets), np.arange(g8), np.arange(16), indexing="ij")
        return philox_gaussian4(b, s, 4, seed, q).reshape(-1)   # [n_sets, g8, 16 x 4]
    if v == PLANAR2D:
        g2 = (d + 1) // 2
        b, s = np.meshgrid(np.arange(g2), np.arange(n_sets))
        ctr = np.stack([b, s, np.full_like(b, 2), np.zeros_like(b)], axis=-1).astype(np.uint64)
        w = philox4x32_10(ctr, _key(seed))
        theta = 2.0 * np.pi * w[..., 0].astype(np.float64) * 2.0 ** -32
        return theta.reshape(-1)
    g = (d + 3) // 4
    b, s = np.meshgrid(np.arange(g), np.arange(n_sets))
    uL = philox_gaussian4(b, s, 0, seed)                  # [n_sets, g, 4]
    if v == FAST:
        return uL.reshape(-1)
    uR = philox_gaussian4(b, s, 1, seed)
    return np.concatenate([uL, uR], axis=-1).reshape(-1)  # [n_sets, g, 8]


def qjl_matrix(m: int, d: int, seed: int = 7) -> np.ndarray:
    """The stage-2 projection S, [m, d] i.i.d. N(0, 1): S[i, 4g:4g+4] is the
    Philox/Box-Muller quadruple of counter (g, i, 3, 0) (stream 3; the HIP
    library's seeded sketch implements the same definition independently)."""
    g4 = (d + 3) // 4
    g, i = np.meshgrid(np.arange(g4), np.arange(m))
    return philox_gaussian4(g, i, 3, seed).reshape(m, 4 * g4)[:, :d].copy()


def unit_gaussian_rows(n: int, d: int, seed: int = 0, dtype=np.float16, chunk: int = 1 << 16):
    """n i.i.d. N(0, I_d) rows scaled to unit norm, rounded to ``dtype``."""
    rng = np.random.default_rng(seed)
    out = np.empty((n, d), dtype=dtype)
    for s in range(0, n, chunk):
        e = min(n, s + chunk)
        z = rng.standard_normal((e - s, d))
        z /= np.linalg.norm(z, axis=1, keepdims=True)
        out[s:e] = z.astype(dtype)
    return out


def kv_stream_torch(batch: int, heads: int, tokens: int, d: int, seed: int, device, dtype=None,
                    corr: float = 0.9):
    """KV-cache-shaped rows [batch, heads, tokens, d]: per (batch, head) an AR(1)
    Gaussian sequence over tokens, g_0 = e_0, g_t = corr g_{t-1} + sqrt(1-corr^2) e_t
    with e_t ~ N(0, I_d), each row then scaled to unit norm.  Drawn with torch's
    seeded generator on ``device`` (a 2-GiB fp16 tensor at the full shape); the
    recurrence is evaluated by a doubling scan, which is exact in real
    arithmetic for a constant coefficient."""
    import torch

    dtype = dtype or torch.float16
    gen = torch.Generator(device=device)
    gen.manual_seed(int(seed))
    out = torch.empty((batch, heads, tokens, d), dtype=dtype, device=device)
    a = float(corr)
    c = float(np.sqrt(1.0 - corr * corr))
    for b in range(batch):
        e = torch.randn((heads, tokens, d), generator=gen, device=device, dtype=torch.float32)
        e[:, 1:] *= c
        step = 1
        coef = a
        while step < tokens:
            e[:, step:] += coef * e[:, :-step].clone()
            coef *= coef
            step *= 2
        e /= torch.linalg.vector_norm(e, dim=-1, keepdim=True)
        out[b] = e.to(dtype)
    return out
