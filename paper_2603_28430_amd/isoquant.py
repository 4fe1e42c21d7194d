"""Python binding of libisoquant.so (declared in include/isoquant.h).

Argument marshalling only: every step of the quantize/dequantize path runs in
the library's HIP kernels.  PyTorch provides device memory and streams; tensors
are passed as raw device pointers together with the current HIP stream.  The
functions carry the C names; device outputs are allocated here when the caller
does not pass them.  A missing library is an ImportError, never a fallback.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libisoquant.so")

ISOQ_FULL, ISOQ_FAST, ISOQ_PLANAR2D, ISOQ_BLOCK8 = 0, 1, 2, 3
ISOQ_F32, ISOQ_F16 = 0, 1
VARIANTS = {"full": ISOQ_FULL, "fast": ISOQ_FAST, "2d": ISOQ_PLANAR2D, "8d": ISOQ_BLOCK8}

STATUS = {0: "ISOQ_OK", 1: "ISOQ_E_INVALID", 2: "ISOQ_E_UNSUPPORTED", 3: "ISOQ_E_NULL",
          4: "ISOQ_E_ALIGN", 5: "ISOQ_E_HIP", 6: "ISOQ_E_NOMEM", 7: "ISOQ_E_DEVICE"}


class IsoqError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        detail = lib.isoq_last_hip_error().decode() if status in (5, 6) else ""
        super().__init__(f"{where}: {STATUS.get(status, status)} ({isoq_status_string(status)})"
                         + (f" [{detail}]" if detail else ""))


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run `python paper_2603_28430_amd/build.py`")
    # PyTorch ships its own HIP runtime (same soname).  Loading torch first
    # makes the library bind to that runtime instead of a second copy, which
    # would not see the GPU that torch has already opened.
    try:
        import torch  # noqa: F401
    except ImportError:
        pass
    L = ctypes.CDLL(LIB_PATH)
    vp, dp, fp, i64 = ctypes.c_void_p, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_float), ctypes.c_int64
    c_int = ctypes.c_int
    L.isoq_params_init.argtypes = [ctypes.POINTER(vp), c_int, c_int, c_int, c_int, dp, dp, ctypes.c_uint64]
    L.isoq_params_destroy.argtypes = [vp]
    L.isoq_params_export.argtypes = [vp, fp, fp, fp]
    L.isoq_params_info.argtypes = [vp] + [ctypes.POINTER(c_int)] * 4
    L.isoq_quantize.argtypes = [vp, c_int, vp, i64, i64, vp, vp, vp]
    L.isoq_dequantize.argtypes = [vp, c_int, vp, vp, i64, i64, vp, vp]
    L.isoq_roundtrip.argtypes = [vp, c_int, vp, i64, i64, vp, vp]
    L.isoq_kv_append.argtypes = [vp, vp, c_int, vp, vp, vp, i64, c_int, vp, vp, vp, vp, i64, c_int, vp]
    L.isoq_sketch_init.argtypes = [ctypes.POINTER(vp), vp, c_int, dp, ctypes.c_uint64]
    L.isoq_sketch_destroy.argtypes = [vp]
    L.isoq_sketch_export.argtypes = [vp, ctypes.POINTER(c_int), fp]
    L.isoq_quantize_qjl.argtypes = [vp, vp, c_int, vp, i64, i64, vp, vp, vp, vp, vp]
    L.isoq_kv_append_qjl.argtypes = [vp, vp, c_int, vp, vp, i64, c_int, vp, vp, vp, vp, i64, c_int, vp]
    L.isoq_kv_scores_qjl.argtypes = [vp, vp, c_int, vp, c_int, c_int, c_int, vp, vp, vp, vp, i64, c_int, vp, c_int,
                                     vp, ctypes.c_float, vp, i64, vp]
    L.isoq_kv_scores.argtypes = [vp, c_int, vp, c_int, c_int, c_int, vp, vp, i64, c_int, vp, c_int, vp,
                                 ctypes.c_float, vp, i64, vp]
    L.isoq_packed_bytes.argtypes = [c_int, c_int]
    L.isoq_packed_bytes.restype = ctypes.c_size_t
    L.isoq_record_bytes.argtypes = [c_int, c_int, c_int]
    L.isoq_record_bytes.restype = ctypes.c_size_t
    L.isoq_raw_params_per_set.argtypes = [c_int, c_int]
    L.isoq_raw_params_per_set.restype = ctypes.c_size_t
    L.isoq_export_params_per_set.argtypes = [c_int, c_int]
    L.isoq_export_params_per_set.restype = ctypes.c_size_t
    L.isoq_codebook_lloyd.argtypes = [c_int, c_int, c_int, dp]
    L.isoq_rotation_draws.argtypes = [c_int, c_int, c_int, ctypes.c_uint64, dp]
    L.isoq_status_string.argtypes = [c_int]
    L.isoq_status_string.restype = ctypes.c_char_p
    L.isoq_last_hip_error.argtypes = []
    L.isoq_last_hip_error.restype = ctypes.c_char_p
    for f in ("isoq_params_init", "isoq_params_destroy", "isoq_params_export", "isoq_params_info",
              "isoq_quantize", "isoq_dequantize", "isoq_roundtrip", "isoq_kv_append", "isoq_kv_scores", "isoq_sketch_init",
              "isoq_sketch_destroy", "isoq_sketch_export", "isoq_quantize_qjl", "isoq_kv_scores_qjl",
              "isoq_codebook_lloyd",
              "isoq_rotation_draws"):
        getattr(L, f).restype = c_int
    return L


lib = _load()


def _check(st: int, where: str):
    if st != 0:
        raise IsoqError(st, where)


def _variant(v) -> int:
    return VARIANTS[v] if isinstance(v, str) else int(v)


def isoq_status_string(status: int) -> str:
    return lib.isoq_status_string(int(status)).decode()


def isoq_packed_bytes(d: int, bits: int) -> int:
    return int(lib.isoq_packed_bytes(int(d), int(bits)))


def isoq_record_bytes(variant, d: int, bits: int) -> int:
    return int(lib.isoq_record_bytes(_variant(variant), int(d), int(bits)))


def isoq_raw_params_per_set(variant, d: int) -> int:
    return int(lib.isoq_raw_params_per_set(_variant(variant), int(d)))


def isoq_export_params_per_set(variant, d: int) -> int:
    return int(lib.isoq_export_params_per_set(_variant(variant), int(d)))


def isoq_codebook_lloyd(bits: int, d: int, iters: int = 200) -> np.ndarray:
    out = np.zeros(1 << bits)
    _check(lib.isoq_codebook_lloyd(int(bits), int(d), int(iters),
                                   out.ctypes.data_as(ctypes.POINTER(ctypes.c_double))),
           "isoq_codebook_lloyd")
    return out


def isoq_rotation_draws(variant, d: int, n_sets: int = 1, seed: int = 1) -> np.ndarray:
    v = _variant(variant)
    out = np.zeros(n_sets * isoq_raw_params_per_set(v, d))
    _check(lib.isoq_rotation_draws(v, int(d), int(n_sets), int(seed),
                                   out.ctypes.data_as(ctypes.POINTER(ctypes.c_double))),
           "isoq_rotation_draws")
    return out


class Params:
    """Owner of an isoq_params handle (freed by close() or garbage collection)."""

    def __init__(self, handle: int, variant: int, d: int, bits: int, n_sets: int):
        self.handle = ctypes.c_void_p(handle)
        self.variant, self.d, self.bits, self.n_sets = variant, d, bits, n_sets

    def close(self):
        if self.handle:
            _check(lib.isoq_params_destroy(self.handle), "isoq_params_destroy")
            self.handle = ctypes.c_void_p(None)

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    @property
    def record_bytes(self) -> int:
        return isoq_record_bytes(self.variant, self.d, self.bits)


def isoq_params_init(variant, d: int, bits: int, n_sets: int = 1, rot=None, codebook=None,
                     seed: int = 1) -> Params:
    """Create a handle on the current device (see include/isoquant.h)."""
    v = _variant(variant)
    dp = ctypes.POINTER(ctypes.c_double)
    rot_a = None if rot is None else np.ascontiguousarray(rot, dtype=np.float64)
    cb_a = None if codebook is None else np.ascontiguousarray(codebook, dtype=np.float64)
    if rot_a is not None and rot_a.size != n_sets * isoq_raw_params_per_set(v, d):
        raise ValueError("rot has the wrong number of raw draws")
    if cb_a is not None and cb_a.size != (1 << bits):
        raise ValueError("codebook must have 2**bits levels")
    h = ctypes.c_void_p()
    _check(lib.isoq_params_init(ctypes.byref(h), v, int(d), int(bits), int(n_sets),
                                None if rot_a is None else rot_a.ctypes.data_as(dp),
                                None if cb_a is None else cb_a.ctypes.data_as(dp), int(seed)),
           "isoq_params_init")
    return Params(h.value, v, int(d), int(bits), int(n_sets))


def isoq_params_destroy(p: Params) -> None:
    p.close()


def isoq_params_export(p: Params):
    """(unit rotation parameters [n_sets * per_set], levels [2^b], thresholds [2^b - 1]), fp32."""
    rot = np.zeros(p.n_sets * isoq_export_params_per_set(p.variant, p.d), np.float32)
    lev = np.zeros(1 << p.bits, np.float32)
    thr = np.zeros((1 << p.bits) - 1, np.float32)
    fp = ctypes.POINTER(ctypes.c_float)
    _check(lib.isoq_params_export(p.handle, rot.ctypes.data_as(fp), lev.ctypes.data_as(fp),
                                  thr.ctypes.data_as(fp)), "isoq_params_export")
    return rot, lev, thr


def isoq_params_info(p: Params):
    vals = [ctypes.c_int() for _ in range(4)]
    _check(lib.isoq_params_info(p.handle, *[ctypes.byref(v) for v in vals]), "isoq_params_info")
    return tuple(v.value for v in vals)


# --- device calls ----------------------------------------------------------------
def _torch():
    import torch
    return torch


def _stream_ptr(stream):
    torch = _torch()
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def _dtype_code(t) -> int:
    torch = _torch()
    if t == torch.float16:
        return ISOQ_F16
    if t == torch.float32:
        return ISOQ_F32
    raise TypeError(f"rows must be float16 or float32, got {t}")


def _is_gpu(t) -> bool:
    return t.is_cuda


def _rows(x, d):
    _device_tensors(x, x=x)
    if x.dim() < 1 or x.shape[-1] != d:
        raise ValueError(f"x: last dimension must be d={d}")
    return x.numel() // d


def _like(name, t, dtypes, numel):
    """Type and size of a tensor argument: one of `dtypes`, `numel` elements."""
    torch = _torch()
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.dtype not in dtypes:
        raise TypeError(f"{name} must be {' or '.join(str(d) for d in dtypes)}, got {t.dtype}")
    if t.numel() != numel:
        raise ValueError(f"{name} must hold {numel} elements, got {t.numel()}")


def _device_tensors(ref, **ts):
    """Every tensor a kernel touches: on the GPU, contiguous, on ref's device
    (a pointer of the wrong kind or into the wrong memory would fault the GPU)."""
    for name, t in ts.items():
        if not _is_gpu(t):
            raise ValueError(f"{name} must be on the GPU")
        if not t.is_contiguous():
            raise ValueError(f"{name} must be contiguous")
        if t.device != ref.device:
            raise ValueError(f"{name} must be on {ref.device}, got {t.device}")


def isoq_roundtrip(p: Params, x, rows_per_set: int = 1, x_hat=None, stream=None):
    """x_hat = stage-1 quantize->dequantize of x (same shape and dtype)."""
    n = _rows(x, p.d)
    _dtype_code(x.dtype)
    if x_hat is None:
        x_hat = _torch().empty_like(x)
    _like("x_hat", x_hat, (x.dtype,), n * p.d)
    _device_tensors(x, x_hat=x_hat)
    _check(lib.isoq_roundtrip(p.handle, _dtype_code(x.dtype), ctypes.c_void_p(x.data_ptr()), n,
                              int(rows_per_set), ctypes.c_void_p(x_hat.data_ptr()), _stream_ptr(stream)),
           "isoq_roundtrip")
    return x_hat


def isoq_quantize(p: Params, x, rows_per_set: int = 1, idx_packed=None, norms=None, stream=None):
    """(packed index records [n, isoq_record_bytes] uint8, norms [n] fp32)."""
    torch = _torch()
    n = _rows(x, p.d)
    if idx_packed is None:
        idx_packed = torch.empty((n, p.record_bytes), dtype=torch.uint8, device=x.device)
    if norms is None:
        norms = torch.empty((n,), dtype=torch.float32, device=x.device)
    _dtype_code(x.dtype)
    _like("idx_packed", idx_packed, (torch.uint8,), n * p.record_bytes)
    _like("norms", norms, (torch.float32,), n)
    _device_tensors(x, idx_packed=idx_packed, norms=norms)
    _check(lib.isoq_quantize(p.handle, _dtype_code(x.dtype), ctypes.c_void_p(x.data_ptr()), n,
                             int(rows_per_set), ctypes.c_void_p(idx_packed.data_ptr()),
                             ctypes.c_void_p(norms.data_ptr()), _stream_ptr(stream)), "isoq_quantize")
    return idx_packed, norms


def isoq_dequantize(p: Params, idx_packed, norms, dtype=None, rows_per_set: int = 1, x_hat=None,
                    stream=None):
    """Rows [n, d] of `dtype` (default float16) from packed records and norms."""
    torch = _torch()
    _like("norms", norms, (torch.float32,), norms.numel() if isinstance(norms, torch.Tensor) else 0)
    n = norms.numel()
    _device_tensors(norms, norms=norms)
    if x_hat is None:
        x_hat = torch.empty((n, p.d), dtype=dtype or torch.float16, device=norms.device)
    _like("idx_packed", idx_packed, (torch.uint8,), n * p.record_bytes)
    _like("x_hat", x_hat, (torch.float16, torch.float32), n * p.d)
    if dtype is not None and x_hat.dtype != dtype:
        raise TypeError(f"x_hat is {x_hat.dtype}, dtype asks for {dtype}")
    _device_tensors(norms, idx_packed=idx_packed, x_hat=x_hat)
    _check(lib.isoq_dequantize(p.handle, _dtype_code(x_hat.dtype), ctypes.c_void_p(idx_packed.data_ptr()),
                               ctypes.c_void_p(norms.data_ptr()), n, int(rows_per_set),
                               ctypes.c_void_p(x_hat.data_ptr()), _stream_ptr(stream)), "isoq_dequantize")
    return x_hat


def _ptr(t):
    return ctypes.c_void_p(None if t is None else t.data_ptr())


def isoq_kv_append(pk: Params, k_new, slot_mapping, k_idx, k_rho, pv: Params = None, v_new=None,
                   v_idx=None, v_rho=None, stream=None):
    """Quantize new rows k_new (and v_new) [n_tokens, n_heads, d] into paged caches
    k_idx (v_idx) [n_blocks, n_heads, block_size, record_bytes] uint8 and k_rho
    (v_rho) [n_blocks, n_heads, block_size] fp32 at the slots slot_mapping
    [n_tokens] int64 (see include/isoquant.h).  The bytes of each
    [block_size, record_bytes] plane hold its records piece-major (pieces of
    P bytes, P = 16 or 8 when it divides record_bytes, else P = record_bytes:
    piece j of position s at byte (j block_size + s) P)."""
    torch = _torch()
    if k_new.dim() != 3 or k_idx.dim() != 4 or k_rho.dim() != 3:
        raise ValueError("k_new [n_tokens, n_heads, d], k_idx [n_blocks, n_heads, block_size, R], "
                         "k_rho [n_blocks, n_heads, block_size]")
    n_tokens, n_heads, d = k_new.shape
    n_blocks, nh, block_size, rb = k_idx.shape
    if d != pk.d or nh != n_heads or rb != pk.record_bytes or tuple(k_rho.shape) != (n_blocks, nh, block_size):
        raise ValueError("cache shapes do not match the rows and the handle")
    if slot_mapping.dtype != torch.int64 or slot_mapping.numel() != n_tokens:
        raise ValueError("slot_mapping must be int64 [n_tokens]")
    if k_idx.dtype != torch.uint8 or k_rho.dtype != torch.float32:
        raise TypeError("k_idx uint8, k_rho float32")
    ts = [k_new, slot_mapping, k_idx, k_rho]
    if v_new is not None:
        if pv is None or v_idx is None or v_rho is None:
            raise ValueError("v_new needs pv, v_idx and v_rho")
        if (tuple(v_new.shape) != tuple(k_new.shape) or tuple(v_idx.shape) != tuple(k_idx.shape)
                or tuple(v_rho.shape) != tuple(k_rho.shape) or v_new.dtype != k_new.dtype):
            raise ValueError("V tensors must have the shapes and dtype of the K tensors")
        ts += [v_new, v_idx, v_rho]
    _device_tensors(k_new, **{f"arg{i}": t for i, t in enumerate(ts)})
    _check(lib.isoq_kv_append(pk.handle, None if pv is None else pv.handle, _dtype_code(k_new.dtype),
                              _ptr(k_new), _ptr(v_new), _ptr(slot_mapping), int(n_tokens), int(n_heads),
                              _ptr(k_idx), _ptr(k_rho), _ptr(v_idx), _ptr(v_rho), int(n_blocks),
                              int(block_size), _stream_ptr(stream)), "isoq_kv_append")


def isoq_kv_scores(pk: Params, q, k_idx, k_rho, block_table, seq_lens, scale: float = 1.0,
                   max_len=None, scores=None, stream=None, sketch=None, k_signs=None, k_gamma=None):
    """Attention logits scale * <q, k_hat> of queries q [n_seqs, n_q_heads, d]
    against the paged key cache k_idx [n_blocks, n_kv_heads, block_size, R] /
    k_rho [n_blocks, n_kv_heads, block_size], with block_table int32
    [n_seqs, max_blocks] and seq_lens int32 [n_seqs].  Returns fp32 scores
    [n_seqs, n_q_heads, max_len]; the kernel does not write positions at or
    past a sequence's length or behind an out-of-range block-table entry: a
    `scores` tensor allocated here holds -inf there, a caller's keeps its
    contents (see include/isoquant.h)."""
    torch = _torch()
    if q.dim() != 3 or k_idx.dim() != 4 or k_rho.dim() != 3 or block_table.dim() != 2:
        raise ValueError("q [n_seqs, n_q_heads, d], k_idx [n_blocks, n_kv_heads, block_size, R], "
                         "k_rho [n_blocks, n_kv_heads, block_size], block_table [n_seqs, max_blocks]")
    n_seqs, n_q_heads, d = q.shape
    n_blocks, n_kv_heads, block_size, rb = k_idx.shape
    if d != pk.d or rb != pk.record_bytes or tuple(k_rho.shape) != (n_blocks, n_kv_heads, block_size):
        raise ValueError("cache shapes do not match the queries and the handle")
    if block_table.shape[0] != n_seqs or seq_lens.numel() != n_seqs:
        raise ValueError("block_table and seq_lens need one row per sequence")
    if block_table.dtype != torch.int32 or seq_lens.dtype != torch.int32:
        raise TypeError("block_table and seq_lens must be int32")
    max_blocks = block_table.shape[1]
    if max_len is None:
        max_len = max_blocks * block_size
    if scores is None:
        # positions the kernel does not write (at or past a sequence's
        # length, or behind an invalid block-table entry) read as -inf, so a
        # softmax over max_len ignores them
        scores = torch.full((n_seqs, n_q_heads, max_len), float("-inf"), dtype=torch.float32, device=q.device)
    elif tuple(scores.shape) != (n_seqs, n_q_heads, max_len) or scores.dtype != torch.float32:
        raise ValueError("scores must be fp32 [n_seqs, n_q_heads, max_len]")
    ts = [q, k_idx, k_rho, block_table, seq_lens, scores]
    if sketch is not None:
        if k_signs is None or k_gamma is None:
            raise ValueError("a sketch needs k_signs and k_gamma")
        if (tuple(k_signs.shape) != (n_blocks, n_kv_heads, block_size, sketch.m // 8) or k_signs.dtype != torch.uint8
                or tuple(k_gamma.shape) != tuple(k_rho.shape) or k_gamma.dtype != torch.float32):
            raise ValueError("k_signs [n_blocks, n_kv_heads, block_size, m/8] uint8, k_gamma like k_rho")
        ts += [k_signs, k_gamma]
    _device_tensors(q, **{f"arg{i}": t for i, t in enumerate(ts)})
    if sketch is None:
        _check(lib.isoq_kv_scores(pk.handle, _dtype_code(q.dtype), _ptr(q), int(n_seqs), int(n_q_heads),
                                  int(n_kv_heads), _ptr(k_idx), _ptr(k_rho), int(n_blocks), int(block_size),
                                  _ptr(block_table), int(max_blocks), _ptr(seq_lens), float(scale),
                                  _ptr(scores), int(max_len), _stream_ptr(stream)), "isoq_kv_scores")
    else:
        _check(lib.isoq_kv_scores_qjl(pk.handle, sketch.handle, _dtype_code(q.dtype), _ptr(q), int(n_seqs),
                                      int(n_q_heads), int(n_kv_heads), _ptr(k_idx), _ptr(k_rho), _ptr(k_signs),
                                      _ptr(k_gamma), int(n_blocks), int(block_size), _ptr(block_table),
                                      int(max_blocks), _ptr(seq_lens), float(scale), _ptr(scores), int(max_len),
                                      _stream_ptr(stream)), "isoq_kv_scores_qjl")
    return scores


def isoq_kv_scores_qjl(pk: Params, sketch, q, k_idx, k_rho, k_signs, k_gamma, block_table, seq_lens,
                       scale: float = 1.0, max_len=None, scores=None, stream=None):
    """isoq_kv_scores with the stage-2 residual correction (see include/isoquant.h)."""
    return isoq_kv_scores(pk, q, k_idx, k_rho, block_table, seq_lens, scale, max_len, scores, stream,
                          sketch=sketch, k_signs=k_signs, k_gamma=k_gamma)


class Sketch:
    """Owner of an isoq_sketch handle (stage-2 projection of a quantizer)."""

    def __init__(self, handle: int, p: Params, m: int):
        self.handle = ctypes.c_void_p(handle)
        self.params, self.m, self.d = p, int(m), p.d

    def close(self):
        if self.handle:
            _check(lib.isoq_sketch_destroy(self.handle), "isoq_sketch_destroy")
            self.handle = ctypes.c_void_p(None)

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def isoq_sketch_init(p: Params, m: int, S=None, seed: int = 7) -> Sketch:
    """Stage-2 sketch of quantizer p: projection S [m, d] (given, or drawn from seed)."""
    dp = ctypes.POINTER(ctypes.c_double)
    S_a = None if S is None else np.ascontiguousarray(S, dtype=np.float64)
    if S_a is not None and S_a.shape != (m, p.d):
        raise ValueError("S must be [m, d]")
    h = ctypes.c_void_p()
    _check(lib.isoq_sketch_init(ctypes.byref(h), p.handle, int(m),
                                None if S_a is None else S_a.ctypes.data_as(dp), int(seed)),
           "isoq_sketch_init")
    return Sketch(h.value, p, m)


def isoq_sketch_destroy(sk: Sketch) -> None:
    sk.close()


def isoq_sketch_export(sk: Sketch):
    """(m, S as used, float32 [m, d])."""
    m = ctypes.c_int()
    S = np.zeros((sk.m, sk.d), np.float32)
    _check(lib.isoq_sketch_export(sk.handle, ctypes.byref(m), S.ctypes.data_as(ctypes.POINTER(ctypes.c_float))),
           "isoq_sketch_export")
    return m.value, S


def isoq_quantize_qjl(p: Params, sk: Sketch, x, rows_per_set: int = 1, idx_packed=None, norms=None,
                      signs=None, gamma=None, stream=None):
    """(records [n, R] uint8, norms [n] fp32, sign sketch [n, m/8] uint8, gamma [n] fp32)."""
    torch = _torch()
    n = _rows(x, p.d)
    dev = x.device
    if idx_packed is None:
        idx_packed = torch.empty((n, p.record_bytes), dtype=torch.uint8, device=dev)
    if norms is None:
        norms = torch.empty((n,), dtype=torch.float32, device=dev)
    if signs is None:
        signs = torch.empty((n, sk.m // 8), dtype=torch.uint8, device=dev)
    if gamma is None:
        gamma = torch.empty((n,), dtype=torch.float32, device=dev)
    _dtype_code(x.dtype)
    _like("idx_packed", idx_packed, (torch.uint8,), n * p.record_bytes)
    _like("norms", norms, (torch.float32,), n)
    _like("signs", signs, (torch.uint8,), n * (sk.m // 8))
    _like("gamma", gamma, (torch.float32,), n)
    _device_tensors(x, idx_packed=idx_packed, norms=norms, signs=signs, gamma=gamma)
    _check(lib.isoq_quantize_qjl(p.handle, sk.handle, _dtype_code(x.dtype), _ptr(x), n, int(rows_per_set),
                                 _ptr(idx_packed), _ptr(norms), _ptr(signs), _ptr(gamma), _stream_ptr(stream)),
           "isoq_quantize_qjl")
    return idx_packed, norms, signs, gamma


def isoq_kv_append_qjl(pk: Params, sk: Sketch, k_new, slot_mapping, k_idx, k_rho, k_signs, k_gamma,
                       stream=None):
    """Quantize new key rows k_new [n_tokens, n_heads, d] with the stage-2
    sketch into the paged caches k_idx [n_blocks, n_heads, block_size, R],
    k_rho and k_gamma [n_blocks, n_heads, block_size] fp32 and k_signs
    [n_blocks, n_heads, block_size, m/8] uint8 at the slots slot_mapping
    [n_tokens] int64 (see include/isoquant.h)."""
    torch = _torch()
    if k_new.dim() != 3 or k_idx.dim() != 4 or k_rho.dim() != 3 or k_signs.dim() != 4 or k_gamma.dim() != 3:
        raise ValueError("k_new [n_tokens, n_heads, d], k_idx [n_blocks, n_heads, block_size, R], "
                         "k_signs [n_blocks, n_heads, block_size, m/8], k_rho and k_gamma [n_blocks, n_heads, "
                         "block_size]")
    n_tokens, n_heads, d = k_new.shape
    n_blocks, nh, block_size, rb = k_idx.shape
    cache = (n_blocks, nh, block_size)
    if (d != pk.d or nh != n_heads or rb != pk.record_bytes or tuple(k_rho.shape) != cache
            or tuple(k_gamma.shape) != cache or tuple(k_signs.shape) != cache + (sk.m // 8,)):
        raise ValueError("cache shapes do not match the rows, the handle and the sketch")
    if slot_mapping.dtype != torch.int64 or slot_mapping.numel() != n_tokens:
        raise ValueError("slot_mapping must be int64 [n_tokens]")
    if (k_idx.dtype != torch.uint8 or k_signs.dtype != torch.uint8 or k_rho.dtype != torch.float32
            or k_gamma.dtype != torch.float32):
        raise TypeError("k_idx and k_signs uint8, k_rho and k_gamma float32")
    _device_tensors(k_new, k_new=k_new, slot_mapping=slot_mapping, k_idx=k_idx, k_rho=k_rho, k_signs=k_signs,
                    k_gamma=k_gamma)
    _check(lib.isoq_kv_append_qjl(pk.handle, sk.handle, _dtype_code(k_new.dtype), _ptr(k_new), _ptr(slot_mapping),
                                  int(n_tokens), int(n_heads), _ptr(k_idx), _ptr(k_rho), _ptr(k_signs),
                                  _ptr(k_gamma), int(n_blocks), int(block_size), _stream_ptr(stream)),
           "isoq_kv_append_qjl")
