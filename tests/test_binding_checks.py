"""CPU checks of the Python binding's argument validation: every tensor a
stage-1 or decoding call hands to a kernel must be a GPU tensor of the right
dtype and size, contiguous, on the device of the input.  A bad argument must
raise TypeError or ValueError before anything is launched.

No GPU is needed: CPU tensors stand in for device tensors (the binding's
placement test is redirected to the CPU), a meta tensor for a tensor that is
not on the device, and the library's launching entry points are replaced by a
stub that fails the test if one is reached."""
import pytest
import torch

import paper_2603_28430_amd as iq
from paper_2603_28430_amd import isoquant as binding


_LAUNCHES = {"isoq_roundtrip", "isoq_quantize", "isoq_dequantize", "isoq_kv_append", "isoq_kv_scores",
             "isoq_quantize_qjl", "isoq_kv_append_qjl", "isoq_kv_scores_qjl"}


class _NoLaunch:
    """The library with its launching entry points replaced by failures
    (host helpers such as isoq_record_bytes still answer)."""

    def __init__(self, real):
        self._real = real

    def __getattr__(self, name):
        if name in _LAUNCHES:
            raise AssertionError(f"{name} was reached with a bad argument")
        return getattr(self._real, name)


@pytest.fixture
def cpu_as_device(monkeypatch):
    monkeypatch.setattr(binding, "_is_gpu", lambda t: t.device.type == "cpu")
    monkeypatch.setattr(binding, "lib", _NoLaunch(binding.lib))


def _params(variant=1, d=128, bits=3):
    return iq.Params(0, variant, d, bits, 1)   # a NULL handle: never passed to the library here


def _raises(fn):
    with pytest.raises((TypeError, ValueError)):
        fn()


def test_roundtrip_checks(cpu_as_device):
    p = _params()
    x = torch.zeros((10, 128), dtype=torch.float16)
    _raises(lambda: iq.isoq_roundtrip(p, x.to("meta")))                                    # input not on the device
    _raises(lambda: iq.isoq_roundtrip(p, x.t()))                                           # not contiguous
    _raises(lambda: iq.isoq_roundtrip(p, torch.zeros((10, 64), dtype=torch.float16)))      # wrong width
    _raises(lambda: iq.isoq_roundtrip(p, x.to(torch.bfloat16)))                            # row type
    _raises(lambda: iq.isoq_roundtrip(p, x, x_hat=torch.zeros((10, 128), dtype=torch.float32)))  # dtype
    _raises(lambda: iq.isoq_roundtrip(p, x, x_hat=torch.zeros((9, 128), dtype=torch.float16)))   # size
    _raises(lambda: iq.isoq_roundtrip(p, x, x_hat=torch.zeros((10, 128), dtype=torch.float16, device="meta")))
    _raises(lambda: iq.isoq_roundtrip(p, x, x_hat=torch.zeros((128, 10), dtype=torch.float16).t()))


def test_quantize_checks(cpu_as_device):
    p = _params()
    x = torch.zeros((10, 128), dtype=torch.float32)
    rec = torch.zeros((10, p.record_bytes), dtype=torch.uint8)
    rho = torch.zeros(10, dtype=torch.float32)
    _raises(lambda: iq.isoq_quantize(p, x, idx_packed=rec.to(torch.int8), norms=rho))
    _raises(lambda: iq.isoq_quantize(p, x, idx_packed=rec[:9], norms=rho))
    _raises(lambda: iq.isoq_quantize(p, x, idx_packed=rec, norms=rho.to(torch.float16)))
    _raises(lambda: iq.isoq_quantize(p, x, idx_packed=rec, norms=rho[:9]))
    _raises(lambda: iq.isoq_quantize(p, x, idx_packed=rec.to("meta"), norms=rho))
    _raises(lambda: iq.isoq_quantize(p, x, idx_packed=rec, norms=rho.to("meta")))
    _raises(lambda: iq.isoq_quantize(p, x, idx_packed=rec, norms=torch.zeros(20)[::2]))


def test_dequantize_checks(cpu_as_device):
    p = _params()
    rec = torch.zeros((10, p.record_bytes), dtype=torch.uint8)
    rho = torch.zeros(10, dtype=torch.float32)
    xh = torch.zeros((10, 128), dtype=torch.float16)
    _raises(lambda: iq.isoq_dequantize(p, rec, rho.to(torch.float64), x_hat=xh))
    _raises(lambda: iq.isoq_dequantize(p, rec, rho.to("meta"), x_hat=xh))
    _raises(lambda: iq.isoq_dequantize(p, rec[:, :40], rho, x_hat=xh))
    _raises(lambda: iq.isoq_dequantize(p, rec.to(torch.int32), rho, x_hat=xh))
    _raises(lambda: iq.isoq_dequantize(p, rec.to("meta"), rho, x_hat=xh))
    _raises(lambda: iq.isoq_dequantize(p, rec, rho, x_hat=xh[:9]))
    _raises(lambda: iq.isoq_dequantize(p, rec, rho, x_hat=xh.to(torch.bfloat16)))
    _raises(lambda: iq.isoq_dequantize(p, rec, rho, x_hat=xh.to("meta")))
    _raises(lambda: iq.isoq_dequantize(p, rec, rho, x_hat=xh, dtype=torch.float32))


def test_quantize_qjl_checks(cpu_as_device):
    p = _params()
    sk = iq.Sketch(0, p, 128)
    x = torch.zeros((10, 128), dtype=torch.float16)
    rec = torch.zeros((10, p.record_bytes), dtype=torch.uint8)
    rho = torch.zeros(10, dtype=torch.float32)
    sg = torch.zeros((10, 16), dtype=torch.uint8)
    gm = torch.zeros(10, dtype=torch.float32)
    ok = dict(idx_packed=rec, norms=rho, signs=sg, gamma=gm)
    for name, bad in (("idx_packed", rec.to(torch.int16)), ("norms", rho[:5]), ("signs", sg[:, :8]),
                      ("signs", sg.to(torch.float32)), ("gamma", gm.to(torch.float64)), ("gamma", gm.to("meta")),
                      ("norms", rho.to("meta"))):
        kw = dict(ok, **{name: bad})
        _raises(lambda: iq.isoq_quantize_qjl(p, sk, x, **kw))


def test_kv_calls_check_placement(cpu_as_device):
    p = _params()
    k = torch.zeros((4, 2, 128), dtype=torch.float16)
    slots = torch.arange(4, dtype=torch.int64)
    cache = torch.zeros((2, 2, 16, p.record_bytes), dtype=torch.uint8)
    rho = torch.zeros((2, 2, 16), dtype=torch.float32)
    _raises(lambda: iq.isoq_kv_append(p, k, slots.to("meta"), cache, rho))
    _raises(lambda: iq.isoq_kv_append(p, k, slots, cache, rho.to("meta")))
    q = torch.zeros((1, 2, 128), dtype=torch.float16)
    table = torch.zeros((1, 2), dtype=torch.int32)
    lens = torch.zeros(1, dtype=torch.int32)
    _raises(lambda: iq.isoq_kv_scores(p, q, cache, rho, table, lens.to("meta")))
    _raises(lambda: iq.isoq_kv_scores(p, q, cache.to("meta"), rho, table, lens))
