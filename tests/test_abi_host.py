"""CPU checks of the C-ABI library: it loads, exports every entry point that
include/isoquant.h declares, rejects bad arguments before touching a device,
and its host-side parameter construction (Lloyd-Max codebook, seeded Philox
draws) agrees with the independent implementations in the oracle and the
workload generator.  No kernel is launched here."""
import ctypes
import os
import re

import numpy as np
import pytest

import oracle
import workloads
import paper_2603_28430_amd as iq
from paper_2603_28430_amd import isoquant as binding

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include",
                      "isoquant.h")


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(isoq_[a-z_0-9]+)\s*\(", text)))


def test_header_declares_the_boundary():
    names = _declared()
    for required in ("isoq_params_init", "isoq_params_destroy", "isoq_params_export",
                     "isoq_quantize", "isoq_dequantize", "isoq_roundtrip", "isoq_kv_append",
                     "isoq_kv_scores", "isoq_packed_bytes", "isoq_record_bytes",
                     "isoq_status_string"):
        assert required in names


def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(iq.LIB_PATH)
    missing = [n for n in _declared() if not hasattr(lib, n)]
    assert not missing, missing


def test_sizes():
    assert iq.isoq_packed_bytes(128, 3) == 48
    assert iq.isoq_packed_bytes(128, 2) == 32
    assert iq.isoq_packed_bytes(128, 4) == 64
    assert iq.isoq_packed_bytes(256, 3) == 96
    assert iq.isoq_packed_bytes(5, 3) == 2
    assert iq.isoq_packed_bytes(0, 3) == 0
    for v in ("full", "fast", "2d", "8d"):
        for d in (128, 256, 512, 6, 13):
            assert iq.isoq_raw_params_per_set(v, d) == workloads.raw_params_per_set(v, d)
            assert iq.isoq_raw_params_per_set(v, d) == oracle.raw_params_per_set(v, d)
            assert iq.isoq_export_params_per_set(v, d) == oracle.table1_params(v, d)
    assert iq.isoq_raw_params_per_set(7, 128) == 0
    # records hold the padded width: 4 ceil(d/4) coordinates, 2-D 2 ceil(d/2),
    # 8-D 8 ceil(d/8)
    for v in ("full", "fast", "2d", "8d"):
        for d in (1, 2, 3, 5, 6, 7, 90, 91, 96, 128, 1000, 1023):
            for b in (2, 3, 4):
                pw = oracle.padded_width(v, d)
                assert iq.isoq_record_bytes(v, d, b) == oracle.record_bytes(pw, b)
                if d % 4 == 0:
                    assert iq.isoq_record_bytes(v, d, b) == iq.isoq_packed_bytes(d, b)
    assert iq.isoq_record_bytes("full", 0, 3) == 0
    assert iq.isoq_record_bytes("2d", 9, 3) == 4 and iq.isoq_record_bytes("full", 9, 3) == 5
    assert iq.isoq_record_bytes("8d", 9, 3) == 6 and iq.isoq_record_bytes("8d", 128, 3) == 48


def test_status_strings():
    for s in range(8):
        assert iq.isoq_status_string(s)
    assert iq.isoq_status_string(99) == "unknown status"


@pytest.mark.parametrize("bits", [2, 3, 4])
@pytest.mark.parametrize("d", [128, 256, 512, 5, 90, 1000])
def test_library_codebook_matches_oracle(bits, d):
    lib_levels = iq.isoq_codebook_lloyd(bits, d, 200)
    ref = oracle.codebook(bits, d, 200)
    np.testing.assert_allclose(lib_levels, ref, rtol=1e-11, atol=1e-14)


def test_library_codebook_converges_to_max_table():
    import json
    g = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "lloyd_max_gaussian.json")))
    for b in (2, 3, 4):
        lv = iq.isoq_codebook_lloyd(b, 1, 5000)
        np.testing.assert_allclose(lv[(1 << b) // 2:], g["levels_positive"][str(b)], atol=6e-4)


@pytest.mark.parametrize("variant", ["full", "fast", "2d", "8d"])
def test_library_seeded_draws_match_workload_generator(variant):
    for seed in (0, 1, 2**40 + 7):
        a = iq.isoq_rotation_draws(variant, 128, 3, seed)
        b = workloads.rotation_draws(variant, 128, 3, seed)
        np.testing.assert_allclose(a, b, rtol=1e-12, atol=1e-12)


def test_argument_validation_before_any_device_call():
    h = ctypes.c_void_p()
    init = binding.lib.isoq_params_init
    dp = ctypes.POINTER(ctypes.c_double)
    assert init(None, 0, 128, 3, 1, None, None, 1) == 3            # NULL out
    assert init(ctypes.byref(h), 5, 128, 3, 1, None, None, 1) == 1  # bad variant
    assert init(ctypes.byref(h), 0, 128, 3, 0, None, None, 1) == 1  # n_sets < 1
    assert init(ctypes.byref(h), 0, 1025, 3, 1, None, None, 1) == 2  # d outside 1..1024
    assert init(ctypes.byref(h), 0, 128, 5, 1, None, None, 1) == 2  # bits outside {2,3,4}
    assert h.value is None
    bad = np.array([-1.0, -0.5, 0.2, 1.0])                          # not symmetric
    assert init(ctypes.byref(h), 0, 128, 2, 1, None, bad.ctypes.data_as(dp), 1) == 1
    unsorted = np.array([-1.0, 0.5, -0.5, 1.0])
    assert init(ctypes.byref(h), 0, 128, 2, 1, None, unsorted.ctypes.data_as(dp), 1) == 1
    zero_q = np.zeros(8 * 32)
    assert init(ctypes.byref(h), 0, 128, 2, 1, zero_q.ctypes.data_as(dp), None, 1) == 1
    # 8-D blocks: a raw matrix with dependent columns has no rotation
    G = workloads.rotation_draws("8d", 128, 1, seed=1).reshape(16, 8, 8)
    G[5, :, 3] = 2.0 * G[5, :, 1]
    assert init(ctypes.byref(h), 3, 128, 3, 1, np.ascontiguousarray(G).ctypes.data_as(dp), None, 1) == 1
    G[5] = 0.0
    assert init(ctypes.byref(h), 3, 128, 3, 1, np.ascontiguousarray(G).ctypes.data_as(dp), None, 1) == 1
    assert init(ctypes.byref(h), 4, 128, 3, 1, None, None, 1) == 1   # no variant 4
    for fn, args in ((binding.lib.isoq_roundtrip, (None, 1, None, 4, 1, None, None)),
                     (binding.lib.isoq_quantize, (None, 1, None, 4, 1, None, None, None)),
                     (binding.lib.isoq_dequantize, (None, 1, None, None, 4, 1, None, None))):
        assert fn(*args) == 3
    # isoq_kv_append: NULL K handle
    assert binding.lib.isoq_kv_append(None, None, 1, None, None, None, 4, 2, None, None, None, None,
                                      8, 16, None) == 3
    # isoq_kv_scores: NULL K handle
    assert binding.lib.isoq_kv_scores(None, 1, None, 1, 1, 1, None, None, 1, 16, None, 1, None, 1.0,
                                      None, 16, None) == 3
    # stage-2 sketch: NULL handles
    sk = ctypes.c_void_p()
    assert binding.lib.isoq_sketch_init(ctypes.byref(sk), None, 128, None, 1) == 3
    assert binding.lib.isoq_sketch_init(None, None, 128, None, 1) == 3
    assert binding.lib.isoq_sketch_destroy(None) == 0
    assert binding.lib.isoq_sketch_export(None, None, None) == 3
    assert binding.lib.isoq_quantize_qjl(None, None, 1, None, 4, 1, None, None, None, None, None) == 3
    assert binding.lib.isoq_kv_scores_qjl(None, None, 1, None, 1, 1, 1, None, None, None, None, 1, 16, None, 1,
                                          None, 1.0, None, 16, None) == 3
    assert binding.lib.isoq_kv_append_qjl(None, None, 1, None, None, 4, 2, None, None, None, None, 8, 16,
                                          None) == 3
    assert binding.lib.isoq_params_destroy(None) == 0
    assert binding.lib.isoq_params_export(None, None, None, None) == 3


def test_init_without_device_reports_hip_error():
    import torch
    if torch.cuda.is_available():
        pytest.skip("a GPU is present")
    with pytest.raises(iq.IsoqError) as e:
        iq.isoq_params_init("full", 128, 3)
    assert e.value.status == 5
