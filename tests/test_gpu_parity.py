"""Parity of the HIP path (through the C ABI) with the CPU oracle, every
variant x d x bits x dtype, plus edge cases.  Needs an MI355X."""
import numpy as np
import pytest

import oracle
import workloads
from parity import Oracle, rel_err

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

import paper_2603_28430_amd as iq  # noqa: E402

DT = {"f16": (torch.float16, np.float16), "f32": (torch.float32, np.float32)}


def make(variant, d, bits, n_sets=1, seed=1):
    rot = workloads.rotation_draws(variant, d, n_sets, seed)
    levels = oracle.codebook(bits, d)
    p = iq.isoq_params_init(variant, d, bits, n_sets, rot=rot, codebook=levels)
    return p, rot, levels


def run_all(p, xg, rows_per_set=1):
    """quantize, dequantize, roundtrip on the same input; outputs on the host."""
    idx, rho = iq.isoq_quantize(p, xg, rows_per_set)
    xdq = iq.isoq_dequantize(p, idx, rho, dtype=xg.dtype, rows_per_set=rows_per_set)
    xrt = iq.isoq_roundtrip(p, xg, rows_per_set)
    torch.cuda.synchronize()
    return idx.cpu().numpy(), rho.cpu().numpy(), xdq.cpu().numpy(), xrt.cpu().numpy()


def check(variant, d, bits, dtype, n, n_sets=1, rows_per_set=1, sample=None, seed=0, x=None):
    tdt, ndt = DT[dtype]
    p, rot, levels = make(variant, d, bits, n_sets)
    if x is None:
        x = workloads.unit_gaussian_rows(n, d, seed=seed, dtype=ndt)
    xg = torch.from_numpy(x).cuda()
    idx, rho, xdq, xrt = run_all(p, xg, rows_per_set)
    # the fused path equals quantize followed by dequantize, bit for bit
    assert np.array_equal(xrt.view(np.uint8), xdq.view(np.uint8))
    rows = None if sample is None else sample
    o = Oracle(variant, d, bits, rot, levels, x, n_sets, rows_per_set, rows=rows)
    sel = slice(None) if rows is None else rows
    idx_g = oracle.unpack(idx[sel], d, bits)
    agree = o.check_indices(idx_g)
    o.check_norms(rho[sel])
    err = o.check_xhat(xrt[sel], ndt)
    return agree, err


@pytest.mark.parametrize("dtype", ["f16", "f32"])
@pytest.mark.parametrize("bits", [2, 3, 4])
@pytest.mark.parametrize("d", [64, 128, 256, 512])
@pytest.mark.parametrize("variant", ["full", "fast", "2d"])
def test_parity_small_ragged(variant, d, bits, dtype):
    # a few hundred row groups: several waves, a ragged last group
    n = {64: 2075, 128: 1037, 256: 521, 512: 263}[d]
    print(f"case {variant} d={d} b={bits} {dtype} n={n}", flush=True)
    check(variant, d, bits, dtype, n)


@pytest.mark.parametrize("variant,d,bits,dtype", [("full", 128, 3, "f16"), ("fast", 256, 2, "f16"),
                                                  ("2d", 128, 4, "f32"), ("full", 512, 3, "f32"),
                                                  ("fast", 64, 3, "f16"), ("full", 64, 4, "f32")])
def test_parity_many_groups_per_wave(variant, d, bits, dtype):
    """Large enough that every wave walks several row groups (prefetch loop and
    its odd tail); sampled rows against the oracle, every row for the
    fused == quantize + dequantize identity."""
    rows_per_wave = 512 // d
    n = 200_003 * rows_per_wave // 4 + 1
    rng = np.random.default_rng(5)
    sample = np.unique(np.concatenate([np.arange(64), np.arange(n - 64, n),
                                       rng.integers(0, n, 3000)]))
    print(f"case {variant} d={d} b={bits} {dtype} n={n}", flush=True)
    check(variant, d, bits, dtype, n, sample=sample)


@pytest.mark.parametrize("rows_per_set", [1, 3, 4, 5, 8, 64, 1000])
@pytest.mark.parametrize("variant", ["full", "fast", "2d"])
def test_parity_multiple_sets(variant, rows_per_set):
    """Parameter set of row r = (r / rows_per_set) mod n_sets; both the
    segment schedule (rows_per_set a multiple of the rows per wave) and the
    generic per-lane path."""
    for d in (64, 128, 256):
        print(f"case {variant} d={d} rps={rows_per_set}", flush=True)
        check(variant, d, 3, "f16", 2003, n_sets=3, rows_per_set=rows_per_set)


@pytest.mark.parametrize("n", [1, 2, 3, 4, 5, 17])
def test_tiny_batches(n):
    for variant in ("full", "fast", "2d"):
        for d in (64, 128, 256, 512):
            check(variant, d, 3, "f16", n)


def test_zero_and_scaled_rows():
    d, bits = 128, 3
    x = workloads.unit_gaussian_rows(64, d, seed=3, dtype=np.float32)
    x[0] = 0.0
    x[1] *= 1e-15                         # squared norms stay inside the fp32 normal range
    x[2] *= 1e15
    x[3, :64] = 0.0                       # a half-zero row: rotated zeros sit on t = 0
    for variant in ("full", "fast", "2d"):
        agree, _ = check(variant, d, bits, "f32", 64, x=x)
        p, rot, levels = make(variant, d, bits)
        xg = torch.from_numpy(x).cuda()
        idx, rho = iq.isoq_quantize(p, xg)
        xh = iq.isoq_roundtrip(p, xg)
        idx0 = oracle.unpack(idx[:1].cpu().numpy(), d, bits)
        assert np.all(idx0 == (1 << bits) // 2 - 1)
        assert float(rho[0]) == 0.0
        assert torch.count_nonzero(xh[0]).item() == 0


def test_fp16_extremes():
    d = 128
    x = workloads.unit_gaussian_rows(32, d, seed=4, dtype=np.float32)
    x[0] *= 1000.0
    x[1] *= 1e-3
    x = x.astype(np.float16)
    for variant in ("full", "fast", "2d"):
        check(variant, d, 3, "f16", 32, x=x)


def test_empty_batch_is_a_noop():
    p, _, _ = make("full", 128, 3)
    x = torch.empty((0, 128), dtype=torch.float16, device="cuda")
    canary = torch.full((16,), 7, dtype=torch.float32, device="cuda")
    out = iq.isoq_roundtrip(p, x)
    idx, rho = iq.isoq_quantize(p, x, norms=canary[:0])
    torch.cuda.synchronize()
    assert out.numel() == 0 and idx.numel() == 0
    assert torch.all(canary == 7)


def test_outputs_stay_inside_their_buffers():
    """Canary bytes around every output survive."""
    d, bits, n = 128, 3, 1037
    for variant in ("full", "fast", "2d"):
        for tdt, ndt in DT.values():
            p, _, _ = make(variant, d, bits)
            x = torch.from_numpy(workloads.unit_gaussian_rows(n, d, 9, ndt)).cuda()
            G = 256
            big = torch.full((n * d + 2 * G,), -3.0, dtype=tdt, device="cuda")
            xh = big[G:G + n * d].view(n, d)
            iq.isoq_roundtrip(p, x, x_hat=xh)
            rb = p.record_bytes
            recs = torch.full((n * rb + 2 * G,), 0xA5, dtype=torch.uint8, device="cuda")
            norms = torch.full((n + 2 * G,), -5.0, dtype=torch.float32, device="cuda")
            iq.isoq_quantize(p, x, idx_packed=recs[G:G + n * rb].view(n, rb), norms=norms[G:G + n])
            big2 = torch.full((n * d + 2 * G,), -3.0, dtype=tdt, device="cuda")
            iq.isoq_dequantize(p, recs[G:G + n * rb].view(n, rb), norms[G:G + n],
                               x_hat=big2[G:G + n * d].view(n, d))
            torch.cuda.synchronize()
            for buf, fill in ((big, -3.0), (big2, -3.0), (recs, 0xA5), (norms, -5.0)):
                assert torch.all(buf[:G] == fill) and torch.all(buf[-G:] == fill)


def test_deterministic_and_in_place():
    d, bits, n = 256, 4, 4099
    p, _, _ = make("full", d, bits)
    x = torch.from_numpy(workloads.unit_gaussian_rows(n, d, 11, np.float16)).cuda()
    a = iq.isoq_roundtrip(p, x)
    b = iq.isoq_roundtrip(p, x)
    y = x.clone()
    iq.isoq_roundtrip(p, y, x_hat=y)           # in place
    torch.cuda.synchronize()
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))
    assert torch.equal(a.view(torch.int16), y.view(torch.int16))


def test_non_default_stream():
    d, bits, n = 128, 3, 50_000
    p, _, _ = make("fast", d, bits)
    x = torch.from_numpy(workloads.unit_gaussian_rows(n, d, 12, np.float16)).cuda()
    ref = iq.isoq_roundtrip(p, x)
    torch.cuda.synchronize()
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        out = torch.empty_like(x)
        iq.isoq_roundtrip(p, x, x_hat=out, stream=s)
    s.synchronize()
    assert torch.equal(out.view(torch.int16), ref.view(torch.int16))


def test_argument_errors_through_the_binding():
    p, _, _ = make("full", 128, 3)
    x = torch.zeros(4 * 128 + 8, dtype=torch.float16, device="cuda")
    bad = x[1:1 + 4 * 128].view(4, 128)       # 2-byte aligned: rejected
    with pytest.raises(iq.IsoqError) as e:
        iq.isoq_roundtrip(p, bad)
    assert e.value.status == 4
    with pytest.raises(iq.IsoqError) as e:
        iq.isoq_roundtrip(p, x[:512].view(4, 128), rows_per_set=0)
    assert e.value.status == 1


def test_library_defaults_match_oracle():
    """codebook=None gives the Lloyd-Max codebook; rot=None gives the seeded
    Philox draws; the exported values are what the oracle computes from the
    same draws."""
    for variant in ("full", "fast", "2d"):
        for d, bits in ((128, 3), (256, 2), (512, 4)):
            p = iq.isoq_params_init(variant, d, bits, 2, seed=1234)
            rot, lev, thr = iq.isoq_params_export(p)
            np.testing.assert_allclose(lev, oracle.codebook(bits, d), rtol=1e-6)
            np.testing.assert_allclose(thr, oracle.thresholds(bits, oracle.codebook(bits, d)),
                                       rtol=1e-6, atol=1e-9)
            raw = workloads.rotation_draws(variant, d, 2, 1234)
            if variant == "2d":
                ref = np.stack([np.cos(raw), np.sin(raw)], -1).reshape(-1)
            else:
                w = 8 if variant == "full" else 4
                q = raw.reshape(-1, 4)
                ref = (q / np.linalg.norm(q, axis=1, keepdims=True)).reshape(-1)
                assert ref.size == 2 * (d // 4) * w
            np.testing.assert_allclose(rot, ref, atol=2e-7)


def test_mse_matches_sphere_theory():
    """Per-coordinate MSE of the fused path on unit vectors equals the 1-D
    sphere-marginal integral (identical for all variants)."""
    from test_oracle_pins import _sphere_mse
    d, bits, n = 128, 3, 1 << 20
    x = torch.from_numpy(workloads.unit_gaussian_rows(n, d, 0, np.float32)).cuda()
    for variant in ("full", "fast", "2d"):
        p, rot, levels = make(variant, d, bits)
        xh = iq.isoq_roundtrip(p, x)
        mse = torch.mean((xh.double() - x.double()) ** 2).item()
        ref = _sphere_mse(d, bits, levels)
        assert abs(mse / ref - 1) < 0.005, (variant, mse, ref)
