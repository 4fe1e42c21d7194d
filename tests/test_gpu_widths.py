"""Parity of the stage-1 kernels at widths outside {64, 128, 256, 512} with
the oracle, through the C ABI: the packed-row kernels (fp16 rows,
d = 16 k up to 504; 3 bits at d = 272, 304, ... 496 excepted) and the
generic kernels (every other width and dtype up to d = 1024; Sec. 5.1 zero
padding when d is not a multiple of the block size; fp16 rows of width 2 mod 4
move in coordinate pairs).

Per case: isoq_quantize, isoq_dequantize and isoq_roundtrip on the same rows;
the fused path equals quantize followed by dequantize bit for bit; indices,
norms and reconstructions against the oracle under the rule of
tests/parity.py; the raw record equals the packing of its own indices (all
pw = padded-width coordinates, bits past pw * bits zero).  Needs an MI355X."""
import numpy as np
import pytest

import oracle
import workloads
from parity import Oracle

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

import paper_2603_28430_amd as iq  # noqa: E402

DT = {"f16": (torch.float16, np.float16), "f32": (torch.float32, np.float32)}

# widths below, between and above the tuned ones; odd, 2 mod 4 and
# multiple-of-4 widths; every row shape of the generic kernels (8 to 64 lanes,
# 1 to 4 slots per lane) and its largest width; packed rows of 2 to 62 lanes
# (d = 16 .. 496: V d/8 a multiple of 4 or not, one row per wave), two
# chunks per lane (192, 288 at 2 and 4 bits, 320), and widths where 3 bits
# falls back to the generic kernels (272, 496)
WIDTHS = [1, 2, 3, 5, 6, 7, 16, 20, 32, 33, 48, 60, 63, 80, 90, 96, 100, 112, 127, 130, 144, 160, 192, 208, 250,
          256 + 4, 272, 288, 320, 384, 496, 511, 640, 1000, 1024]


def check(variant, d, bits, dtype, n, n_sets=1, rows_per_set=1, x=None, sample=None, seed=0):
    tdt, ndt = DT[dtype]
    rot = workloads.rotation_draws(variant, d, n_sets, seed=1)
    levels = oracle.codebook(bits, d)
    p = iq.isoq_params_init(variant, d, bits, n_sets, rot=rot, codebook=levels)
    if x is None:
        x = workloads.unit_gaussian_rows(n, d, seed=seed, dtype=ndt)
    xg = torch.from_numpy(x).cuda()
    idx, rho = iq.isoq_quantize(p, xg, rows_per_set)
    xdq = iq.isoq_dequantize(p, idx, rho, dtype=tdt, rows_per_set=rows_per_set)
    xrt = iq.isoq_roundtrip(p, xg, rows_per_set)
    torch.cuda.synchronize()
    idx, rho, xdq, xrt = idx.cpu().numpy(), rho.cpu().numpy(), xdq.cpu().numpy(), xrt.cpu().numpy()
    assert np.array_equal(xrt.view(np.uint8), xdq.view(np.uint8))
    pw = oracle.padded_width(variant, d)
    assert idx.shape[1] == oracle.record_bytes(pw, bits) == iq.isoq_record_bytes(variant, d, bits)
    sel = slice(None) if sample is None else sample
    idx_g = oracle.unpack(idx[sel], pw, bits)
    np.testing.assert_array_equal(oracle.pack(idx_g, bits), idx[sel])
    o = Oracle(variant, d, bits, rot, levels, x, n_sets, rows_per_set, rows=sample)
    o.check_indices(idx_g)
    o.check_norms(rho[sel])
    o.check_xhat(xrt[sel], ndt)
    p.close()


@pytest.mark.parametrize("d", WIDTHS)
@pytest.mark.parametrize("variant", ["full", "fast", "2d"])
def test_widths_parity(variant, d):
    # several blocks and a ragged last group for every row shape
    n = 1037 if d <= 256 else 263
    for bits in (2, 3, 4):
        for dtype in ("f16", "f32"):
            print(f"case {variant} d={d} b={bits} {dtype} n={n}", flush=True)
            check(variant, d, bits, dtype, n, seed=d + bits)


# 480 is a multiple of the packed kernels' block heights at d = 80, 96, 160
# and 192 (96, 80, 48 and 40 rows), so each block there has one set
@pytest.mark.parametrize("rows_per_set", [1, 5, 64, 480, 1000])
@pytest.mark.parametrize("variant,d", [("full", 90), ("fast", 96), ("2d", 75), ("full", 80), ("2d", 160),
                                       ("full", 192)])
def test_widths_multiple_sets(variant, d, rows_per_set):
    print(f"case {variant} d={d} sets=3 rps={rows_per_set}", flush=True)
    check(variant, d, 3, "f16", 2003, n_sets=3, rows_per_set=rows_per_set)


@pytest.mark.parametrize("n", [1, 2, 3, 5, 33])
def test_widths_tiny_batches(n):
    for variant in ("full", "fast", "2d"):
        for d in (3, 60, 80, 90, 96, 192, 1000):
            print(f"case {variant} d={d} n={n}", flush=True)
            check(variant, d, 3, "f32", n, seed=n)


def test_widths_zero_and_scaled_rows():
    for variant, d in (("full", 90), ("fast", 60), ("2d", 91)):
        x = workloads.unit_gaussian_rows(64, d, seed=3, dtype=np.float32)
        x[0] = 0.0
        x[1] *= 1e-15
        x[2] *= 1e15
        x[3, : d // 2] = 0.0
        print(f"case {variant} d={d} zero and scaled rows", flush=True)
        check(variant, d, 3, "f32", 64, x=x)
        p = iq.isoq_params_init(variant, d, 3, 1)
        xg = torch.from_numpy(x).cuda()
        idx, rho = iq.isoq_quantize(p, xg)
        xh = iq.isoq_roundtrip(p, xg)
        pw = oracle.padded_width(variant, d)
        assert np.all(oracle.unpack(idx[:1].cpu().numpy(), pw, 3) == 3)
        assert float(rho[0]) == 0.0 and torch.count_nonzero(xh[0]).item() == 0


@pytest.mark.parametrize("variant,d,dtype", [("full", 96, "f16"), ("fast", 80, "f16"), ("2d", 90, "f32"),
                                             ("full", 1000, "f32"), ("fast", 192, "f16"), ("full", 90, "f16")])
def test_widths_large_sampled(variant, d, dtype):
    """Many row groups per block and a grid of thousands of blocks: sampled
    rows against the oracle, every row for the fused identity."""
    n = 1_000_003 if d <= 128 else 100_003
    rng = np.random.default_rng(6)
    sample = np.unique(np.concatenate([np.arange(64), np.arange(n - 64, n), rng.integers(0, n, 3000)]))
    print(f"case {variant} d={d} {dtype} n={n}", flush=True)
    check(variant, d, 3, dtype, n, sample=sample)


def test_widths_unsupported_calls():
    """Widths outside the generic range, and the sketch at a width outside
    its own (d = 100), return ISOQ_E_UNSUPPORTED before any launch (append
    and logits take every width)."""
    with pytest.raises(iq.IsoqError) as e:
        iq.isoq_params_init("full", 1025, 3, 1)
    assert e.value.status == 2
    p = iq.isoq_params_init("fast", 100, 3, 1)
    with pytest.raises(iq.IsoqError) as e:
        iq.isoq_sketch_init(p, 64)
    assert e.value.status == 2


@pytest.mark.parametrize("variant,d,dtype", [("full", 90, "f16"), ("fast", 96, "f32"), ("2d", 1000, "f16"),
                                             ("fast", 7, "f32"), ("fast", 80, "f16"), ("2d", 320, "f16")])
def test_widths_guard_bands_determinism_stream_in_place(variant, d, dtype):
    """Canary bytes around every output survive; a second call writes the
    same bytes; a non-default stream gives the same result; the round trip
    may overwrite its input; n = 0 writes nothing."""
    tdt, ndt = DT[dtype]
    n, G = 517, 64
    p = iq.isoq_params_init(variant, d, 3, 1, rot=workloads.rotation_draws(variant, d, 1, seed=1))
    x = torch.from_numpy(workloads.unit_gaussian_rows(n, d, seed=4, dtype=ndt)).cuda()
    R = p.record_bytes
    big_y = torch.full((n * d + 2 * G,), -3.0, dtype=tdt, device="cuda")
    big_r = torch.full((n * R + 2 * G,), 0xA5, dtype=torch.uint8, device="cuda")
    big_n = torch.full((n + 2 * G,), -5.0, dtype=torch.float32, device="cuda")
    big_d = torch.full((n * d + 2 * G,), -3.0, dtype=tdt, device="cuda")
    y, rec, nrm, dq = (big_y[G:G + n * d].view(n, d), big_r[G:G + n * R].view(n, R), big_n[G:G + n],
                       big_d[G:G + n * d].view(n, d))
    iq.isoq_roundtrip(p, x, x_hat=y)
    iq.isoq_quantize(p, x, idx_packed=rec, norms=nrm)
    iq.isoq_dequantize(p, rec, nrm, x_hat=dq)
    torch.cuda.synchronize()
    for big, val in ((big_y, -3.0), (big_r, 0xA5), (big_n, -5.0), (big_d, -3.0)):
        assert torch.all(big[:G] == val) and torch.all(big[-G:] == val)
    assert torch.equal(y, dq)
    # determinism
    y2 = iq.isoq_roundtrip(p, x)
    rec2, nrm2 = iq.isoq_quantize(p, x)
    torch.cuda.synchronize()
    assert torch.equal(y2, y) and torch.equal(rec2, rec) and torch.equal(nrm2, nrm)
    # non-default stream
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        y3 = torch.empty_like(x)
        iq.isoq_roundtrip(p, x, x_hat=y3, stream=s)
    s.synchronize()
    assert torch.equal(y3, y)
    # in place
    xi = x.clone()
    iq.isoq_roundtrip(p, xi, x_hat=xi)
    torch.cuda.synchronize()
    assert torch.equal(xi, y)
    # empty batch
    e = torch.empty((0, d), dtype=tdt, device="cuda")
    canary = torch.full((4,), 7.0, dtype=torch.float32, device="cuda")
    out = iq.isoq_roundtrip(p, e)
    idx0, _ = iq.isoq_quantize(p, e, norms=canary[:0])
    torch.cuda.synchronize()
    assert out.numel() == 0 and idx0.numel() == 0 and torch.all(canary == 7.0)
