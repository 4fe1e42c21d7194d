"""Parity at the full workload sizes, in the launch configuration the benchmark
times: sampled rows against the oracle (which computes them one by one), and
properties that hold at any size for every row (fused == quantize+dequantize
bit for bit; norms against an fp64 reduction; per-coordinate MSE against the
sphere-marginal integral).  Needs an MI355X."""
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
from test_oracle_pins import _sphere_mse  # noqa: E402

_X = {}


def rows(n, d, dtype):
    key = (n, d, dtype)
    if key not in _X:
        _X.clear()
        _X[key] = workloads.unit_gaussian_rows(n, d, seed=0, dtype=dtype)
    return _X[key]


def sample_rows(n, k=4096, seed=7):
    rng = np.random.default_rng(seed)
    return np.unique(np.concatenate([np.arange(32), np.arange(n - 32, n), rng.integers(0, n, k)]))


def full_size_case(variant, d, bits, n, np_dtype, mse_tol=0.005):
    x = rows(n, d, np_dtype)
    rot = workloads.rotation_draws(variant, d, 1, seed=1)
    levels = oracle.codebook(bits, d)
    p = iq.isoq_params_init(variant, d, bits, 1, rot=rot, codebook=levels)
    xg = torch.from_numpy(x).cuda()
    idx, rho = iq.isoq_quantize(p, xg)
    xdq = iq.isoq_dequantize(p, idx, rho, dtype=xg.dtype)
    xrt = iq.isoq_roundtrip(p, xg)
    torch.cuda.synchronize()
    assert torch.equal(xrt.view(torch.uint8), xdq.view(torch.uint8)), "fused != quantize+dequantize"
    ref_rho = torch.linalg.vector_norm(xg.double(), dim=1)
    assert torch.all((rho.double() - ref_rho).abs() <= 1e-6 * ref_rho).item()
    s = sample_rows(n)
    o = Oracle(variant, d, bits, rot, levels, x, rows=s)
    st = torch.from_numpy(s).cuda()
    o.check_indices(oracle.unpack(idx[st].cpu().numpy(), d, bits))
    o.check_norms(rho[st].cpu().numpy())
    o.check_xhat(xrt[st].cpu().numpy(), np_dtype)
    mse = torch.mean((xrt.double() - xg.double()) ** 2).item()
    ref = _sphere_mse(d, bits, levels)
    assert abs(mse / ref - 1) < mse_tol, (mse, ref)
    return mse


def test_config_full_fp32_d128_n4096_every_row():
    """Full roundtrip fp32, 4,096 x d=128, 3 bits: every row against the oracle."""
    d, bits, n = 128, 3, 4096
    x = workloads.unit_gaussian_rows(n, d, seed=0, dtype=np.float32)
    rot = workloads.rotation_draws("full", d, 1, seed=1)
    levels = oracle.codebook(bits, d)
    p = iq.isoq_params_init("full", d, bits, 1, rot=rot, codebook=levels)
    xg = torch.from_numpy(x).cuda()
    xrt = iq.isoq_roundtrip(p, xg)
    idx, rho = iq.isoq_quantize(p, xg)
    torch.cuda.synchronize()
    o = Oracle("full", d, bits, rot, levels, x)
    o.check_indices(oracle.unpack(idx.cpu().numpy(), d, bits))
    o.check_norms(rho.cpu().numpy())
    o.check_xhat(xrt.cpu().numpy(), np.float32)


@pytest.mark.parametrize("bits", [2, 3, 4])
@pytest.mark.parametrize("variant", ["full", "fast", "2d"])
def test_config_fp16_d128_n1m(variant, bits):
    print(f"case {variant} d=128 b={bits} fp16 n=1048576", flush=True)
    full_size_case(variant, 128, bits, 1 << 20, np.float16)


@pytest.mark.parametrize("bits", [2, 3, 4])
@pytest.mark.parametrize("variant", ["full", "fast"])
def test_config_fp16_d256_n1m(variant, bits):
    print(f"case {variant} d=256 b={bits} fp16 n=1048576", flush=True)
    full_size_case(variant, 256, bits, 1 << 20, np.float16)


@pytest.mark.parametrize("bits", [2, 3, 4])
@pytest.mark.parametrize("variant", ["full", "fast"])
def test_config_fp32_d512_n262144(variant, bits):
    print(f"case {variant} d=512 b={bits} fp32 n=262144", flush=True)
    full_size_case(variant, 512, bits, 262144, np.float32, mse_tol=0.01)


def test_config_kv_cache_fast_3bit_quantize():
    """K and V [8, 32, 32768, 128] fp16, one quaternion set per head
    (rows_per_set = 32768, n_sets = 32), Fast, 3 bits, quantize only."""
    B, Hh, T, d, bits = 8, 32, 32768, 128, 3
    rot = workloads.rotation_draws("fast", d, Hh, seed=1)
    levels = oracle.codebook(bits, d)
    p = iq.isoq_params_init("fast", d, bits, Hh, rot=rot, codebook=levels)
    n = B * Hh * T
    rng = np.random.default_rng(8)
    sample = np.unique(np.concatenate([
        (h * T + np.arange(256)) for h in range(Hh)] + [rng.integers(0, n, 16384), [n - 1]]))
    st = torch.from_numpy(sample).cuda()
    for name, seed in (("K", 2), ("V", 3)):
        print(f"case kv {name}", flush=True)
        kv = workloads.kv_stream_torch(B, Hh, T, d, seed, "cuda")
        flat = kv.view(n, d)
        idx, rho = iq.isoq_quantize(p, flat, rows_per_set=T)
        torch.cuda.synchronize()
        x_s = flat[st].cpu().numpy()
        # oracle on the sampled rows, with their true row numbers
        o = Oracle("fast", d, bits, rot, levels, x_s, n_sets=Hh, rows_per_set=T, rows=sample,
                   selected=True)
        o.check_indices(oracle.unpack(idx[st].cpu().numpy(), d, bits))
        o.check_norms(rho[st].cpu().numpy())
        ref_rho = torch.linalg.vector_norm(flat.double(), dim=1)
        assert torch.all((rho.double() - ref_rho).abs() <= 1e-6 * ref_rho).item()
        del kv, flat, idx, rho, ref_rho
        torch.cuda.empty_cache()

