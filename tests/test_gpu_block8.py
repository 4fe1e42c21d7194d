"""8-D grouped blocks (Table 3's block-size axis; Haar(SO(8)) blocks, Sec. 5.7)
through the C ABI against the oracle: the tuned kernels at d = 64, 128, 256
and 512, the packed-row and generic kernels at other widths (zero padding of
the last block when d is not a multiple of 8), several parameter sets, the
exported rotations, and the decoding calls (append into a paged cache, logits
against it).  The parity rule is the one of tests/parity.py.  Needs an MI355X."""
import numpy as np
import pytest

import oracle
import workloads

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

import paper_2603_28430_amd as iq  # noqa: E402
from test_gpu_kv_append import run_case as append_case  # noqa: E402
from test_gpu_kv_scores import run_case as scores_case  # noqa: E402
from test_gpu_parity import check as check_tuned  # noqa: E402
from test_gpu_widths import check as check_width  # noqa: E402


@pytest.mark.parametrize("dtype", ["f16", "f32"])
@pytest.mark.parametrize("bits", [2, 3, 4])
@pytest.mark.parametrize("d", [64, 128, 256, 512])
def test_block8_tuned_widths(d, bits, dtype):
    n = {64: 2075, 128: 1037, 256: 521, 512: 263}[d]
    print(f"case 8d d={d} b={bits} {dtype} n={n}", flush=True)
    check_tuned("8d", d, bits, dtype, n)


def test_block8_many_groups_per_wave():
    d, n = 128, 200_003
    rng = np.random.default_rng(5)
    sample = np.unique(np.concatenate([np.arange(64), np.arange(n - 64, n), rng.integers(0, n, 3000)]))
    print(f"case 8d d={d} b=3 f16 n={n}", flush=True)
    check_tuned("8d", d, 3, "f16", n, sample=sample)


# padded (d mod 8 != 0) and unpadded widths outside the tuned four: the
# generic kernels (8-coordinate slots, 8 to 64 lanes per row, one or two
# slots per lane) and, for fp16 rows of width 16 k up to 504, the packed rows
# (one or two 8-coordinate chunks per lane)
WIDTHS8 = [1, 5, 13, 20, 72, 80, 96, 100, 120, 160, 192, 200, 320, 504, 513, 1000, 1024]


@pytest.mark.parametrize("d", WIDTHS8)
def test_block8_other_widths(d):
    n = 1037 if d <= 256 else 263
    for bits in (2, 3, 4):
        for dtype in ("f16", "f32"):
            print(f"case 8d d={d} b={bits} {dtype} n={n}", flush=True)
            check_width("8d", d, bits, dtype, n, seed=d + bits)


@pytest.mark.parametrize("d,dtype,rows_per_set", [(128, "f16", 64), (128, "f32", 5), (256, "f16", 1),
                                                  (100, "f32", 7), (96, "f16", 480), (96, "f16", 3)])
def test_block8_multiple_sets(d, dtype, rows_per_set):
    print(f"case 8d d={d} {dtype} sets=3 rows_per_set={rows_per_set}", flush=True)
    if d in (64, 128, 256, 512):
        check_tuned("8d", d, 3, dtype, 1500, n_sets=3, rows_per_set=rows_per_set)
    else:
        check_width("8d", d, 3, dtype, 1500, n_sets=3, rows_per_set=rows_per_set)


def test_block8_exported_rotations_are_the_oracles():
    """The library's Householder Q (signs fixed, det +1) equals the oracle's
    Gram-Schmidt Q to fp32 rounding; the seeded init draws the same G as the
    workload generator."""
    d, n_sets = 128, 3
    G = workloads.rotation_draws("8d", d, n_sets, seed=11)
    p = iq.isoq_params_init("8d", d, 3, n_sets, rot=G)
    rot, _, _ = iq.isoq_params_export(p)
    rot = rot.reshape(n_sets, d // 8, 8, 8)
    for s in range(n_sets):
        for i in range(d // 8):
            Q = oracle.orthonormalize8(G.reshape(n_sets, d // 8, 8, 8)[s, i])
            np.testing.assert_allclose(rot[s, i], Q, atol=2e-7)
            assert abs(np.linalg.det(rot[s, i].astype(np.float64)) - 1.0) < 1e-5
    p2 = iq.isoq_params_init("8d", d, 3, n_sets, seed=11)
    np.testing.assert_array_equal(iq.isoq_params_export(p2)[0], iq.isoq_params_export(p)[0])
    p.close()
    p2.close()


def test_block8_zero_rows_and_scale():
    d, bits = 128, 3
    rot = workloads.rotation_draws("8d", d, 1, seed=1)
    lev = oracle.codebook(bits, d)
    p = iq.isoq_params_init("8d", d, bits, 1, rot=rot, codebook=lev)
    x = np.zeros((70, d), np.float32)
    x[1::2] = workloads.unit_gaussian_rows(35, d, seed=3, dtype=np.float32) * 1e3
    xg = torch.from_numpy(x).cuda()
    idx, rho = iq.isoq_quantize(p, xg)
    xh = iq.isoq_roundtrip(p, xg)
    torch.cuda.synchronize()
    idx, rho, xh = idx.cpu().numpy(), rho.cpu().numpy(), xh.cpu().numpy()
    zi = oracle.unpack(idx[0::2], d, bits)
    assert np.all(zi == (1 << bits) // 2 - 1) and np.all(rho[0::2] == 0) and np.all(xh[0::2] == 0)
    o_idx, o_rho, o_xh = oracle.stage1("8d", d, bits, rot, lev, x[1::2])
    g = oracle.unpack(idx[1::2], d, bits)
    o = oracle.stage1("8d", d, bits, rot, lev, x[1::2], want_ytil=True)[3]
    near = np.abs(o[..., None] - oracle.thresholds(bits, lev)).min(-1) <= 1e-6
    assert np.all((g == o_idx) | near)
    np.testing.assert_allclose(rho[1::2], o_rho, rtol=1e-6)


@pytest.mark.parametrize("d,bits,dtype", [(128, 3, "f16"), (128, 2, "f32"), (64, 4, "f16"), (256, 3, "f32"),
                                          (512, 3, "f16")])
def test_block8_append(d, bits, dtype):
    append_case("8d", d, bits, dtype, n_tokens=97, n_heads=4, block_size=16, n_blocks=9, sets_k=4, sets_v=1,
                seed=d + bits)


@pytest.mark.parametrize("d,bits", [(96, 3), (80, 2), (160, 4), (192, 3)])
def test_block8_append_head_widths(d, bits):
    append_case("8d", d, bits, "f16", n_tokens=97, n_heads=6, block_size=16, n_blocks=9, sets_k=6, sets_v=1,
                seed=d + bits)


@pytest.mark.parametrize("d,bits,dtype", [(128, 3, "f16"), (128, 4, "f32"), (64, 2, "f16"), (96, 3, "f16"),
                                          (192, 3, "f32"), (512, 3, "f16")])
def test_block8_scores(d, bits, dtype):
    scores_case("8d", d, bits, dtype, n_seqs=3, n_q=4, n_kv=2, bs=16, seq_lens=[1, 150, 33])
