"""Quantize-on-append of key rows with the stage-2 sketch (isoq_kv_append_qjl).

Each written slot must hold exactly what isoq_quantize_qjl produces for the
same row with the same rotation set and projection (records, norms, sign
sketches and gammas bit for bit: the kernels share the encoder, and a row's
projection does not depend on the other rows of its tile); isoq_quantize_qjl
itself is checked against the oracle in test_gpu_qjl.py.  Every other slot
keeps its canary bytes, skipped slots write nothing, and the cache then
serves isoq_kv_scores_qjl.  Needs an MI355X."""
import numpy as np
import pytest

import workloads
from cache_layout import from_cache

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

import paper_2603_28430_amd as iq  # noqa: E402

CANARY_B, CANARY_F = 0xA5, -7.25


def run_case(variant, d, bits, m, dtype, n_tokens, n_heads, block_size, n_blocks, n_sets, seed, skip_every=0):
    print(f"case {variant} d={d} b={bits} m={m} {dtype} tokens={n_tokens} heads={n_heads} bs={block_size} "
          f"sets={n_sets}", flush=True)
    tdt = torch.float16 if dtype == "f16" else torch.float32
    rot = workloads.rotation_draws(variant, d, n_sets, seed=1)
    p = iq.isoq_params_init(variant, d, bits, n_sets, rot=rot)
    sk = iq.isoq_sketch_init(p, m, S=workloads.qjl_matrix(m, d, seed=seed))
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    x = torch.randn((n_tokens, n_heads, d), generator=g, device="cuda").to(tdt)
    slots = torch.randperm(n_blocks * block_size, generator=g, device="cuda")[:n_tokens].to(torch.int64)
    if skip_every:
        slots[::skip_every] = -1
        slots[1::skip_every] = n_blocks * block_size + 3
    R, mb = p.record_bytes, m // 8
    rec = torch.full((n_blocks, n_heads, block_size, R), CANARY_B, dtype=torch.uint8, device="cuda")
    sg = torch.full((n_blocks, n_heads, block_size, mb), CANARY_B, dtype=torch.uint8, device="cuda")
    rho = torch.full((n_blocks, n_heads, block_size), CANARY_F, dtype=torch.float32, device="cuda")
    gam = torch.full((n_blocks, n_heads, block_size), CANARY_F, dtype=torch.float32, device="cuda")
    iq.isoq_kv_append_qjl(p, sk, x, slots, rec, rho, sg, gam)
    # reference: the row encoder on the same rows, head h with set h (or 0)
    refs = []
    for h in range(n_heads):
        ph = p if n_sets == 1 else iq.isoq_params_init(variant, d, bits, 1,
                                                       rot=rot[h * len(rot) // n_sets:(h + 1) * len(rot) // n_sets])
        skh = sk if n_sets == 1 else iq.isoq_sketch_init(ph, m, S=workloads.qjl_matrix(m, d, seed=seed))
        refs.append([t.cpu().numpy() for t in iq.isoq_quantize_qjl(ph, skh, x[:, h].contiguous())])
    torch.cuda.synchronize()
    rec, sg, rho, gam = from_cache(rec.cpu().numpy()), sg.cpu().numpy(), rho.cpu().numpy(), gam.cpu().numpy()
    s_np = slots.cpu().numpy()
    written = np.zeros((n_blocks, n_heads, block_size), bool)
    tok = np.flatnonzero((s_np >= 0) & (s_np < n_blocks * block_size))
    b, pos = s_np[tok] // block_size, s_np[tok] % block_size
    for h in range(n_heads):
        r_idx, r_rho, r_sg, r_gam = refs[h]
        np.testing.assert_array_equal(rec[b, h, pos], r_idx[tok])
        np.testing.assert_array_equal(sg[b, h, pos], r_sg[tok])
        np.testing.assert_array_equal(rho[b, h, pos].view(np.uint32), r_rho[tok].view(np.uint32))
        np.testing.assert_array_equal(gam[b, h, pos].view(np.uint32), r_gam[tok].view(np.uint32))
        written[b, h, pos] = True
    assert np.all(rec[~written] == CANARY_B) and np.all(sg[~written] == CANARY_B)
    assert np.all(rho[~written] == CANARY_F) and np.all(gam[~written] == CANARY_F)
    return p, sk


@pytest.mark.parametrize("bits", [2, 3, 4])
@pytest.mark.parametrize("variant", ["full", "fast", "2d"])
def test_append_qjl_matches_row_encoder(variant, bits):
    run_case(variant, 128, bits, 128, "f16", n_tokens=150, n_heads=4, block_size=16, n_blocks=12, n_sets=4,
             seed=bits)


@pytest.mark.parametrize("d,m,dtype,n_sets", [(128, 64, "f32", 1), (256, 64, "f16", 2), (256, 64, "f32", 1),
                                              (64, 128, "f16", 2), (64, 64, "f32", 1), (512, 64, "f16", 2),
                                              (512, 64, "f32", 1)])
def test_append_qjl_shapes(d, m, dtype, n_sets):
    run_case("full", d, 3, m, dtype, n_tokens=70, n_heads=2, block_size=8, n_blocks=10, n_sets=n_sets, seed=d)


@pytest.mark.parametrize("variant,d,bits,m,n_sets", [("full", 80, 3, 128, 1), ("fast", 96, 3, 128, 6),
                                                     ("2d", 160, 2, 64, 6), ("full", 192, 4, 128, 6),
                                                     ("fast", 192, 3, 64, 1), ("fast", 80, 2, 64, 6),
                                                     ("2d", 96, 4, 128, 1), ("full", 160, 3, 128, 6)])
def test_append_qjl_head_widths(variant, d, bits, m, n_sets):
    # fp16 rows at the head widths: the packed-row kernels
    run_case(variant, d, bits, m, "f16", n_tokens=97, n_heads=6, block_size=16, n_blocks=9, n_sets=n_sets,
             seed=d + bits)


def test_append_qjl_head_width_decode_and_long():
    run_case("fast", 96, 3, 128, "f16", n_tokens=32, n_heads=8, block_size=16, n_blocks=40, n_sets=8, seed=5,
             skip_every=5)
    run_case("fast", 192, 3, 64, "f16", n_tokens=9000, n_heads=4, block_size=16, n_blocks=600, n_sets=4,
             seed=6, skip_every=97)


def test_append_qjl_decode_step_and_skipped_slots():
    # one token per sequence (a decode step) with some padding slots; and a
    # long append that makes blocks walk several token ranges of their head
    run_case("fast", 128, 3, 128, "f16", n_tokens=32, n_heads=8, block_size=16, n_blocks=40, n_sets=8, seed=5,
             skip_every=5)
    run_case("fast", 128, 3, 128, "f16", n_tokens=20000, n_heads=8, block_size=16, n_blocks=1300, n_sets=8,
             seed=6, skip_every=97)


def test_append_qjl_then_corrected_scores():
    """Keys appended with the sketch, then scored with the correction: the
    logit error against <q, x> averages to zero (residual signs are
    symmetric over i.i.d. keys)."""
    variant, d, bits, m, T, bs = "fast", 128, 2, 128, 8192, 16
    p = iq.isoq_params_init(variant, d, bits, 1, rot=workloads.rotation_draws(variant, d, 1, seed=1))
    sk = iq.isoq_sketch_init(p, m, S=workloads.qjl_matrix(m, d, seed=7))
    x = torch.from_numpy(workloads.unit_gaussian_rows(T, d, seed=3, dtype=np.float16)).cuda().view(T, 1, d)
    nb = T // bs
    perm = torch.randperm(nb, device="cuda").to(torch.int32)
    t = torch.arange(T, device="cuda")
    slots = (perm[t // bs].to(torch.int64) * bs + t % bs)
    rec = torch.zeros((nb, 1, bs, p.record_bytes), dtype=torch.uint8, device="cuda")
    sg = torch.zeros((nb, 1, bs, m // 8), dtype=torch.uint8, device="cuda")
    rho = torch.zeros((nb, 1, bs), dtype=torch.float32, device="cuda")
    gam = torch.zeros((nb, 1, bs), dtype=torch.float32, device="cuda")
    iq.isoq_kv_append_qjl(p, sk, x, slots, rec, rho, sg, gam)
    qv = np.random.default_rng(2).standard_normal(d)
    qv /= np.linalg.norm(qv)
    q = torch.from_numpy(qv.astype(np.float32)).cuda().view(1, 1, d)
    lens = torch.tensor([T], dtype=torch.int32, device="cuda")
    sc = iq.isoq_kv_scores_qjl(p, sk, q, rec, rho, sg, gam, perm.view(1, nb), lens, 1.0)
    torch.cuda.synchronize()
    est = sc.cpu().numpy()[0, 0].astype(np.float64)
    truth = x.view(T, d).cpu().numpy().astype(np.float64) @ qv
    err = est - truth
    assert abs(err.mean()) < 4 * err.std() / np.sqrt(T), (err.mean(), err.std())


def test_append_qjl_argument_errors():
    p = iq.isoq_params_init("fast", 128, 3, 2)
    sk = iq.isoq_sketch_init(p, 128)
    p1 = iq.isoq_params_init("fast", 128, 3, 1)
    z = lambda *s, dt=torch.uint8: torch.zeros(s, dtype=dt, device="cuda")
    x = z(4, 2, 128, dt=torch.float16)
    slots = torch.arange(4, dtype=torch.int64, device="cuda")
    rec, sg = z(2, 2, 16, 48), z(2, 2, 16, 16)
    rho, gam = z(2, 2, 16, dt=torch.float32), z(2, 2, 16, dt=torch.float32)
    with pytest.raises(iq.IsoqError) as e:      # sketch of another handle's shape
        iq.isoq_kv_append_qjl(p1, sk, x, slots, rec, rho, sg, gam)
    assert e.value.status == 1
    with pytest.raises(ValueError):             # sign records of the wrong width
        iq.isoq_kv_append_qjl(p, sk, x, slots, rec, rho, z(2, 2, 16, 8), gam)
    p3 = iq.isoq_params_init("fast", 128, 3, 3)
    sk3 = iq.isoq_sketch_init(p3, 128)
    with pytest.raises(iq.IsoqError) as e:      # 3 sets for 2 heads
        iq.isoq_kv_append_qjl(p3, sk3, x, slots, rec, rho, sg, gam)
    assert e.value.status == 1
    lib = iq.isoquant.lib
    assert lib.isoq_kv_append_qjl(p.handle, sk.handle, 1, x.data_ptr(), slots.data_ptr(), 4, 2, rec.data_ptr(),
                                  rho.data_ptr(), None, gam.data_ptr(), 2, 16, None) == 3


def test_append_qjl_empty_is_a_noop():
    p = iq.isoq_params_init("fast", 128, 3, 1)
    sk = iq.isoq_sketch_init(p, 64)
    x = torch.empty((0, 2, 128), dtype=torch.float16, device="cuda")
    slots = torch.empty((0,), dtype=torch.int64, device="cuda")
    rec = torch.full((2, 2, 16, 48), CANARY_B, dtype=torch.uint8, device="cuda")
    sg = torch.full((2, 2, 16, 8), CANARY_B, dtype=torch.uint8, device="cuda")
    rho = torch.full((2, 2, 16), CANARY_F, dtype=torch.float32, device="cuda")
    gam = torch.full((2, 2, 16), CANARY_F, dtype=torch.float32, device="cuda")
    iq.isoq_kv_append_qjl(p, sk, x, slots, rec, rho, sg, gam)
    torch.cuda.synchronize()
    assert torch.all(rec == CANARY_B) and torch.all(sg == CANARY_B)
    assert torch.all(rho == CANARY_F) and torch.all(gam == CANARY_F)
