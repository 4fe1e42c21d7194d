"""Attention logits with the stage-2 residual correction (isoq_kv_scores_qjl)
against the oracle's two-stage estimate scale * (<q, x_hat> + sqrt(pi/2)/m *
gamma * <S q, 2 z - 1>) (oracle.qjl_inner_product).

Caches are built on the host from the oracle's own encoding of synthetic
keys (records and sign sketches packed by the oracle's packer, norms and
gamma as the oracle computes them), placed by the layout definition of the
header.  Tolerance: the stage-1 term as in test_gpu_kv_scores plus, for the
correction, sqrt(pi/2)/m |scale| gamma (m/4 + d + 16) 2^-23 sum_i sum_j |S_ij q_j|
(S q in fp32 from an fp32 copy of S, m/4 table entries summed in fp32).
The end-to-end test (GPU encode -> cache -> GPU logits) is statistical: the
estimate is unbiased for <q, x> and obeys the QJL variance bound, which
takes no HIP output into the oracle.  Needs an MI355X."""
import numpy as np
import pytest

import oracle
import workloads
from cache_layout import to_cache

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

import paper_2603_28430_amd as iq  # noqa: E402

CANARY = -12345.0


def build(variant, d, bits, m, n_seqs, n_kv, bs, seq_lens, n_sets, seed):
    rng = np.random.default_rng(seed)
    rot = workloads.rotation_draws(variant, d, n_sets, seed=1)
    levels = oracle.codebook(bits, d)
    S = workloads.qjl_matrix(m, d, seed=seed + 3)
    per = oracle.raw_params_per_set(variant, d)
    max_blocks = max(1, max((L + bs - 1) // bs for L in seq_lens))
    n_blocks = n_seqs * max_blocks + 2
    perm = rng.permutation(n_blocks)
    table = np.full((n_seqs, max_blocks), -1, np.int32)
    R = oracle.record_bytes(d, bits)
    rec = np.zeros((n_blocks, n_kv, bs, R), np.uint8)
    rho = np.zeros((n_blocks, n_kv, bs), np.float32)
    sg = np.zeros((n_blocks, n_kv, bs, m // 8), np.uint8)
    gam = np.zeros((n_blocks, n_kv, bs), np.float32)
    keys = {}
    for s in range(n_seqs):
        L = seq_lens[s]
        nb = (L + bs - 1) // bs
        table[s, :nb] = perm[s * max_blocks:s * max_blocks + nb]
        for h in range(n_kv):
            hs = h if n_sets > 1 else 0
            x = workloads.unit_gaussian_rows(L, d, seed=1000 + 17 * s + h, dtype=np.float16)
            z, g, _, idx, r, xh = oracle.qjl_encode(variant, d, bits, rot[hs * per:(hs + 1) * per], levels, S, x)
            keys[s, h] = (x, idx, r.astype(np.float32), z, g.astype(np.float32))
            if L:
                t = np.arange(L)
                blk = table[s, t // bs]
                rec[blk, h, t % bs] = oracle.pack(idx, bits)
                rho[blk, h, t % bs] = r
                sg[blk, h, t % bs] = oracle.pack(z, 1)
                gam[blk, h, t % bs] = g
    return rot, levels, S, table, rec, rho, sg, gam, keys, n_blocks


def run_case(variant, d, bits, m, dtype, n_seqs, n_q, n_kv, bs, seq_lens, n_sets=None, scale=0.088, seed=0):
    print(f"case {variant} d={d} b={bits} m={m} {dtype} heads={n_q}/{n_kv} lens={seq_lens}", flush=True)
    n_sets = n_kv if n_sets is None else n_sets
    rot, levels, S, table, rec, rho, sg, gam, keys, n_blocks = build(variant, d, bits, m, n_seqs, n_kv, bs,
                                                                     seq_lens, n_sets, seed)
    p = iq.isoq_params_init(variant, d, bits, n_sets, rot=rot, codebook=levels)
    sk = iq.isoq_sketch_init(p, m, S=S)
    ndt = np.float16 if dtype == "f16" else np.float32
    rng = np.random.default_rng(seed + 1)
    q = (workloads.unit_gaussian_rows(n_seqs * n_q, d, seed=seed + 7, dtype=np.float64) *
         rng.uniform(0.5, 4.0, (n_seqs * n_q, 1))).astype(ndt).reshape(n_seqs, n_q, d)
    ml = table.shape[1] * bs
    out = torch.full((n_seqs, n_q, ml), CANARY, dtype=torch.float32, device="cuda")
    T = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    iq.isoq_kv_scores_qjl(p, sk, T(q), T(to_cache(rec)), T(rho), T(sg), T(gam), T(table),
                          T(np.asarray(seq_lens, np.int32)), scale, max_len=ml, scores=out)
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    G = n_q // n_kv
    per = oracle.raw_params_per_set(variant, d)
    nf = d // (1 if bits == 4 else 2)
    for (s, h), (x, idx, r, z, g) in keys.items():
        L = len(r)
        hs = h if n_sets > 1 else 0
        xh = oracle.dequantize(variant, d, bits, rot[hs * per:(hs + 1) * per], levels, idx, r) if L else None
        for gi in range(G):
            hq = h * G + gi
            qv = q[s, hq].astype(np.float64)
            if L:
                ref = scale * oracle.qjl_inner_product(qv, xh, z, g, S)
                b1 = (nf + 8) * 2.0 ** -23 * abs(scale) * r * np.linalg.norm(qv) * np.linalg.norm(levels[idx], axis=1)
                b2 = (np.sqrt(np.pi / 2) / m * abs(scale) * g * (m / 4 + d + 16) * 2.0 ** -23 *
                      np.abs(S * qv[None, :]).sum())
                err = np.abs(got[s, hq, :L].astype(np.float64) - ref)
                assert np.all(err <= b1 + b2 + 1e-30), (s, hq, float((err / (b1 + b2)).max()))
            assert np.all(got[s, hq, L:] == CANARY)


@pytest.mark.parametrize("bits", [2, 3, 4])
@pytest.mark.parametrize("variant", ["full", "fast", "2d"])
def test_scores_qjl_d128_m128(variant, bits):
    run_case(variant, 128, bits, 128, "f16", n_seqs=2, n_q=2, n_kv=2, bs=16, seq_lens=[1100, 45], seed=bits)


@pytest.mark.parametrize("d,m,dtype", [(128, 64, "f32"), (256, 64, "f16"), (256, 64, "f32"), (64, 64, "f16"),
                                       (64, 128, "f32")])
def test_scores_qjl_shapes(d, m, dtype):
    run_case("full", d, 3, m, dtype, n_seqs=2, n_q=2, n_kv=2, bs=16, seq_lens=[700, 31], seed=d + m)


@pytest.mark.parametrize("d,m,dtype,bits", [(80, 128, "f16", 3), (96, 64, "f32", 3), (160, 128, "f16", 2),
                                            (192, 64, "f16", 4), (192, 128, "f32", 3), (512, 64, "f16", 3),
                                            (512, 64, "f32", 2)])
def test_scores_qjl_head_widths_and_512(d, m, dtype, bits):
    run_case("fast", d, bits, m, dtype, n_seqs=2, n_q=2, n_kv=2, bs=16, seq_lens=[700, 31], seed=d + m)


@pytest.mark.parametrize("n_q,n_kv,n_sets", [(8, 2, 2), (4, 1, 1), (6, 2, 1)])
def test_scores_qjl_grouped(n_q, n_kv, n_sets):
    run_case("fast", 128, 3, 128, "f16", n_seqs=2, n_q=n_q, n_kv=n_kv, bs=16, seq_lens=[300, 1030],
             n_sets=n_sets, seed=n_q)


def test_scores_qjl_end_to_end_unbiased():
    """Keys encoded by isoq_quantize_qjl on the GPU, placed in a cache, scored
    by isoq_kv_scores_qjl: the logit error against <q, x> averages to zero
    over i.i.d. keys (their residuals are sign-symmetric, the codebook being
    symmetric, so the mean vanishes for any fixed S) and its variance obeys
    the QJL bound; the stage-1 logits equal <q, x_hat> of the GPU's own
    reconstruction."""
    variant, d, bits, m, n_tok, bs = "fast", 128, 2, 128, 8192, 16
    p = iq.isoq_params_init(variant, d, bits, 1, rot=workloads.rotation_draws(variant, d, 1, seed=1))
    S = workloads.qjl_matrix(m, d, seed=5)
    sk = iq.isoq_sketch_init(p, m, S=S)
    x = workloads.unit_gaussian_rows(n_tok, d, seed=3, dtype=np.float16)
    xg = torch.from_numpy(x).cuda()
    idx, rho, sg, gam = iq.isoq_quantize_qjl(p, sk, xg)
    xh = iq.isoq_dequantize(p, idx, rho, dtype=torch.float32)
    # one sequence, blocks in order: cache row t = position t
    nb = n_tok // bs
    rec = to_cache(idx.view(nb, 1, bs, -1))
    cr = rho.view(nb, 1, bs).contiguous()
    cs = sg.view(nb, 1, bs, -1).contiguous()
    cg = gam.view(nb, 1, bs).contiguous()
    table = torch.arange(nb, dtype=torch.int32, device="cuda").view(1, nb)
    lens = torch.tensor([n_tok], dtype=torch.int32, device="cuda")
    qv = np.random.default_rng(2).standard_normal(d)
    qv /= np.linalg.norm(qv)
    q = torch.from_numpy(qv.astype(np.float32)).cuda().view(1, 1, d)
    sc = iq.isoq_kv_scores_qjl(p, sk, q, rec, cr, cs, cg, table, lens, 1.0)
    base = iq.isoq_kv_scores(p, q, rec, cr, table, lens, 1.0)
    torch.cuda.synchronize()
    est = sc.cpu().numpy()[0, 0].astype(np.float64)
    stage1 = base.cpu().numpy()[0, 0].astype(np.float64)
    truth = x.astype(np.float64) @ qv
    err = est - truth
    se = err.std() / np.sqrt(n_tok)
    assert abs(err.mean()) < 4 * se, (err.mean(), se)
    np.testing.assert_allclose(stage1, xh.cpu().numpy().astype(np.float64) @ qv, rtol=1e-4, atol=1e-5)
    r2 = ((x.astype(np.float64) - xh.cpu().numpy()) ** 2).sum(1)
    assert err.var() <= 1.1 * (np.pi / (2 * m) * r2).mean()


def test_scores_qjl_argument_errors():
    p = iq.isoq_params_init("fast", 128, 3, 2)
    sk = iq.isoq_sketch_init(p, 128)
    p1 = iq.isoq_params_init("fast", 128, 3, 1)
    z = lambda *s, dt=torch.uint8: torch.zeros(s, dtype=dt, device="cuda")
    q = z(1, 2, 128, dt=torch.float16)
    rec, rho, sg, gam = z(2, 2, 16, 48), z(2, 2, 16, dt=torch.float32), z(2, 2, 16, 16), z(2, 2, 16, dt=torch.float32)
    tab, lens = z(1, 2, dt=torch.int32), torch.ones((1,), dtype=torch.int32, device="cuda")
    with pytest.raises(iq.IsoqError) as e:     # sketch of another handle
        iq.isoq_kv_scores_qjl(p1, sk, q, rec, rho, sg, gam, tab, lens)
    assert e.value.status == 1
    with pytest.raises(ValueError):            # sign records of the wrong width
        iq.isoq_kv_scores_qjl(p, sk, q, rec, rho, z(2, 2, 16, 8), gam, tab, lens)
    lib = iq.isoquant.lib
    assert lib.isoq_kv_scores_qjl(p.handle, None, 1, q.data_ptr(), 1, 2, 2, rec.data_ptr(), rho.data_ptr(),
                                  sg.data_ptr(), gam.data_ptr(), 2, 16, tab.data_ptr(), 2, lens.data_ptr(),
                                  1.0, gam.data_ptr(), 32, None) == 3
