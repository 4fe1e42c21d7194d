"""The decoding-side calls at the sizes and launch configurations bench.py
times, on sampled outputs the oracle computes one by one, plus properties
that hold for every output.

- isoq_kv_append, 8 sequences x 4,096 tokens x 32 heads, K and V, d = 128
  and the head widths 80, 96, 192 (packed rows), Fast, 3 bits, fp16, one
  rotation set per head, 16-position blocks placed at
  random: sampled slots against the oracle's quantization of their rows
  (tests/parity.py rule); every slot against isoq_quantize of the same rows
  (bit for bit); untouched slots keep their canary.
- isoq_kv_scores (d = 128, 80, 96, 192) and isoq_kv_scores_qjl (d = 128,
  m = 128), 8 sequences x 32 heads x 32,768 positions: the cache holds
  seeded random records, norms, sign
  sketches and gammas drawn on the host; sampled logits against
  oracle.attention_scores / oracle.qjl_inner_product with the tolerances of
  test_gpu_kv_scores.py and test_gpu_kv_scores_qjl.py.
- isoq_quantize_qjl, 1,048,576 fp16 rows, m = 128: records and norms equal
  isoq_quantize's for every row; sampled rows' signs and gammas against the
  oracle with the error band of test_gpu_qjl.py.
- isoq_kv_append_qjl, the keys of the prefill above (m = 128, one rotation
  set per head): every slot's record, norm, sign sketch and gamma equal
  isoq_quantize_qjl's for the same row (bit for bit), untouched slots keep
  their canary; the row encoder itself is checked against the oracle above
  and in test_gpu_qjl.py.
Needs an MI355X."""
import numpy as np
import pytest

import oracle
import workloads
from cache_layout import from_cache, to_cache
from parity import Oracle

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

import paper_2603_28430_amd as iq  # noqa: E402

D, BITS = 128, 3


# d = 128 (the tuned append) and the head widths the bench also times (packed
# rows; 80 keeps its 30-byte records whole in the cache, 192 has 8-byte pieces)
@pytest.mark.parametrize("D", [128, 80, 96, 192])
def test_kv_append_prefill_full_size(D):
    H, n_seq, per_seq, bs = 32, 8, 4096, 16
    T = n_seq * per_seq
    n_blocks = 2 * T // bs
    print(f"case kv append {n_seq}x{per_seq} tokens x {H} heads d={D}", flush=True)
    levels = oracle.codebook(BITS, D)
    rk = workloads.rotation_draws("fast", D, H, seed=1)
    rv = workloads.rotation_draws("fast", D, H, seed=2)
    pk = iq.isoq_params_init("fast", D, BITS, H, rot=rk, codebook=levels)
    pv = iq.isoq_params_init("fast", D, BITS, H, rot=rv, codebook=levels)
    k = workloads.kv_stream_torch(1, H, T, D, 2, "cuda")[0].transpose(0, 1).contiguous()   # [T, H, d]
    v = workloads.kv_stream_torch(1, H, T, D, 3, "cuda")[0].transpose(0, 1).contiguous()
    g = torch.Generator(device="cuda")
    g.manual_seed(11)
    blocks_per_seq = per_seq // bs
    tables = torch.randperm(n_blocks, device="cuda", generator=g)[: n_seq * blocks_per_seq].view(n_seq, -1)
    pos = torch.arange(per_seq, device="cuda")
    slots = (tables[:, pos // bs] * bs + pos % bs).reshape(-1).to(torch.int64)
    R = pk.record_bytes
    caches = [torch.full((n_blocks, H, bs, R), 0xA5, dtype=torch.uint8, device="cuda") for _ in range(2)]
    rhos = [torch.full((n_blocks, H, bs), -5.0, dtype=torch.float32, device="cuda") for _ in range(2)]
    iq.isoq_kv_append(pk, k, slots, caches[0], rhos[0], pv, v, caches[1], rhos[1])
    # every row against the row encoder: rows [T * H] with set h = row mod H
    for p, x, cache, rho in ((pk, k, caches[0], rhos[0]), (pv, v, caches[1], rhos[1])):
        ri, rr = iq.isoq_quantize(p, x.view(T * H, D), rows_per_set=1)
        s = slots.view(T, 1)
        blk, off = s // bs, s % bs
        hh = torch.arange(H, device="cuda").view(1, H)
        got_i = from_cache(cache)[blk, hh, off]          # [T, H, R]
        got_r = rho[blk, hh, off]            # [T, H]
        assert torch.equal(got_i.view(T * H, R), ri)
        assert torch.equal(got_r.view(T * H), rr)
        written = torch.zeros((n_blocks, H, bs), dtype=torch.bool, device="cuda")
        written[blk, hh, off] = True
        assert bool(torch.all(cache[~written] == 0xA5)) and bool(torch.all(rho[~written] == -5.0))
    # sampled (token, head) rows against the oracle
    rng = np.random.default_rng(3)
    t = rng.integers(0, T, 3000)
    h = rng.integers(0, H, 3000)
    rows = np.unique(t * H + h)
    s_np = slots.cpu().numpy()
    for rot, x, cache, rho in ((rk, k, caches[0], rhos[0]), (rv, v, caches[1], rhos[1])):
        xs = x.view(T * H, D)[torch.from_numpy(rows).cuda()].cpu().numpy()
        o = Oracle("fast", D, BITS, rot, levels, xs, n_sets=H, rows_per_set=1, rows=rows, selected=True)
        tt, hh = rows // H, rows % H
        blk, off = s_np[tt] // bs, s_np[tt] % bs
        c_np, r_np = from_cache(cache.cpu().numpy()), rho.cpu().numpy()
        o.check_indices(oracle.unpack(c_np[blk, hh, off], D, BITS))
        o.check_norms(r_np[blk, hh, off])


def _random_cache(B, H, T, bs, m, seed, D=D):
    rng = np.random.default_rng(seed)
    nb = B * T // bs
    R = D * BITS // 8
    rec = rng.integers(0, 256, (nb, H, bs, R), dtype=np.uint8)
    rho = rng.uniform(0.5, 1.5, (nb, H, bs)).astype(np.float32)
    sg = rng.integers(0, 256, (nb, H, bs, m // 8), dtype=np.uint8) if m else None
    gam = rng.uniform(0.0, 0.3, (nb, H, bs)).astype(np.float32) if m else None
    table = rng.permutation(nb).astype(np.int32).reshape(B, T // bs)
    q = rng.standard_normal((B, H, D)).astype(np.float16)
    return rec, rho, sg, gam, table, q


# d = 128 with and without the sketch; the head widths the bench also times
@pytest.mark.parametrize("m,D", [(0, 128), (128, 128), (0, 80), (0, 96), (0, 192)])
def test_kv_scores_full_size(m, D):
    B, H, T, bs, scale = 8, 32, 32768, 16, 0.0884
    print(f"case kv scores {B}x{H}x{T} d={D} m={m}", flush=True)
    levels = oracle.codebook(BITS, D)
    rot = workloads.rotation_draws("fast", D, H, seed=1)
    p = iq.isoq_params_init("fast", D, BITS, H, rot=rot, codebook=levels)
    rec, rho, sg, gam, table, q = _random_cache(B, H, T, bs, m, seed=21 + m + D, D=D)
    T_ = lambda a: torch.from_numpy(a).cuda()
    lens = torch.full((B,), T, dtype=torch.int32, device="cuda")
    if m:
        S = workloads.qjl_matrix(m, D, seed=9)
        sk = iq.isoq_sketch_init(p, m, S=S)
        out = iq.isoq_kv_scores_qjl(p, sk, T_(q), T_(to_cache(rec)), T_(rho), T_(sg), T_(gam), T_(table), lens, scale,
                                    max_len=T)
    else:
        out = iq.isoq_kv_scores(p, T_(q), T_(to_cache(rec)), T_(rho), T_(table), lens, scale, max_len=T)
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    assert np.all(np.isfinite(got))
    rng = np.random.default_rng(4)
    n = 2000
    ss, hh, tt = rng.integers(0, B, n), rng.integers(0, H, n), rng.integers(0, T, n)
    c = levels.astype(np.float64)
    nf = D // 2
    for s, h, t in zip(ss, hh, tt):
        blk, off = table[s, t // bs], t % bs
        idx = oracle.unpack(rec[blk, h, off][None], D, BITS)
        r = rho[blk, h, off:off + 1].astype(np.float64)
        qv = q[s, h].astype(np.float64)
        ref = oracle.attention_scores("fast", D, BITS, rot, c, qv, idx, r, scale, set_index=h)[0]
        bound = (nf + 8) * 2.0 ** -23 * scale * r[0] * np.linalg.norm(qv) * np.linalg.norm(c[idx[0]])
        if m:
            z = oracle.unpack(sg[blk, h, off][None], m, 1)
            g_ = gam[blk, h, off:off + 1].astype(np.float64)
            xh = oracle.dequantize("fast", D, BITS, rot[h * len(rot) // H:(h + 1) * len(rot) // H], c, idx, r)
            ref = scale * oracle.qjl_inner_product(qv, xh, z, g_, S)[0]
            bound += (np.sqrt(np.pi / 2) / m * scale * g_[0] * (m / 4 + D + 16) * 2.0 ** -23 *
                      np.abs(S * qv[None, :]).sum())
        err = abs(float(got[s, h, t]) - ref)
        assert err <= bound + 1e-30, (s, h, t, err, bound)


def test_quantize_qjl_full_size():
    n, m = 1 << 20, 128
    print(f"case quantize qjl n={n} m={m}", flush=True)
    levels = oracle.codebook(BITS, D)
    rot = workloads.rotation_draws("full", D, 1, seed=1)
    p = iq.isoq_params_init("full", D, BITS, 1, rot=rot, codebook=levels)
    S = workloads.qjl_matrix(m, D, seed=13)
    sk = iq.isoq_sketch_init(p, m, S=S)
    x = workloads.unit_gaussian_rows(n, D, seed=0, dtype=np.float16)
    xg = torch.from_numpy(x).cuda()
    idx, rho, sg, gam = iq.isoq_quantize_qjl(p, sk, xg)
    qi, qr = iq.isoq_quantize(p, xg)
    torch.cuda.synchronize()
    assert torch.equal(idx, qi) and torch.equal(rho, qr)
    rng = np.random.default_rng(5)
    rows = np.unique(np.concatenate([np.arange(64), np.arange(n - 64, n), rng.integers(0, n, 3000)]))
    xs = x[rows]
    signs = oracle.unpack(sg[torch.from_numpy(rows).cuda()].cpu().numpy(), m, 1)
    gamma = gam[torch.from_numpy(rows).cuda()].cpu().numpy().astype(np.float64)
    z, g_o, p_o, idx_o, rho_o, _ = oracle.qjl_encode("full", D, BITS, rot, levels, S, xs)
    _, _, _, yt = oracle.stage1("full", D, BITS, rot, levels, xs, want_ytil=True)
    thr = oracle.thresholds(BITS, levels)
    keep = ~(np.abs(yt[..., None] - thr).min(-1) <= 1e-6).any(1)
    e = yt - levels[idx_o]
    Sp = np.stack([oracle.encode("full", D, rot, Si) for Si in S])     # S T^-1 rows
    tau = 2 * rho_o[:, None] * ((2.0 ** -10 + 8e-6) * (np.abs(e) @ np.abs(Sp).T) + 6e-7 * np.abs(Sp).sum(1)[None])
    decided = (np.abs(p_o) > tau) & keep[:, None]
    assert not (decided & (signs != z)).any()
    assert (signs == z)[keep].mean() >= 0.97
    assert np.all(np.abs(gamma - g_o)[keep] <= 2e-5 * rho_o[keep] + 1e-30)


def test_kv_append_qjl_prefill_full_size():
    H, n_seq, per_seq, bs, m = 32, 8, 4096, 16, 128
    T = n_seq * per_seq
    n_blocks = 2 * T // bs
    print(f"case kv append qjl {n_seq}x{per_seq} tokens x {H} heads m={m}", flush=True)
    levels = oracle.codebook(BITS, D)
    rot = workloads.rotation_draws("fast", D, H, seed=1)
    S = workloads.qjl_matrix(m, D, seed=17)
    p = iq.isoq_params_init("fast", D, BITS, H, rot=rot, codebook=levels)
    sk = iq.isoq_sketch_init(p, m, S=S)
    k = workloads.kv_stream_torch(1, H, T, D, 2, "cuda")[0].transpose(0, 1).contiguous()   # [T, H, d]
    g = torch.Generator(device="cuda")
    g.manual_seed(12)
    tables = torch.randperm(n_blocks, device="cuda", generator=g)[: n_seq * (per_seq // bs)].view(n_seq, -1)
    pos = torch.arange(per_seq, device="cuda")
    slots = (tables[:, pos // bs] * bs + pos % bs).reshape(-1).to(torch.int64)
    R, mb = p.record_bytes, m // 8
    rec = torch.full((n_blocks, H, bs, R), 0xA5, dtype=torch.uint8, device="cuda")
    sg = torch.full((n_blocks, H, bs, mb), 0xA5, dtype=torch.uint8, device="cuda")
    rho = torch.full((n_blocks, H, bs), -5.0, dtype=torch.float32, device="cuda")
    gam = torch.full((n_blocks, H, bs), -5.0, dtype=torch.float32, device="cuda")
    iq.isoq_kv_append_qjl(p, sk, k, slots, rec, rho, sg, gam)
    blk, off = slots // bs, slots % bs
    got_i, got_s = from_cache(rec), sg
    per = len(rot) // H
    for h in range(H):
        ph = iq.isoq_params_init("fast", D, BITS, 1, rot=rot[h * per:(h + 1) * per], codebook=levels)
        skh = iq.isoq_sketch_init(ph, m, S=S)
        ri, rr, rs, rg = iq.isoq_quantize_qjl(ph, skh, k[:, h].contiguous())
        assert torch.equal(got_i[blk, h, off], ri), h
        assert torch.equal(got_s[blk, h, off], rs), h
        assert torch.equal(rho[blk, h, off].view(torch.int32), rr.view(torch.int32)), h
        assert torch.equal(gam[blk, h, off].view(torch.int32), rg.view(torch.int32)), h
        skh.close()
        ph.close()
    written = torch.zeros((n_blocks, H, bs), dtype=torch.bool, device="cuda")
    written[blk.view(T, 1), torch.arange(H, device="cuda").view(1, H), off.view(T, 1)] = True
    assert bool(torch.all(rec[~written] == 0xA5)) and bool(torch.all(sg[~written] == 0xA5))
    assert bool(torch.all(rho[~written] == -5.0)) and bool(torch.all(gam[~written] == -5.0))
