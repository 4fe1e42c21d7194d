"""Attention logits against a paged cache of quantized keys (isoq_kv_scores)
against the oracle's definition scale * <q, dequantized key>.

Caches are built on the host: index records packed by the oracle's packer
(random indices, or the oracle's own quantization of synthetic keys) and
norms, placed by the header's layout definition (slot of position t of a
sequence: block block_table[t // block_size], position t % block_size; a cache
block holds [n_kv_heads][block_size] records).  No input of the oracle comes
from the HIP path.

Tolerance: the kernel rotates the query in fp32 and sums d/F table entries in
fp32 (F = 2 coordinates per entry for 2 and 3 bits, 1 for 4 bits), so
|s_gpu - s| <= (d/F + 8) * 2^-23 * scale * rho * sum_j |(Tq)_j c_j|, and
sum_j |(Tq)_j c_j| <= ||q|| ||c[idx]|| (Cauchy-Schwarz, T orthogonal).  At
widths without a tuned logit kernel the sum runs over the pw coordinates of
the zero-padded record one by one (fp32 fused multiply-adds): pw + 8 terms.
Needs an MI355X."""
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
TUNED = (64, 80, 96, 128, 160, 192, 256, 512)   # widths with a tuned logit kernel


def sum_terms(variant, d, bits):
    """Rounded additions of the logit sum (see the tolerance above)."""
    if d in TUNED:
        return d // (1 if bits == 4 else 2)
    return oracle.padded_width(variant, d)


def make(variant, d, bits, n_sets, seed=1):
    rot = workloads.rotation_draws(variant, d, n_sets, seed)
    levels = oracle.codebook(bits, d)
    return iq.isoq_params_init(variant, d, bits, n_sets, rot=rot, codebook=levels), rot, levels


class Cache:
    """Host model of a paged key cache: unpacked indices and norms per
    (sequence, kv head, position), packed and scattered into the device layout."""

    def __init__(self, rng, d, bits, n_seqs, n_kv, bs, seq_lens, extra_blocks=3, keys=None, pw=None):
        """pw: coordinates per record (the padded width), default d."""
        pw = d if pw is None else pw
        self.d, self.bits, self.bs, self.n_kv = d, bits, bs, n_kv
        K = 1 << bits
        max_blocks = max(1, max((L + bs - 1) // bs for L in seq_lens))
        self.n_blocks = n_seqs * max_blocks + extra_blocks
        perm = rng.permutation(self.n_blocks)
        self.table = np.full((n_seqs, max_blocks), -1, np.int32)
        for s in range(n_seqs):
            nb = (seq_lens[s] + bs - 1) // bs
            self.table[s, :nb] = perm[s * max_blocks:s * max_blocks + nb]
        R = oracle.record_bytes(pw, bits)
        self.rec = np.zeros((self.n_blocks, n_kv, bs, R), np.uint8)
        self.rho = np.zeros((self.n_blocks, n_kv, bs), np.float32)
        self.idx, self.norms = {}, {}
        for s in range(n_seqs):
            for h in range(n_kv):
                L = seq_lens[s]
                if keys is None:
                    idx = rng.integers(0, K, (L, pw)).astype(np.uint8)
                    rho = rng.uniform(0.2, 2.0, L).astype(np.float32)
                else:
                    idx, rho = keys(s, h, L)
                self.idx[s, h], self.norms[s, h] = idx, rho.astype(np.float32)
                if L:
                    t = np.arange(L)
                    blk = self.table[s, t // bs]
                    self.rec[blk, h, t % bs] = oracle.pack(idx, bits)
                    self.rho[blk, h, t % bs] = rho
        self.seq_lens = np.asarray(seq_lens, np.int32)

    def device(self):
        return (torch.from_numpy(to_cache(self.rec)).cuda(), torch.from_numpy(self.rho).cuda(),
                torch.from_numpy(self.table).cuda(), torch.from_numpy(self.seq_lens).cuda())


def expected(variant, d, bits, rot, levels, n_sets, q, cache, scale, G):
    """Oracle logits and tolerance bounds, per (s, hq): arrays over positions."""
    out = {}
    c = np.asarray(levels, np.float64)
    nf = sum_terms(variant, d, bits)
    for (s, h), idx in cache.idx.items():
        rho = cache.norms[s, h].astype(np.float64)
        for g in range(G):
            hq = h * G + g
            qv = q[s, hq].astype(np.float64)
            if len(rho):
                ref = oracle.attention_scores(variant, d, bits, rot, c, qv, idx, rho, scale,
                                              set_index=h if n_sets > 1 else 0)
                bound = (nf + 8) * 2.0 ** -23 * abs(scale) * rho * np.linalg.norm(qv) * \
                    np.linalg.norm(c[idx], axis=1)
            else:
                ref = bound = np.zeros(0)
            out[s, hq] = (ref, bound)
    return out


def run_case(variant, d, bits, dtype, n_seqs, n_q, n_kv, bs, seq_lens, n_sets=None, scale=0.088,
             max_len=None, seed=0, keys=None):
    print(f"case {variant} d={d} b={bits} {dtype} seqs={n_seqs} heads={n_q}/{n_kv} bs={bs} "
          f"lens={list(seq_lens)[:6]} max_len={max_len}", flush=True)
    rng = np.random.default_rng(seed)
    n_sets = n_kv if n_sets is None else n_sets
    p, rot, levels = make(variant, d, bits, n_sets)
    cache = Cache(rng, d, bits, n_seqs, n_kv, bs, seq_lens, keys=keys, pw=oracle.padded_width(variant, d))
    ndt = np.float16 if dtype == "f16" else np.float32
    q = (workloads.unit_gaussian_rows(n_seqs * n_q, d, seed=seed + 7, dtype=np.float64) *
         rng.uniform(0.5, 4.0, (n_seqs * n_q, 1))).astype(ndt).reshape(n_seqs, n_q, d)
    rec, rho, table, lens = cache.device()
    ml = cache.table.shape[1] * bs if max_len is None else max_len
    out = torch.full((n_seqs, n_q, ml), CANARY, dtype=torch.float32, device="cuda")
    iq.isoq_kv_scores(p, torch.from_numpy(q).cuda(), rec, rho, table, lens, scale, max_len=ml,
                      scores=out)
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    exp = expected(variant, d, bits, rot, levels, n_sets, q, cache, scale, n_q // n_kv)
    for (s, hq), (ref, bound) in exp.items():
        L = min(len(ref), ml)
        err = np.abs(got[s, hq, :L].astype(np.float64) - ref[:L])
        assert np.all(err <= bound[:L] + 1e-30), (s, hq, float((err / np.maximum(bound[:L], 1e-30)).max()))
        assert np.all(got[s, hq, L:] == CANARY), f"positions past the length were written ({s}, {hq})"
    return got, exp


@pytest.mark.parametrize("bits", [2, 3, 4])
@pytest.mark.parametrize("variant", ["full", "fast", "2d"])
@pytest.mark.parametrize("dtype", ["f16", "f32"])
def test_scores_d128(variant, bits, dtype):
    run_case(variant, 128, bits, dtype, n_seqs=3, n_q=4, n_kv=4, bs=16, seq_lens=[1100, 17, 300],
             seed=bits)


@pytest.mark.parametrize("d,bits", [(64, 2), (64, 3), (64, 4), (256, 2), (256, 3), (256, 4), (512, 2), (512, 3),
                                    (512, 4), (80, 2), (80, 3), (80, 4), (96, 2), (96, 3), (96, 4), (160, 2),
                                    (160, 3), (160, 4), (192, 2), (192, 3), (192, 4)])
def test_scores_wide(d, bits):
    run_case("full", d, bits, "f16", n_seqs=2, n_q=2, n_kv=2, bs=32, seq_lens=[1500, 70], seed=d + bits)


@pytest.mark.parametrize("variant,d,bits,dtype", [("fast", 96, 3, "f32"), ("2d", 96, 3, "f16"), ("fast", 160, 3, "f16"),
                                                  ("2d", 192, 2, "f32"), ("fast", 80, 3, "f16"), ("2d", 80, 3, "f32")])
def test_scores_head_widths(variant, d, bits, dtype):
    """Widths 80, 96, 160 and 192: records of 7.5, 9, 15 and 18 words at 3 bits
    (2-, 4- and 8-byte record loads), grouped query heads."""
    run_case(variant, d, bits, dtype, n_seqs=2, n_q=8, n_kv=2, bs=16, seq_lens=[700, 33], seed=d + 3)


@pytest.mark.parametrize("variant,d,bits,dtype", [("full", 100, 3, "f16"), ("fast", 72, 2, "f32"), ("2d", 98, 4, "f16"),
                                                  ("2d", 7, 3, "f32"), ("8d", 40, 3, "f16"), ("8d", 9, 2, "f32"),
                                                  ("full", 13, 4, "f32"), ("fast", 1000, 3, "f16"), ("full", 1, 2, "f16"),
                                                  ("fast", 130, 3, "f32"), ("8d", 1024, 4, "f16"), ("2d", 250, 2, "f32")])
def test_scores_generic_widths(variant, d, bits, dtype):
    """Widths without a tuned logit kernel: records of the zero-padded width
    (odd widths, 2-D rows of 4k + 2 coordinates, 8-D rows with a partial
    block), grouped query heads, a sequence across two chunks."""
    run_case(variant, d, bits, dtype, n_seqs=2, n_q=6, n_kv=3, bs=16, seq_lens=[1100, 37], seed=d + bits)


def test_scores_generic_widths_lengths_and_sets():
    """d = 100: empty, one-token and block-straddling sequences, max_len
    cutting a sequence short, one rotation set for every head."""
    run_case("full", 100, 3, "f16", n_seqs=5, n_q=4, n_kv=2, bs=7, seq_lens=[0, 1, 6, 1025, 2100], max_len=2000,
             n_sets=1, seed=6)


def test_scores_head_widths_lengths():
    """d = 96: empty, one-token and block-straddling sequences, and max_len
    cutting a sequence short."""
    run_case("full", 96, 3, "f16", n_seqs=5, n_q=8, n_kv=8, bs=7, seq_lens=[0, 1, 6, 1025, 2100], max_len=2000,
             seed=5)


@pytest.mark.parametrize("d,bs,n_kv", [(96, 16, 8), (128, 7, 16), (192, 5, 8), (80, 16, 8)])
def test_scores_xcd_head_order(d, bs, n_kv):
    """A head's records of one cache block not ending on a 128-byte line
    (16 x 36, 7 x 48, 5 x 72 bytes) with a multiple of 8 key heads: blocks take
    heads in XCD order, each head's logits must still be its own."""
    run_case("fast", d, 3, "f16", n_seqs=2, n_q=2 * n_kv, n_kv=n_kv, bs=bs, seq_lens=[300, 41], seed=d + bs)


@pytest.mark.parametrize("n_q,n_kv,n_sets", [(8, 2, 2), (8, 2, 1), (6, 1, 1), (32, 8, 8)])
def test_scores_grouped_query_heads(n_q, n_kv, n_sets):
    run_case("fast", 128, 3, "f16", n_seqs=2, n_q=n_q, n_kv=n_kv, bs=16, seq_lens=[600, 45],
             n_sets=n_sets, seed=n_q + n_kv)


def test_scores_lengths_and_truncation():
    # empty, single, partial block, exactly one chunk, across chunks; odd block size
    run_case("full", 128, 3, "f32", n_seqs=6, n_q=2, n_kv=2, bs=7, seq_lens=[0, 1, 6, 1024, 1025, 2600],
             seed=11)
    # max_len shorter than some sequences
    run_case("fast", 128, 3, "f16", n_seqs=3, n_q=2, n_kv=2, bs=16, seq_lens=[300, 90, 0], max_len=100,
             seed=12)


@pytest.mark.parametrize("d", [128, 100])
def test_scores_invalid_blocks_are_skipped(d):
    rng = np.random.default_rng(4)
    bits, bs = 3, 16
    p, rot, levels = make("full", d, bits, 2)
    cache = Cache(rng, d, bits, 2, 2, bs, [100, 64], pw=oracle.padded_width("full", d))
    cache.table[0, 1] = -1                       # positions 16..31 of sequence 0
    cache.table[1, 2] = cache.n_blocks + 5       # positions 32..47 of sequence 1
    rec, rho, table, lens = cache.device()
    q = torch.from_numpy(workloads.unit_gaussian_rows(4, d, seed=5, dtype=np.float16)).cuda().view(2, 2, d)
    ml = cache.table.shape[1] * bs
    out = torch.full((2, 2, ml), CANARY, dtype=torch.float32, device="cuda")
    iq.isoq_kv_scores(p, q, rec, rho, table, lens, 1.0, max_len=ml, scores=out)
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    assert np.all(got[0, :, 16:32] == CANARY) and np.all(got[1, :, 32:48] == CANARY)
    assert np.all(got[0, :, :16] != CANARY) and np.all(got[0, :, 32:100] != CANARY)
    assert np.all(got[1, :, :32] != CANARY) and np.all(got[1, :, 48:64] != CANARY)


def test_scores_allocated_by_the_binding_are_minus_inf_where_not_written():
    """Positions the kernel leaves alone (past a sequence's length, behind an
    invalid block-table entry) read as -inf in a scores tensor the binding
    allocates, and every written logit equals the one written into a
    caller's buffer."""
    rng = np.random.default_rng(6)
    d, bits, bs = 128, 3, 16
    p, rot, levels = make("fast", d, bits, 2)
    cache = Cache(rng, d, bits, 2, 2, bs, [100, 37])
    cache.table[0, 2] = -1                       # positions 32..47 of sequence 0
    rec, rho, table, lens = cache.device()
    q = torch.from_numpy(workloads.unit_gaussian_rows(4, d, seed=8, dtype=np.float16)).cuda().view(2, 2, d)
    ml = cache.table.shape[1] * bs
    got = iq.isoq_kv_scores(p, q, rec, rho, table, lens, 0.5, max_len=ml)
    ref = torch.full((2, 2, ml), CANARY, dtype=torch.float32, device="cuda")
    iq.isoq_kv_scores(p, q, rec, rho, table, lens, 0.5, max_len=ml, scores=ref)
    torch.cuda.synchronize()
    got, ref = got.cpu().numpy(), ref.cpu().numpy()
    written = ref != CANARY
    assert np.all(np.isneginf(got[~written]))
    np.testing.assert_array_equal(got[written], ref[written])
    assert not written[0, :, 32:48].any() and not written[0, :, 100:].any() and not written[1, :, 37:].any()
    assert written[0, :, :32].all() and written[1, :, :37].all()


def test_scores_of_keys_quantized_by_the_oracle():
    """Realistic keys: the oracle's own quantization of unit Gaussian rows with
    the rotation of their head (AR(1)-free, seed-fixed)."""
    variant, d, bits = "fast", 128, 3
    _, rot, levels = make(variant, d, bits, 4)

    def keys(s, h, L):
        x = workloads.unit_gaussian_rows(L, d, seed=1000 + 10 * s + h, dtype=np.float16)
        per = oracle.raw_params_per_set(variant, d)
        idx, rho, _ = oracle.stage1(variant, d, bits, rot[h * per:(h + 1) * per], levels, x)
        return idx, rho

    run_case(variant, d, bits, "f16", n_seqs=2, n_q=4, n_kv=4, bs=16, seq_lens=[700, 333], keys=keys,
             seed=21)


@pytest.mark.parametrize("variant,d", [("full", 128), ("full", 96), ("fast", 192), ("2d", 80), ("fast", 100),
                                       ("2d", 90), ("8d", 44)])
def test_append_then_scores_end_to_end(variant, d):
    """Keys appended by isoq_kv_append, logits from isoq_kv_scores, against
    the oracle's logits of the oracle's quantization of the same key rows
    (keys with a coordinate within 1e-6 of a threshold, where either cell is
    admissible, are left out)."""
    bits, H, bs = 3, 4, 16
    pk, rot, levels = make(variant, d, bits, H)
    n_tok = 900
    x = workloads.unit_gaussian_rows(n_tok * H, d, seed=31, dtype=np.float16)
    n_blocks = (n_tok + bs - 1) // bs + 2
    rng = np.random.default_rng(8)
    table = rng.permutation(n_blocks)[:(n_tok + bs - 1) // bs].astype(np.int32)
    slots = (table[np.arange(n_tok) // bs] * bs + np.arange(n_tok) % bs).astype(np.int64)
    R = pk.record_bytes
    k_idx = torch.zeros((n_blocks, H, bs, R), dtype=torch.uint8, device="cuda")
    k_rho = torch.zeros((n_blocks, H, bs), dtype=torch.float32, device="cuda")
    iq.isoq_kv_append(pk, torch.from_numpy(x).cuda().view(n_tok, H, d), torch.from_numpy(slots).cuda(),
                      k_idx, k_rho)
    q = torch.from_numpy(workloads.unit_gaussian_rows(H, d, seed=32, dtype=np.float16)).cuda().view(1, H, d)
    scores = iq.isoq_kv_scores(pk, q, k_idx, k_rho, torch.from_numpy(table[None]).cuda(),
                               torch.tensor([n_tok], dtype=torch.int32, device="cuda"), 0.1)
    torch.cuda.synchronize()
    got = scores.cpu().numpy()[0]
    per = oracle.raw_params_per_set(variant, d)
    thr = oracle.thresholds(bits, levels)
    kept = 0
    for h in range(H):
        xh = x.reshape(n_tok, H, d)[:, h]
        rot_h = rot[h * per:(h + 1) * per]
        idx, rho, _, yt = oracle.stage1(variant, d, bits, rot_h, levels, xh, want_ytil=True)
        near = (np.abs(yt[..., None] - thr).min(-1) <= 1e-6).any(1)
        qv = q.cpu().numpy()[0, h].astype(np.float64)
        ref = oracle.attention_scores(variant, d, bits, rot_h, levels, qv, idx, rho, 0.1)
        bound = (sum_terms(variant, d, bits) + 8) * 2.0 ** -23 * 0.1 * rho * np.linalg.norm(qv) * np.linalg.norm(levels[idx], axis=1)
        ok = ~near
        kept += ok.sum()
        err = np.abs(got[h, :n_tok].astype(np.float64) - ref)
        assert np.all(err[ok] <= bound[ok] + 1e-30), float((err[ok] / bound[ok]).max())
    assert kept >= 0.99 * n_tok * H


def test_scores_argument_errors():
    p, _, _ = make("fast", 128, 3, 3)
    lib = iq.isoquant.lib
    q = torch.zeros((1, 4, 128), dtype=torch.float16, device="cuda")
    rec = torch.zeros((2, 4, 16, 48), dtype=torch.uint8, device="cuda")
    rho = torch.zeros((2, 4, 16), dtype=torch.float32, device="cuda")
    tab = torch.zeros((1, 2), dtype=torch.int32, device="cuda")
    lens = torch.ones((1,), dtype=torch.int32, device="cuda")
    out = torch.full((1, 4, 32), CANARY, dtype=torch.float32, device="cuda")

    def raw(n_q=4, n_kv=4, scale=1.0, qp=None, recp=None, bs=16):
        return lib.isoq_kv_scores(p.handle, iq.ISOQ_F16, qp or q.data_ptr(), 1, n_q, n_kv,
                                  recp or rec.data_ptr(), rho.data_ptr(), 2, bs, tab.data_ptr(), 2,
                                  lens.data_ptr(), scale, out.data_ptr(), 32, None)

    assert raw() == 1                          # 3 sets for 4 kv heads
    p4, _, _ = make("fast", 128, 3, 4)
    p = p4
    assert raw(n_q=6, n_kv=4) == 1             # query heads not a multiple of kv heads
    assert raw(scale=float("inf")) == 1
    assert raw(bs=0) == 1
    assert raw(qp=q.data_ptr() + 2) == 4       # queries not 16-byte aligned
    assert raw(recp=rec.data_ptr() + 4) == 4   # records not 16-byte aligned
    torch.cuda.synchronize()
    assert torch.all(out == CANARY).item(), "an error path launched work"
    assert raw() == 0
