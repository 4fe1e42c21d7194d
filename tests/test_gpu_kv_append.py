"""Quantize-on-append into a paged K/V cache (isoq_kv_append) against the
oracle.  Rows are (token, head) pairs; head h uses rotation set h (or set 0
with one set).  Every written slot must hold the oracle's indices and norm of
its row, every other slot must keep its previous bytes, and the records must
equal those isoq_quantize writes for the same rows, bit for bit.  The cache
placement (slot s -> block s // block_size, position s % block_size, a block
holding [n_heads][block_size] records) is the layout definition of the header,
written out here in numpy.  Needs an MI355X."""
import numpy as np
import pytest

import oracle
import workloads
from cache_layout import from_cache
from parity import Oracle

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

import paper_2603_28430_amd as iq  # noqa: E402

DT = {"f16": (torch.float16, np.float16), "f32": (torch.float32, np.float32)}
CANARY_BYTE, CANARY_RHO = 0xA5, -7.0


def make(variant, d, bits, n_sets, seed):
    rot = workloads.rotation_draws(variant, d, n_sets, seed)
    levels = oracle.codebook(bits, d)
    return iq.isoq_params_init(variant, d, bits, n_sets, rot=rot, codebook=levels), rot, levels


def new_cache(n_blocks, n_heads, block_size, rec):
    idx = torch.full((n_blocks, n_heads, block_size, rec), CANARY_BYTE, dtype=torch.uint8, device="cuda")
    rho = torch.full((n_blocks, n_heads, block_size), CANARY_RHO, dtype=torch.float32, device="cuda")
    return idx, rho


def cache_rows(slots, n_heads, block_size):
    """Flat cache row of (token t, head h), [n_tokens, n_heads]."""
    blk, pos = np.divmod(np.asarray(slots, np.int64), block_size)
    return (blk[:, None] * n_heads + np.arange(n_heads)[None, :]) * block_size + pos[:, None]


def check_tensor(variant, d, bits, rot, levels, n_sets, x, slots, n_heads, block_size, n_blocks,
                 cidx, crho, p, before_idx=None, before_rho=None):
    """x: host rows [n_tokens * n_heads, d]; cidx/crho: the cache after the call."""
    n_slots = n_blocks * block_size
    n_tokens = len(slots)
    rec = p.record_bytes
    ci = from_cache(cidx.cpu().numpy()).reshape(-1, rec)
    cr = crho.cpu().numpy().reshape(-1)
    valid_t = np.flatnonzero((slots >= 0) & (slots < n_slots))
    written = np.zeros(len(cr), bool)
    if len(valid_t):
        crow = cache_rows(slots[valid_t], n_heads, block_size).reshape(-1)
        rows = (valid_t[:, None] * n_heads + np.arange(n_heads)[None, :]).reshape(-1)
        o = Oracle(variant, d, bits, rot, levels, x[rows], n_sets=n_sets, rows_per_set=1, rows=rows,
                   selected=True)
        o.check_indices(oracle.unpack(ci[crow], oracle.padded_width(variant, d), bits))
        o.check_norms(cr[crow])
        # the same records as the plain encoder on the same rows and sets
        xg = torch.from_numpy(np.ascontiguousarray(x)).cuda()
        qi, qr = iq.isoq_quantize(p, xg, 1)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(ci[crow], qi.cpu().numpy()[rows])
        np.testing.assert_array_equal(cr[crow], qr.cpu().numpy()[rows])
        written[crow] = True
    prev_i = np.full_like(ci, CANARY_BYTE) if before_idx is None else from_cache(before_idx).reshape(-1, rec)
    prev_r = np.full_like(cr, CANARY_RHO) if before_rho is None else before_rho.reshape(-1)
    np.testing.assert_array_equal(ci[~written], prev_i[~written])
    np.testing.assert_array_equal(cr[~written], prev_r[~written])
    return int(written.sum())


def slot_mapping(rng, n_tokens, n_slots, skip_frac):
    slots = rng.permutation(n_slots)[:n_tokens].astype(np.int64)
    kill = rng.random(n_tokens) < skip_frac
    k = int(kill.sum())
    neg = -1 - rng.integers(0, 1000, k)
    big = n_slots + rng.integers(0, 1000, k)
    slots[kill] = np.where(rng.random(k) < 0.5, neg, big)
    return slots


def run_case(variant, d, bits, dtype, n_tokens, n_heads, block_size, n_blocks, sets_k, sets_v,
             seed=0, with_v=True, skip_frac=0.1):
    print(f"case {variant} d={d} b={bits} {dtype} tokens={n_tokens} heads={n_heads} "
          f"bs={block_size} blocks={n_blocks} sets={sets_k}/{sets_v} v={with_v}", flush=True)
    tdt, ndt = DT[dtype]
    rng = np.random.default_rng(seed)
    slots = slot_mapping(rng, n_tokens, n_blocks * block_size, skip_frac)
    pk, rot_k, lev = make(variant, d, bits, sets_k, seed=1)
    xk = workloads.unit_gaussian_rows(n_tokens * n_heads, d, seed=seed + 10, dtype=ndt)
    k_idx, k_rho = new_cache(n_blocks, n_heads, block_size, pk.record_bytes)
    st = torch.from_numpy(slots).cuda()
    kg = torch.from_numpy(xk).cuda().view(n_tokens, n_heads, d)
    if with_v:
        pv, rot_v, _ = make(variant, d, bits, sets_v, seed=2)
        xv = workloads.unit_gaussian_rows(n_tokens * n_heads, d, seed=seed + 20, dtype=ndt)
        v_idx, v_rho = new_cache(n_blocks, n_heads, block_size, pv.record_bytes)
        vg = torch.from_numpy(xv).cuda().view(n_tokens, n_heads, d)
        iq.isoq_kv_append(pk, kg, st, k_idx, k_rho, pv, vg, v_idx, v_rho)
    else:
        iq.isoq_kv_append(pk, kg, st, k_idx, k_rho)
    torch.cuda.synchronize()
    w = check_tensor(variant, d, bits, rot_k, lev, sets_k, xk, slots, n_heads, block_size, n_blocks,
                     k_idx, k_rho, pk)
    if with_v:
        check_tensor(variant, d, bits, rot_v, lev, sets_v, xv, slots, n_heads, block_size, n_blocks,
                     v_idx, v_rho, pv)
    return w


@pytest.mark.parametrize("bits", [2, 3, 4])
@pytest.mark.parametrize("variant", ["full", "fast", "2d"])
@pytest.mark.parametrize("dtype", ["f16", "f32"])
def test_append_d128_sets_per_head(variant, bits, dtype):
    run_case(variant, 128, bits, dtype, n_tokens=97, n_heads=8, block_size=16, n_blocks=9,
             sets_k=8, sets_v=8, seed=bits)


@pytest.mark.parametrize("d", [64, 256, 512])
@pytest.mark.parametrize("variant", ["full", "fast"])
def test_append_wide_rows(variant, d):
    run_case(variant, d, 3, "f16", n_tokens=41, n_heads=4, block_size=32, n_blocks=3, sets_k=4,
             sets_v=1, seed=d)


@pytest.mark.parametrize("variant,d,bits", [("full", 96, 3), ("fast", 96, 2), ("2d", 96, 4), ("fast", 160, 3),
                                            ("full", 160, 4), ("full", 192, 3), ("fast", 192, 2), ("2d", 192, 3),
                                            ("fast", 80, 3), ("full", 80, 2), ("2d", 80, 4), ("full", 80, 3)])
def test_append_head_widths(variant, d, bits):
    """fp16 rows at d = 80, 96, 160 and 192 (packed-row kernels; two chunks
    per lane at 192; at 80 and 3 bits lane pairs write the records): sets per
    head for K, one set for V, skipped slots."""
    run_case(variant, d, bits, "f16", n_tokens=97, n_heads=6, block_size=16, n_blocks=9, sets_k=6, sets_v=1,
             seed=d + bits)


@pytest.mark.parametrize("variant,d,n_heads,bs", [("fast", 96, 16, 16), ("full", 160, 8, 16), ("2d", 96, 8, 5),
                                                  ("fast", 192, 8, 1), ("full", 80, 8, 16)])
def test_append_head_widths_xcd_head_order(variant, d, n_heads, bs):
    """Rows of 192 and 320 bytes share cache lines between heads, so with a
    head count that is a multiple of 8 the blocks take heads in XCD order;
    every (token, head) row must still land in its own cache row (odd block
    sizes, one-slot blocks, and 384-byte rows that keep head order)."""
    run_case(variant, d, 3, "f16", n_tokens=150, n_heads=n_heads, block_size=bs, n_blocks=(200 + bs - 1) // bs,
             sets_k=n_heads, sets_v=1, seed=d + n_heads + bs)


@pytest.mark.parametrize("variant,d,bits,dtype", [("fast", 96, 3, "f32"), ("full", 80, 4, "f32"), ("2d", 160, 2, "f32"),
                                                  ("full", 192, 3, "f32"), ("8d", 96, 3, "f32"), ("full", 13, 3, "f16"),
                                                  ("fast", 72, 2, "f32"), ("2d", 98, 3, "f16"), ("full", 100, 4, "f16"),
                                                  ("8d", 40, 2, "f16"), ("fast", 130, 3, "f16"), ("2d", 7, 4, "f32"),
                                                  ("full", 1, 2, "f16"), ("full", 1000, 3, "f32"), ("8d", 9, 4, "f32")])
def test_append_generic_widths(variant, d, bits, dtype):
    """Shapes without a one-launch kernel (fp32 rows at 80, 96, 160 and 192,
    every other width; odd widths, 2-D rows of 4k + 2 coordinates, 8-D rows
    with a partial block): the width-generic encoder, one launch per tensor
    over its (token, head) rows.  Sets per head for K, one set for V, odd
    block size, skipped slots."""
    run_case(variant, d, bits, dtype, n_tokens=53, n_heads=5, block_size=7, n_blocks=10, sets_k=5, sets_v=1,
             seed=d + bits)


@pytest.mark.parametrize("dtype", ["f16", "f32"])
def test_append_generic_many_blocks(dtype):
    """Enough (token, head) rows for many launch blocks of the generic
    encoder, rows of one token spread over several waves' row groups."""
    run_case("fast", 72, 3, dtype, n_tokens=700, n_heads=12, block_size=16, n_blocks=60, sets_k=12, sets_v=12,
             seed=7)


@pytest.mark.parametrize("n_heads,block_size,sets_k,sets_v", [(1, 1, 1, 1), (5, 48, 5, 1),
                                                               (3, 7, 1, 3), (32, 16, 32, 32),
                                                               (40, 64, 1, 1)])
def test_append_shapes_and_sets(n_heads, block_size, sets_k, sets_v):
    n_slots_needed = 70
    n_blocks = (n_slots_needed + block_size - 1) // block_size + 1
    run_case("fast", 128, 3, "f16", n_tokens=min(67, n_blocks * block_size), n_heads=n_heads,
             block_size=block_size, n_blocks=n_blocks, sets_k=sets_k, sets_v=sets_v,
             seed=n_heads * 100 + block_size)


def test_append_keys_only_and_all_skipped():
    run_case("full", 128, 3, "f16", n_tokens=33, n_heads=4, block_size=16, n_blocks=4, sets_k=4,
             sets_v=4, with_v=False, seed=5)
    w = run_case("full", 128, 3, "f16", n_tokens=20, n_heads=4, block_size=16, n_blocks=4, sets_k=4,
                 sets_v=4, skip_frac=1.1, seed=6)
    assert w == 0


def test_append_zero_tokens_is_a_noop():
    pk, _, _ = make("fast", 128, 3, 2, seed=1)
    k_idx, k_rho = new_cache(2, 2, 16, pk.record_bytes)
    empty = torch.empty((0, 2, 128), dtype=torch.float16, device="cuda")
    iq.isoq_kv_append(pk, empty, torch.empty((0,), dtype=torch.int64, device="cuda"), k_idx, k_rho)
    torch.cuda.synchronize()
    assert torch.all(k_idx == CANARY_BYTE).item() and torch.all(k_rho == CANARY_RHO).item()


def test_decode_steps_build_the_same_cache_as_one_encode():
    """A prefill then single-token decode steps for a batch of sequences with
    their own block tables; the cache equals the one-shot encoding of every
    row placed at its slot."""
    variant, d, bits, n_heads, bs, B = "full", 128, 3, 4, 16, 5
    pk, rot, lev = make(variant, d, bits, n_heads, seed=1)
    pv, rot_v, _ = make(variant, d, bits, n_heads, seed=2)
    n_blocks = 40
    rng = np.random.default_rng(3)
    tables = rng.permutation(n_blocks)[:B * 8].reshape(B, 8)   # 8 blocks per sequence
    prefill = rng.integers(1, 40, B)
    steps = 12
    k_idx, k_rho = new_cache(n_blocks, n_heads, bs, pk.record_bytes)
    v_idx, v_rho = new_cache(n_blocks, n_heads, bs, pv.record_bytes)
    all_slots, all_k, all_v = [], [], []

    def slot_of(b, t):
        return tables[b, t // bs] * bs + t % bs

    def append(slots, seed):
        xk = workloads.unit_gaussian_rows(len(slots) * n_heads, d, seed=seed, dtype=np.float16)
        xv = workloads.unit_gaussian_rows(len(slots) * n_heads, d, seed=seed + 5000, dtype=np.float16)
        iq.isoq_kv_append(pk, torch.from_numpy(xk).cuda().view(-1, n_heads, d),
                          torch.tensor(slots, dtype=torch.int64, device="cuda"), k_idx, k_rho, pv,
                          torch.from_numpy(xv).cuda().view(-1, n_heads, d), v_idx, v_rho)
        all_slots.extend(slots)
        all_k.append(xk)
        all_v.append(xv)

    append([slot_of(b, t) for b in range(B) for t in range(prefill[b])], seed=100)
    for s in range(steps):
        append([slot_of(b, prefill[b] + s) for b in range(B)], seed=200 + s)
    torch.cuda.synchronize()
    slots = np.array(all_slots, np.int64)
    check_tensor(variant, d, bits, rot, lev, n_heads, np.concatenate(all_k), slots, n_heads, bs,
                 n_blocks, k_idx, k_rho, pk)
    check_tensor(variant, d, bits, rot_v, lev, n_heads, np.concatenate(all_v), slots, n_heads, bs,
                 n_blocks, v_idx, v_rho, pv)


def test_append_argument_errors():
    pk, _, _ = make("fast", 128, 3, 4, seed=1)
    p3, _, _ = make("fast", 128, 3, 3, seed=1)
    p256, _, _ = make("fast", 256, 3, 1, seed=1)
    k_idx, k_rho = new_cache(2, 4, 16, pk.record_bytes)
    kg = torch.zeros((3, 4, 128), dtype=torch.float16, device="cuda")
    st = torch.arange(3, dtype=torch.int64, device="cuda")
    lib = iq.isoquant.lib

    kp, ip = kg.data_ptr(), k_idx.data_ptr()

    def raw(p_k, p_v, k, v, vi, vr, n_heads=4, ki=ip, bs=16):
        return lib.isoq_kv_append(p_k.handle, None if p_v is None else p_v.handle, iq.ISOQ_F16,
                                  k, v, st.data_ptr(), 3, n_heads, ki, k_rho.data_ptr(), vi, vr, 2,
                                  bs, None)

    assert raw(pk, p3, kp, kp, ip, k_rho.data_ptr()) == 1      # V sets neither 1 nor n_heads
    assert raw(p3, None, kp, None, None, None) == 1              # K sets neither 1 nor n_heads
    assert raw(pk, p256, kp, kp, ip, k_rho.data_ptr()) == 1    # d differs
    assert raw(pk, None, kp, kp, None, None) == 3                # V rows without V handle
    assert raw(pk, None, kp + 2, None, None, None) == 4          # rows not 16-byte aligned
    assert raw(pk, None, kp, None, None, None, ki=ip + 1) == 4   # records not 4-byte aligned
    assert raw(pk, None, kp, None, None, None, n_heads=0) == 1
    assert raw(pk, None, kp, None, None, None, bs=0) == 1
    torch.cuda.synchronize()
    assert torch.all(k_idx == CANARY_BYTE).item(), "an error path launched work"
    with pytest.raises(ValueError):
        iq.isoq_kv_append(pk, kg, st, k_idx[:, :2].contiguous(), k_rho)
