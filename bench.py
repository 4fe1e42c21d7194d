#!/usr/bin/env python3
"""Throughput of the IsoQuant stage-1 path on one MI355X.

One step = one fused quantize->dequantize pass (isoq_roundtrip) over the whole
batch: 1,048,576 unit-norm Gaussian fp16 vectors, d = 128, 3 bits,
IsoQuant-Full (the headline configuration).  Inputs are resident in HBM
before timing starts; the timed loop rotates over several input/output buffer
sets so that the 256 MB Infinity Cache cannot serve them.  Timing uses HIP
events on the stream the kernels are launched on.  The JSON line also carries
the roofline of the kernel (algorithmic bytes per launch / average launch
time against 8 TB/s), the HBM traffic counted by rocprofv3 when a profile of
the same kernel source is committed under profiles/, side measurements
(quantize, dequantize, other variants and bit widths, a plain device copy of
the same size) and the CPU oracle timed on a bounded sample on the host.

    python bench.py [--steps K] [--warmup W] [--variant full|fast|2d] [--bits 3]
                    [--d 128] [--dtype f16|f32] [--n N] [--mode roundtrip|quantize|dequantize]
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import threading
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBPS = 8000.0          # MI355X HBM3E, vendor figure
METRIC = "fused quant-dequant vectors/s + effective HBM GB/s (% peak), d=128 3-bit fp16"
# every source the round-trip kernels are compiled from (the VALU encoder and,
# for fp16 rows at d = 64, 128 and 256, the matrix-core one)
KERNEL_SRCS = [os.path.join(ROOT, "paper_2603_28430_amd", "csrc", f)
               for f in ("isoq_kernels.hip", "isoq_kernels.h", "isoq_kernels_m.hip", "isoq_stage1.h",
                         "isoq_stage1m.h", "isoq_device.h", "isoq_internal.h")]
PROFILES = os.path.join(ROOT, "profiles")


def kernel_source_hash() -> str:
    h = hashlib.sha256()
    for path in KERNEL_SRCS:
        with open(path, "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def algorithmic_bytes(mode: str, n: int, d: int, bits: int, esz: int) -> int:
    """Bytes one launch must move: rows in/out, packed records (d*bits/8) and
    fp32 norms; rotation parameters and codebook (a few KB) are left out."""
    rec = (d * bits + 7) // 8
    if mode == "roundtrip":
        return n * 2 * d * esz
    if mode == "quantize":
        return n * (d * esz + rec + 4)
    return n * (rec + 4 + d * esz)


def kernel_name(variant: str, d: int, bits: int, dtype: str, mode: str) -> str:
    """The kernel a stage-1 launch runs: fp16 rows at d = 64, 128 and 256
    (Full, Fast, 8-D) take the matrix-core encoder, everything else the VALU
    one."""
    quad = dtype == "f16" and variant != "2d" and d in (64, 128, 256) and mode != "dequantize"
    return f"{'stage1m_kernel' if quad else 'stage1_kernel'}<{variant},{d},{bits},{dtype},{mode}>"


def measured_traffic(tag: str):
    """HBM bytes per launch from a committed rocprofv3 PMC summary of the same
    kernel source (or None)."""
    path = os.path.join(PROFILES, f"{tag}_pmc.md")
    if not os.path.exists(path):
        return None
    text = open(path).read()
    m = re.search(r"kernel_source_sha256:\s*([0-9a-f]+)", text)
    t = re.search(r"hbm_bytes_per_launch:\s*([0-9.eE+]+)", text)
    if not m or not t or m.group(1) != kernel_source_hash():
        return None
    return float(t.group(1))


def time_launches(fn, steps: int, warmup: int, torch, warm_seconds: float = 0.0):
    """Average milliseconds per launch over `steps` launches (events on the
    current stream, which is the stream every launch uses).  Before timing:
    `warmup` launches, then more until `warm_seconds` have passed (the first
    launches after a pause run at lower clocks)."""
    for i in range(warmup):
        fn(i)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    while time.perf_counter() - t0 < warm_seconds:
        for i in range(20):
            fn(i)
        torch.cuda.synchronize()
    s = torch.cuda.Event(enable_timing=True)
    e = torch.cuda.Event(enable_timing=True)
    s.record()
    for i in range(steps):
        fn(i)
    e.record()
    e.synchronize()
    torch.cuda.synchronize()
    return s.elapsed_time(e) / steps


# Host threads for the CPU baseline: the CPU share of one GPU on the GPU
# boxes (16 cores per GPU), or fewer where fewer are available.
CPU_SHARE = 16


def graph_launch_us(fn, launches, torch, replays=20):
    """Device time per launch of `fn` with the host out of the way: `launches`
    calls captured in one HIP graph on a side stream (the binding launches on
    the current stream, which is the capture stream inside the capture),
    replayed `replays` times between HIP events.  None if capture fails."""
    try:
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            fn(0)
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=side):
            for i in range(launches):
                fn(i)
        g.replay()
        torch.cuda.synchronize()
        s = torch.cuda.Event(enable_timing=True)
        e = torch.cuda.Event(enable_timing=True)
        s.record()
        for _ in range(replays):
            g.replay()
        e.record()
        e.synchronize()
        return s.elapsed_time(e) * 1e3 / (replays * launches)
    except Exception as exc:  # capture unsupported: report the host-bound time only
        print(f"# graph timing unavailable: {exc}", file=sys.stderr, flush=True)
        return None


def cpu_baseline(variant, d, bits, x_np, rot, levels, seconds: float):
    """The oracle (plain C, double precision) on the first rows of the same
    workload, rows split across host threads (all the cores of one GPU's CPU
    share), and on one thread.  Returns the JSON object."""
    import numpy as np

    import oracle

    try:
        avail = len(os.sched_getaffinity(0))
    except AttributeError:
        avail = os.cpu_count() or 1
    threads = max(1, min(CPU_SHARE, avail))
    probe = 2000
    xd = np.ascontiguousarray(x_np[:probe], dtype=np.float64)
    rho = np.zeros(probe)
    xh = np.zeros((probe, d))
    t0 = time.perf_counter()
    oracle.stage1_range(variant, d, bits, rot, levels, xd, 0, probe, rho=rho, xh=xh)
    per_row = (time.perf_counter() - t0) / probe
    # one thread: a bounded sample of about a quarter of the time budget
    rows1 = int(min(len(x_np), max(1000, 0.25 * seconds / per_row)))
    x1 = np.ascontiguousarray(x_np[:rows1], dtype=np.float64)
    r1, h1 = np.zeros(rows1), np.zeros((rows1, d))
    t0 = time.perf_counter()
    oracle.stage1_range(variant, d, bits, rot, levels, x1, 0, rows1, rho=r1, xh=h1)
    single = rows1 / (time.perf_counter() - t0)
    rows = int(min(len(x_np), max(threads * 1000, seconds * threads / per_row)))
    xd = np.ascontiguousarray(x_np[:rows], dtype=np.float64)
    rho = np.zeros(rows)
    xh = np.zeros((rows, d))
    bounds = np.linspace(0, rows, threads + 1).astype(np.int64)
    passes = 0
    t0 = time.perf_counter()
    while True:
        work = [threading.Thread(target=oracle.stage1_range,
                                 args=(variant, d, bits, rot, levels, xd, int(bounds[i]),
                                       int(bounds[i + 1])), kwargs={"rho": rho, "xh": xh})
                for i in range(threads)]
        for w in work:
            w.start()
        for w in work:
            w.join()
        passes += 1
        dt = time.perf_counter() - t0
        if dt >= seconds or passes >= 100:
            break
    return {"value": rows * passes / dt, "unit": "vectors/s", "cores": threads, "threads": threads,
            "single_thread_value": single, "host_cpus": os.cpu_count(), "host_cpus_available": avail,
            "kind": "oracle",
            "sample": f"first {rows} of the {len(x_np)} input rows x {passes} passes, fp64 C oracle "
                      f"(Algorithm 1, indices not stored), rows split over {threads} threads (one GPU's "
                      f"CPU share of {CPU_SHARE} cores; {avail} available, {os.cpu_count()} on the host), "
                      f"{dt:.1f} s; single_thread_value: the first {rows1} rows on one thread"}


APPEND_CASES = (("decode_32x1", 32, 1), ("prefill_8x4096", 8, 4096))
# --case: run one append workload only (a profile then covers one workload)
CASE = None


def _cases(cases):
    return tuple(c for c in cases if CASE is None or c[0].startswith(CASE))


def block8_side(torch, workloads):
    """8-D grouped blocks (one 8x8 orthogonal matrix per 8 coordinates): round
    trip and quantize of the headline rows (1,048,576 unit-norm fp16 vectors,
    d = 128, 3 bits) and of 262,144 fp32 rows at d = 512.  Algorithmic bytes
    per row as for the other variants."""
    import numpy as np

    import paper_2603_28430_amd as iq

    out = {}
    for d, n, tdt, ndt in ((128, 1 << 20, torch.float16, np.float16), (512, 1 << 18, torch.float32, np.float32)):
        esz = 2 if tdt == torch.float16 else 4
        print(f"# block8 d={d}", file=sys.stderr, flush=True)
        x0 = torch.from_numpy(workloads.unit_gaussian_rows(n, d, seed=0, dtype=ndt)).cuda()
        xs = [x0] + [x0.clone() for _ in range(2)]
        ys = [torch.empty_like(x0) for _ in range(3)]
        p = iq.isoq_params_init("8d", d, 3, 1, rot=workloads.rotation_draws("8d", d, 1, seed=1))
        R = p.record_bytes
        recs = [iq.isoq_quantize(p, xs[i]) for i in range(3)]
        res = {}
        for mode in ("roundtrip", "quantize"):
            if mode == "roundtrip":
                fn = lambda i: iq.isoq_roundtrip(p, xs[i % 3], x_hat=ys[i % 3])
                b = n * 2 * d * esz
            else:
                fn = lambda i: iq.isoq_quantize(p, xs[i % 3], idx_packed=recs[i % 3][0], norms=recs[i % 3][1])
                b = n * (d * esz + R + 4)
            ms = time_launches(fn, 50, 5, torch, 0.2)
            res[mode] = {"us": ms * 1e3, "vectors_per_s": n / (ms / 1e3), "GBps": b / ms / 1e6,
                         "frac": b / ms / 1e6 / PEAK_HBM_GBPS}
        p.close()
        out[f"d{d}_{'f16' if esz == 2 else 'f32'}_n{n}_b3"] = res
        del x0, xs, ys, recs
        torch.cuda.empty_cache()
    return out


def kv_append_side(torch, workloads, d=128, cases=APPEND_CASES):
    """isoq_kv_append (quantize K and V into a paged cache, one launch): a
    decode step (32 sequences x 1 token) and a prefill-sized append (8
    sequences x 4,096 tokens), 32 heads, d = 128 (or d), Fast, 3 bits, fp16,
    block size 16, one quaternion set per head; each sequence owns randomly
    placed cache blocks and fills them in order.  Algorithmic bytes per row:
    the fp16 row, the record (48 bytes at d = 128) and the 4-byte norm (plus 8
    bytes of slot per token)."""
    import paper_2603_28430_amd as iq

    H, bs, bits = 32, 16, 3
    res = {}
    for name, n_seq, per_seq in _cases(cases):
        n_tok = n_seq * per_seq
        n_blocks = max(4096, 2 * n_tok // bs)
        print(f"# kv append {name}", file=sys.stderr, flush=True)
        rot = workloads.rotation_draws("fast", d, H, seed=1)
        pk = iq.isoq_params_init("fast", d, bits, H, rot=rot)
        pv = iq.isoq_params_init("fast", d, bits, H, rot=workloads.rotation_draws("fast", d, H, seed=2))
        # per-head AR(1) token streams, laid out token-major [n_tok, H, d]
        k = workloads.kv_stream_torch(1, H, n_tok, d, 2, "cuda")[0].transpose(0, 1).contiguous()
        v = workloads.kv_stream_torch(1, H, n_tok, d, 3, "cuda")[0].transpose(0, 1).contiguous()
        # sequence b, position t (decode: the next position of a 1,000-token history)
        blocks_per_seq = (per_seq + 1000 + bs - 1) // bs + 1
        tables = torch.randperm(n_blocks, device="cuda")[: n_seq * blocks_per_seq].view(n_seq, -1)
        pos = torch.arange(per_seq, device="cuda") + (1000 if per_seq == 1 else 0)
        slots = (tables[:, pos // bs] * bs + pos % bs).reshape(-1).to(torch.int64)
        R = pk.record_bytes
        caches = [torch.empty((n_blocks, H, bs, R), dtype=torch.uint8, device="cuda") for _ in range(2)]
        rhos = [torch.empty((n_blocks, H, bs), dtype=torch.float32, device="cuda") for _ in range(2)]
        fn = lambda i: iq.isoq_kv_append(pk, k, slots, caches[0], rhos[0], pv, v, caches[1], rhos[1])
        steps = 200 if n_tok < 1000 else 50
        ms = time_launches(fn, steps, 10, torch, 0.2)
        b = 2 * n_tok * (H * (d * 2 + R + 4) + 8)
        res[name] = _append_entry(n_tok, H, ms, b, fn, torch)
        pk.close()
        pv.close()
        del k, v, caches, rhos
    return res


def _append_entry(n_tok, H, ms, b, fn, torch):
    """JSON entry of an append measurement.  A decode step (a few tokens) is
    shorter than the host's per-call cost (~10 us through ctypes), so its
    back-to-back event time measures the host: there the device time comes
    from the same launches replayed from a HIP graph, and GBps / frac use it
    (frac is null if graph capture is unavailable)."""
    e = {"tokens": n_tok, "heads": H, "us_per_call": ms * 1e3}
    if n_tok >= 1000:
        e.update(GBps=b / ms / 1e6, frac=b / ms / 1e6 / PEAK_HBM_GBPS)
        return e
    us = graph_launch_us(fn, 50, torch)
    e["us_per_launch_graph"] = us
    e["GBps"] = None if us is None else b / us / 1e3
    e["frac"] = None if us is None else b / us / 1e3 / PEAK_HBM_GBPS
    return e


def kv_cache_side(torch, workloads):
    """The K/V cache stream [8, 32, 32768, 128] fp16, Fast 3-bit quantize only
    (packed records and norms out), one quaternion set per head
    (rows_per_set = 32,768): one step is the K tensor then the V tensor.
    Algorithmic bytes per row: the fp16 row, the 48-byte record, the 4-byte
    norm."""
    import paper_2603_28430_amd as iq

    B, H, T, d, bits = 8, 32, 32768, 128, 3
    print("# config kv cache", file=sys.stderr, flush=True)
    kv = [workloads.kv_stream_torch(B, H, T, d, seed, "cuda").view(B * H * T, d) for seed in (2, 3)]
    p = iq.isoq_params_init("fast", d, bits, H, rot=workloads.rotation_draws("fast", d, H, seed=1))
    n = B * H * T
    recs = [torch.empty((n, p.record_bytes), dtype=torch.uint8, device="cuda") for _ in range(2)]
    norms = [torch.empty((n,), dtype=torch.float32, device="cuda") for _ in range(2)]
    fn = lambda i: iq.isoq_quantize(p, kv[i % 2], T, idx_packed=recs[i % 2], norms=norms[i % 2])
    ms = time_launches(fn, 40, 4, torch, 0.2)
    b = n * (d * 2 + p.record_bytes + 4)
    step = 2 * ms  # K and V: two launches of the same size
    p.close()
    del kv, recs, norms
    torch.cuda.empty_cache()
    return {"shape": [B, H, T, d], "tensors": 2, "ms_per_step": step, "rows_per_s": 2 * n / (step / 1e3),
            "GBps": 2 * b / step / 1e6, "frac": 2 * b / step / 1e6 / PEAK_HBM_GBPS}


def head_widths_side(torch, workloads):
    """The decoding calls at the attention head widths 80, 96 and 192
    (packed-row append, logits with 2-, 4- and 8-byte record loads): the
    prefill-sized append and the logits of kv_append_side and kv_scores_side
    at those widths."""
    return {f"d{d}": {"kv_append": kv_append_side(torch, workloads, d, (("prefill_8x4096", 8, 4096),)),
                      "kv_scores": kv_scores_side(torch, workloads, d)} for d in (80, 96, 192)}


def kv_append_qjl_side(torch, workloads):
    """isoq_kv_append_qjl (key rows with the stage-2 sketch into a paged
    cache, one launch): the decode step and the prefill-sized append of
    kv_append_side, keys only, m = 128.  Algorithmic bytes per (token, head)
    row: the fp16 row, the 48-byte record, the 4-byte norm, 16 sign bytes and
    the 4-byte gamma (plus 8 bytes of slot per token)."""
    import paper_2603_28430_amd as iq

    H, d, bs, bits, m = 32, 128, 16, 3, 128
    res = {}
    for name, n_seq, per_seq in _cases(APPEND_CASES):
        n_tok = n_seq * per_seq
        n_blocks = max(4096, 2 * n_tok // bs)
        print(f"# kv append qjl {name}", file=sys.stderr, flush=True)
        pk = iq.isoq_params_init("fast", d, bits, H, rot=workloads.rotation_draws("fast", d, H, seed=1))
        sk = iq.isoq_sketch_init(pk, m)
        k = workloads.kv_stream_torch(1, H, n_tok, d, 2, "cuda")[0].transpose(0, 1).contiguous()
        blocks_per_seq = (per_seq + 1000 + bs - 1) // bs + 1
        tables = torch.randperm(n_blocks, device="cuda")[: n_seq * blocks_per_seq].view(n_seq, -1)
        pos = torch.arange(per_seq, device="cuda") + (1000 if per_seq == 1 else 0)
        slots = (tables[:, pos // bs] * bs + pos % bs).reshape(-1).to(torch.int64)
        R = pk.record_bytes
        rec = torch.empty((n_blocks, H, bs, R), dtype=torch.uint8, device="cuda")
        sg = torch.empty((n_blocks, H, bs, m // 8), dtype=torch.uint8, device="cuda")
        rho = torch.empty((n_blocks, H, bs), dtype=torch.float32, device="cuda")
        gam = torch.empty((n_blocks, H, bs), dtype=torch.float32, device="cuda")
        fn = lambda i: iq.isoq_kv_append_qjl(pk, sk, k, slots, rec, rho, sg, gam)
        steps = 200 if n_tok < 1000 else 50
        ms = time_launches(fn, steps, 10, torch, 0.2)
        b = n_tok * (H * (d * 2 + R + 4 + m // 8 + 4) + 8)
        res[name] = _append_entry(n_tok, H, ms, b, fn, torch)
        sk.close()
        pk.close()
        del k, rec, sg, rho, gam
    return res


def kv_scores_side(torch, workloads, d=128):
    """isoq_kv_scores: attention logits of one decoding query per head against
    a paged cache of quantized keys, 8 sequences x 32,768 positions x 32 heads,
    d = 128 (or d), Fast, 3 bits, block size 16, blocks placed at random.  The
    cache content is random index bytes and norms (the cost does not depend on
    it).  Algorithmic bytes per key: its record (48 bytes at d = 128), 4-byte
    norm and 4-byte logit."""
    import paper_2603_28430_amd as iq

    B, H, T, bs, bits = 8, 32, 32768, 16, 3
    print("# kv scores", file=sys.stderr, flush=True)
    p = iq.isoq_params_init("fast", d, bits, H, rot=workloads.rotation_draws("fast", d, H, seed=1))
    nb = B * T // bs
    gen = torch.Generator(device="cuda")
    gen.manual_seed(4)
    rec = torch.randint(0, 256, (nb, H, bs, p.record_bytes), dtype=torch.uint8, device="cuda", generator=gen)
    rho = torch.rand((nb, H, bs), device="cuda", generator=gen) + 0.5
    table = torch.randperm(nb, device="cuda", generator=gen).to(torch.int32).view(B, T // bs)
    lens = torch.full((B,), T, dtype=torch.int32, device="cuda")
    q = torch.randn((B, H, d), device="cuda", generator=gen).to(torch.float16)
    out = torch.empty((B, H, T), dtype=torch.float32, device="cuda")
    fn = lambda i: iq.isoq_kv_scores(p, q, rec, rho, table, lens, 0.0884, max_len=T, scores=out)
    ms = time_launches(fn, 50, 5, torch, 0.2)
    keys = B * H * T
    b = keys * (p.record_bytes + 4 + 4)
    p.close()
    return {"shape": [B, H, T, d], "us_per_call": ms * 1e3, "keys_per_s": keys / (ms / 1e3),
            "GBps": b / ms / 1e6, "frac": b / ms / 1e6 / PEAK_HBM_GBPS}


def kv_scores_qjl_side(torch, workloads):
    """isoq_kv_scores_qjl: the logits of kv_scores_side with the stage-2
    correction, m = 128 and 64 sign bits per key (same cache shape, random
    records, norms, signs and gammas).  Algorithmic bytes per key: record,
    norm, m/8 sign bytes, gamma and the logit."""
    import paper_2603_28430_amd as iq

    B, H, T, d, bs, bits = 8, 32, 32768, 128, 16, 3
    p = iq.isoq_params_init("fast", d, bits, H, rot=workloads.rotation_draws("fast", d, H, seed=1))
    nb = B * T // bs
    gen = torch.Generator(device="cuda")
    gen.manual_seed(4)
    rec = torch.randint(0, 256, (nb, H, bs, p.record_bytes), dtype=torch.uint8, device="cuda", generator=gen)
    rho = torch.rand((nb, H, bs), device="cuda", generator=gen) + 0.5
    gam = torch.rand((nb, H, bs), device="cuda", generator=gen) * 0.2
    table = torch.randperm(nb, device="cuda", generator=gen).to(torch.int32).view(B, T // bs)
    lens = torch.full((B,), T, dtype=torch.int32, device="cuda")
    q = torch.randn((B, H, d), device="cuda", generator=gen).to(torch.float16)
    out = torch.empty((B, H, T), dtype=torch.float32, device="cuda")
    res = {}
    for m in (128, 64):
        print(f"# kv scores qjl m={m}", file=sys.stderr, flush=True)
        sk = iq.isoq_sketch_init(p, m)
        sg = torch.randint(0, 256, (nb, H, bs, m // 8), dtype=torch.uint8, device="cuda", generator=gen)
        fn = lambda i: iq.isoq_kv_scores_qjl(p, sk, q, rec, rho, sg, gam, table, lens, 0.0884, max_len=T,
                                             scores=out)
        ms = time_launches(fn, 50, 5, torch, 0.2)
        keys = B * H * T
        b = keys * (p.record_bytes + 4 + m // 8 + 4 + 4)
        res[f"m{m}"] = {"shape": [B, H, T, d], "us_per_call": ms * 1e3, "keys_per_s": keys / (ms / 1e3),
                        "GBps": b / ms / 1e6, "frac": b / ms / 1e6 / PEAK_HBM_GBPS}
        sk.close()
        del sg
    p.close()
    return res


def qjl_side(torch, workloads):
    """isoq_quantize_qjl: stage-1 quantize plus the stage-2 residual sketch,
    1,048,576 unit-norm fp16 rows, d = 128, 3 bits, m = 128 and 64 sign bits.
    Algorithmic bytes per row: the fp16 row, the 48-byte record, the 4-byte
    norm, m/8 sign bytes and the 4-byte gamma; the projection adds 2 m d flops
    per row on MFMA."""
    import numpy as np

    import paper_2603_28430_amd as iq

    n, d, bits = 1 << 20, 128, 3
    print("# qjl quantize", file=sys.stderr, flush=True)
    x0 = torch.from_numpy(workloads.unit_gaussian_rows(n, d, seed=0, dtype=np.float16)).cuda()
    xs = [x0] + [x0.clone() for _ in range(3)]
    out = {}
    for variant in ("full", "fast"):
        p = iq.isoq_params_init(variant, d, bits, 1, rot=workloads.rotation_draws(variant, d, 1, seed=1))
        for m in (128, 64):
            sk = iq.isoq_sketch_init(p, m)
            bufs = [iq.isoq_quantize_qjl(p, sk, xs[i]) for i in range(4)]
            fn = lambda i: iq.isoq_quantize_qjl(p, sk, xs[i % 4], idx_packed=bufs[i % 4][0], norms=bufs[i % 4][1],
                                                signs=bufs[i % 4][2], gamma=bufs[i % 4][3])
            ms = time_launches(fn, 100, 10, torch, 0.2)
            b = n * (d * 2 + d * bits // 8 + 4 + m // 8 + 4)
            out[f"{variant}_m{m}"] = {"us": ms * 1e3, "vectors_per_s": n / (ms / 1e3), "GBps": b / ms / 1e6,
                                      "frac": b / ms / 1e6 / PEAK_HBM_GBPS,
                                      "mfma_TFLOPs": 2.0 * m * d * n / ms / 1e9}
            sk.close()
        p.close()
    return out


def qjl_widths_side(torch, workloads):
    """The stage-2 sketch at the other widths: isoq_quantize_qjl on fp16
    unit-norm rows, Fast, 3 bits, m = 128 at the head widths 80, 96, 160 and
    192 (1,048,576 rows, packed-row kernels) and m = 64 at d = 512 (262,144
    rows); and the prefill-sized isoq_kv_append_qjl (8 x 4096 tokens x 32
    heads, m = 128) at 96 and 192.  Algorithmic bytes as in qjl_side and
    kv_append_qjl_side."""
    import numpy as np

    import paper_2603_28430_amd as iq

    bits, out = 3, {}
    for d, m, n in ((80, 128, 1 << 20), (96, 128, 1 << 20), (160, 128, 1 << 20), (192, 128, 1 << 20),
                    (512, 64, 1 << 18)):
        print(f"# qjl quantize d={d}", file=sys.stderr, flush=True)
        x0 = torch.from_numpy(workloads.unit_gaussian_rows(n, d, seed=0, dtype=np.float16)).cuda()
        xs = [x0] + [x0.clone() for _ in range(3)]
        p = iq.isoq_params_init("fast", d, bits, 1, rot=workloads.rotation_draws("fast", d, 1, seed=1))
        sk = iq.isoq_sketch_init(p, m)
        bufs = [iq.isoq_quantize_qjl(p, sk, xs[i]) for i in range(4)]
        fn = lambda i: iq.isoq_quantize_qjl(p, sk, xs[i % 4], idx_packed=bufs[i % 4][0], norms=bufs[i % 4][1],
                                            signs=bufs[i % 4][2], gamma=bufs[i % 4][3])
        ms = time_launches(fn, 50, 5, torch, 0.2)
        b = n * (d * 2 + p.record_bytes + 4 + m // 8 + 4)
        out[f"quantize_d{d}_m{m}"] = {"us": ms * 1e3, "GBps": b / ms / 1e6, "frac": b / ms / 1e6 / PEAK_HBM_GBPS}
        sk.close()
        p.close()
        del x0, xs, bufs
    H, bs, m, n_tok = 32, 16, 128, 8 * 4096
    for d in (96, 192):
        print(f"# kv append qjl d={d}", file=sys.stderr, flush=True)
        pk = iq.isoq_params_init("fast", d, bits, H, rot=workloads.rotation_draws("fast", d, H, seed=1))
        sk = iq.isoq_sketch_init(pk, m)
        k = workloads.kv_stream_torch(1, H, n_tok, d, 2, "cuda")[0].transpose(0, 1).contiguous()
        n_blocks = 2 * n_tok // bs
        slots = torch.randperm(n_blocks * bs, device="cuda")[:n_tok].to(torch.int64)
        R = pk.record_bytes
        rec = torch.empty((n_blocks, H, bs, R), dtype=torch.uint8, device="cuda")
        sg = torch.empty((n_blocks, H, bs, m // 8), dtype=torch.uint8, device="cuda")
        rho = torch.empty((n_blocks, H, bs), dtype=torch.float32, device="cuda")
        gam = torch.empty((n_blocks, H, bs), dtype=torch.float32, device="cuda")
        fn = lambda i: iq.isoq_kv_append_qjl(pk, sk, k, slots, rec, rho, sg, gam)
        ms = time_launches(fn, 50, 5, torch, 0.2)
        b = n_tok * (H * (d * 2 + R + 4 + m // 8 + 4) + 8)
        out[f"append_prefill_d{d}_m{m}"] = {"us": ms * 1e3, "GBps": b / ms / 1e6,
                                            "frac": b / ms / 1e6 / PEAK_HBM_GBPS}
        sk.close()
        pk.close()
        del k, rec, sg, rho, gam
    return out


def widths_side(torch, workloads):
    """Widths outside {128, 256, 512} (Sec. 5.1 zero padding where needed):
    round trip and quantize of 1,048,576 unit-norm rows (262,144 for d = 1000),
    Full and Fast, 3 bits; d = 64 runs the tuned kernels, fp16 d = 80, 96, 160
    and 192 the packed-row kernels, d = 90 and the fp32 rows the generic ones.  Algorithmic
    bytes per row as for the
    tuned widths: 2 d s for the round trip, d s + record + 4 for quantize (s =
    bytes per element, record = ceil(pw * 3 / 8))."""
    import numpy as np

    import paper_2603_28430_amd as iq

    out = {}
    for d, dtype, n in ((64, "f16", 1 << 20), (80, "f16", 1 << 20), (96, "f16", 1 << 20), (90, "f16", 1 << 20),
                        (160, "f16", 1 << 20), (192, "f16", 1 << 20), (96, "f32", 1 << 20), (1000, "f32", 1 << 18)):
        tdt, ndt, esz = (torch.float16, np.float16, 2) if dtype == "f16" else (torch.float32, np.float32, 4)
        name = f"d{d}_{dtype}_n{n}"
        print(f"# widths {name}", file=sys.stderr, flush=True)
        x0 = torch.from_numpy(workloads.unit_gaussian_rows(n, d, seed=0, dtype=ndt)).cuda()
        xs = [x0] + [x0.clone() for _ in range(2)]
        ys = [torch.empty_like(x0) for _ in range(3)]
        res = {}
        for variant in ("full", "fast"):
            p = iq.isoq_params_init(variant, d, 3, 1, rot=workloads.rotation_draws(variant, d, 1, seed=1))
            R = p.record_bytes
            recs = [iq.isoq_quantize(p, xs[i]) for i in range(3)]
            for mode in ("roundtrip", "quantize"):
                if mode == "roundtrip":
                    fn = lambda i: iq.isoq_roundtrip(p, xs[i % 3], x_hat=ys[i % 3])
                    b = n * 2 * d * esz
                else:
                    fn = lambda i: iq.isoq_quantize(p, xs[i % 3], idx_packed=recs[i % 3][0], norms=recs[i % 3][1])
                    b = n * (d * esz + R + 4)
                ms = time_launches(fn, 50, 5, torch, 0.2)
                res[f"{variant}_{mode}"] = {"us": ms * 1e3, "vectors_per_s": n / (ms / 1e3), "GBps": b / ms / 1e6,
                                            "frac": b / ms / 1e6 / PEAK_HBM_GBPS}
            p.close()
        out[name] = res
        del x0, xs, ys
        torch.cuda.empty_cache()
    return out


def other_configs(measure, entry, torch, np, workloads):
    """Side measurements of the other workloads (their parity is tested in
    tests/test_gpu_full_sizes.py): d = 256 fp16 and d = 512 fp32 round trips
    and quantize, Full and Fast, 2-4 bits; the K/V cache stream
    [8, 32, 32768, 128] fp16, Fast 3-bit quantize, one quaternion set per head
    (one step = K then V)."""
    out = {}
    for name, d_, n_, tdt, ndt in (("d256_f16_n1048576", 256, 1 << 20, torch.float16, np.float16),
                                   ("d512_f32_n262144", 512, 1 << 18, torch.float32, np.float32)):
        print(f"# config {name}", file=sys.stderr, flush=True)
        x0 = torch.from_numpy(workloads.unit_gaussian_rows(n_, d_, seed=0, dtype=ndt)).cuda()
        ins = [x0] + [x0.clone() for _ in range(2)]
        outs_ = [torch.empty_like(x0) for _ in range(3)]
        res = {}
        for variant in ("full", "fast"):
            for b_ in (2, 3, 4):
                res[f"{variant}_b{b_}"] = entry(*measure(variant, b_, "roundtrip", 50, 5, 0.2, ins, outs_, d_))
                res[f"{variant}_b{b_}_quantize"] = entry(*measure(variant, b_, "quantize", 50, 5, 0.2, ins,
                                                                  outs_, d_))
        out[name] = res
        del x0, ins, outs_
        torch.cuda.empty_cache()
    out["kv_append"] = kv_append_side(torch, workloads)
    out["kv_append_qjl"] = kv_append_qjl_side(torch, workloads)
    out["kv_scores"] = kv_scores_side(torch, workloads)
    out["qjl_quantize"] = qjl_side(torch, workloads)
    out["qjl_widths"] = qjl_widths_side(torch, workloads)
    out["kv_scores_qjl"] = kv_scores_qjl_side(torch, workloads)
    out["widths"] = widths_side(torch, workloads)
    out["head_widths"] = head_widths_side(torch, workloads)
    out["block8"] = block8_side(torch, workloads)
    out["kv_cache_fast_b3_quantize"] = kv_cache_side(torch, workloads)
    return out


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--variant", default="full", choices=["full", "fast", "2d"])
    ap.add_argument("--bits", type=int, default=3)
    ap.add_argument("--d", type=int, default=128)
    ap.add_argument("--dtype", default="f16", choices=["f16", "f32"])
    ap.add_argument("--n", type=int, default=1 << 20)
    ap.add_argument("--mode", default="roundtrip", choices=["roundtrip", "quantize", "dequantize"])
    ap.add_argument("--buffer-sets", type=int, default=4)
    ap.add_argument("--warm-seconds", type=float, default=1.0)
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-extras", action="store_true")
    ap.add_argument("--no-configs", action="store_true",
                    help="skip the side measurements of the d=256, d=512 and KV-cache workloads")
    ap.add_argument("--side", choices=["kv-append", "kv-append-qjl", "kv-scores", "kv-scores-qjl", "qjl",
                                       "qjl-widths", "widths", "head-widths", "kv-cache", "block8"],
                    help="run only this side measurement and print its JSON")
    ap.add_argument("--case", choices=["decode", "prefill"],
                    help="with --side kv-append or kv-append-qjl: that workload only")
    ap.add_argument("--copy-only", action="store_true",
                    help="only time a plain device copy of the input size (counter calibration)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU; --gpus {args.gpus} is not supported (rows are "
              "independent, so a multi-GPU run is N copies of this one).", file=sys.stderr)
        return 2

    import numpy as np
    import torch

    import paper_2603_28430_amd as iq
    import workloads

    torch.cuda.set_device(0)
    if args.side:
        global CASE
        CASE = args.case
        fn = {"kv-append": kv_append_side, "kv-append-qjl": kv_append_qjl_side, "kv-scores": kv_scores_side,
              "kv-scores-qjl": kv_scores_qjl_side, "qjl": qjl_side, "widths": widths_side,
              "head-widths": head_widths_side, "kv-cache": kv_cache_side, "block8": block8_side,
              "qjl-widths": qjl_widths_side}[args.side]
        print(json.dumps({"side": args.side, **fn(torch, workloads)}), flush=True)
        return 0
    tdt, ndt, esz = {"f16": (torch.float16, np.float16, 2), "f32": (torch.float32, np.float32, 4)}[args.dtype]
    n, d, bits, S = args.n, args.d, args.bits, max(1, args.buffer_sets)
    print(f"# inputs: {n} x {d} {args.dtype}", file=sys.stderr, flush=True)
    x_np = workloads.unit_gaussian_rows(n, d, seed=0, dtype=ndt)
    x0 = torch.from_numpy(x_np).cuda()
    xs = [x0] + [x0.clone() for _ in range(S - 1)]
    outs = [torch.empty_like(x0) for _ in range(S)]

    if args.copy_only:
        ms = time_launches(lambda i: outs[i % S].copy_(xs[i % S]), args.steps, args.warmup, torch,
                           args.warm_seconds)
        b = 2 * x0.numel() * esz
        print(json.dumps({"copy_bytes_per_launch": b, "ms_per_launch": ms, "GBps": b / ms / 1e6}))
        return 0

    def setup(variant, bits_, d_=d, n_sets=1):
        rot = workloads.rotation_draws(variant, d_, n_sets, seed=1)
        return iq.isoq_params_init(variant, d_, bits_, n_sets, rot=rot), rot

    def measure(variant, bits_, mode, steps, warmup, warm_seconds=0.0, ins=None, outs_=None,
                d_=d, n_sets=1, rows_per_set=1):
        """ms per launch of `mode` over the buffer sets `ins` (rows) / `outs_`."""
        ins = xs if ins is None else ins
        outs_ = outs if outs_ is None else outs_
        S_ = len(ins)
        n_ = ins[0].numel() // d_
        p, _ = setup(variant, bits_, d_, n_sets)
        if mode == "roundtrip":
            fn = lambda i: iq.isoq_roundtrip(p, ins[i % S_], rows_per_set, x_hat=outs_[i % S_])
        else:
            recs = [torch.empty((n_, p.record_bytes), dtype=torch.uint8, device="cuda") for _ in range(S_)]
            norms = [torch.empty((n_,), dtype=torch.float32, device="cuda") for _ in range(S_)]
            for i in range(S_):
                iq.isoq_quantize(p, ins[i], rows_per_set, idx_packed=recs[i], norms=norms[i])
            if mode == "quantize":
                fn = lambda i: iq.isoq_quantize(p, ins[i % S_], rows_per_set, idx_packed=recs[i % S_],
                                                norms=norms[i % S_])
            else:
                fn = lambda i: iq.isoq_dequantize(p, recs[i % S_], norms[i % S_], rows_per_set=rows_per_set,
                                                  x_hat=outs_[i % S_])
        ms = time_launches(fn, steps, warmup, torch, warm_seconds)
        b = algorithmic_bytes(mode, n_, d_, bits_, ins[0].element_size())
        p.close()
        return ms, b, n_

    def entry(ms, b, n_):
        return {"ms": ms, "vectors_per_s": n_ / (ms / 1e3), "GBps": b / ms / 1e6,
                "frac": b / ms / 1e6 / PEAK_HBM_GBPS}

    # ---- the timed headline: K steps of the fused path ----
    print(f"# timing {args.mode} {args.variant} b={bits}", file=sys.stderr, flush=True)
    ms, abytes, _ = measure(args.variant, bits, args.mode, args.steps, args.warmup, args.warm_seconds)
    gbps = abytes / ms / 1e6
    tag = f"{args.mode}_{args.variant}_d{d}_b{bits}_{args.dtype}_n{n}"
    result = {
        "metric": METRIC,
        "value": n / (ms / 1e3),
        "unit": "vectors/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic: i.i.d. N(0,1) rows scaled to unit norm (seed 0), raw rotation draws "
                "from Philox4x32-10 (seed 1), Lloyd-Max codebook for N(0,1/d), 200 iterations",
        "config": {"workload": f"IsoQuant-{args.variant} stage-1 {args.mode}, {n} vectors x d={d}, "
                               f"{bits}-bit, {args.dtype} rows (fp32 arithmetic)",
                   "variant": args.variant, "d": d, "bits": bits, "io_dtype": args.dtype, "n": n,
                   "mode": args.mode, "buffer_sets": S},
        "effective_GBps": gbps,
        "pct_of_peak_hbm": 100.0 * gbps / PEAK_HBM_GBPS,
        "roofline": {"bound": "hbm", "achieved": gbps, "peak": PEAK_HBM_GBPS, "unit": "GB/s",
                     "frac": gbps / PEAK_HBM_GBPS, "traffic": measured_traffic(tag),
                     "algorithmic_bytes_per_launch": abytes,
                     "kernel": kernel_name(args.variant, d, bits, args.dtype, args.mode),
                     "kernel_source_sha256": kernel_source_hash()},
    }

    if not args.no_extras:
        extra = {}
        print("# side measurements", file=sys.stderr, flush=True)
        cms = time_launches(lambda i: outs[i % S].copy_(xs[i % S]), 50, 5, torch, 0.2)
        extra["device_copy_same_size"] = {"GBps": 2 * x0.numel() * esz / cms / 1e6, "ms": cms}
        paths = {}
        for mode in ("quantize", "dequantize"):
            paths[mode] = entry(*measure(args.variant, bits, mode, 100, 10, 0.2))
        extra["paths"] = paths
        sweep = {}
        for variant in ("full", "fast", "2d"):
            for b_ in (2, 3, 4):
                sweep[f"{variant}_b{b_}"] = entry(*measure(variant, b_, "roundtrip", 100, 10, 0.2))
                if d == 128 and args.dtype == "f16" and n == 1 << 20:
                    sweep[f"{variant}_b{b_}_quantize"] = entry(*measure(variant, b_, "quantize", 100, 10, 0.2))
        extra["roundtrip_sweep"] = sweep
        del xs[1:], outs[1:]
        if not args.no_configs:
            extra["configs"] = other_configs(measure, entry, torch, np, workloads)
        result["extra"] = extra

    if not args.no_cpu_baseline:
        import oracle

        print("# cpu baseline (oracle)", file=sys.stderr, flush=True)
        _, rot = setup(args.variant, bits)
        levels = oracle.codebook(bits, d)
        result["cpu_baseline"] = cpu_baseline(args.variant, d, bits, x_np, rot, levels,
                                              args.cpu_seconds)
    print(json.dumps(result), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
