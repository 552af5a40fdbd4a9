"""Decode-step throughput of the shared KV pool on one MI355X.

A step is one pass of the hot path over one batch: append one new token per
request (page allocation + scatter through the page table), then batched
decode attention over every request's whole context (split planning,
attention kernel, split merge). Steps cycle over several layers, each with
its own copy of the batch's KV in its own pool, so that consecutive steps
never find their KV in the 256 MiB Infinity Cache, as when a model's layers
are decoded one after another.

The headline line measures the DeepSeek-V3-shaped batch (8 requests of 128K
tokens at 128 query heads), the largest single-GPU workload; the same run
also measures the V2-Lite-shaped, mixed-model and 512K-burst batches and
reports each under "per_config". Requests are loaded one token short of
their configured context (and short by the warmup's appends), so the first
timed step of every layer attends over exactly the configured lengths.

Prints one JSON line. value = algorithmic bytes moved per second over the
timed steps (KV read once, queries, outputs, lse, page-table entries, and
the appended rows read and written), in GB/s.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--config 3] [--also 2,4,5]
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0  # MI355X HBM3E
MFMA_BF16_PEAK_TFLOPS = 2500.0  # MI355X dense bf16 matrix-core peak
MAX_SETTLE_CALLS = 4000
PROFILE_NAMES = {2: "decode_v2lite_mla16", 3: "decode_v3_mla128", 4: "decode_mixed", 5: "decode_burst_mla128"}
KERNEL_NAMES = {2: "cp::decode_kernel (narrow matrix MLA-16)", 3: "cp::decode_mla_kernel (MLA-128)",
                4: "cp::decode_kernel (narrow matrix MLA-16 / MQA-32 / GQA-32:4)",
                5: "cp::decode_mla_kernel (MLA-128)"}
WORKLOAD_NAMES = {
    1: "tiny MLA-16 decode: 4 requests {128,256,384,512} tokens, 64-page pool",
    2: "DeepSeek-V2-Lite-shaped MLA-16 decode: 32 requests, log-uniform 1K-32K tokens, 2 GiB pool",
    3: "DeepSeek-V3-shaped MLA-128 decode: 8 requests x 128K tokens",
    4: "mixed MLA-16/MQA-32/GQA-32x4 decode: 48 requests, Zipf(1.2) models, log-uniform 512-64K tokens, 8 GiB pool",
    5: "MLA-128 burst: 1 request at 512K tokens in a 2 GiB pool 90% full",
}


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=20, help="untimed warmup steps (each appends a token)")
    ap.add_argument("--settle-seconds", type=float, default=0.3,
                    help="GPU time of decode-only calls (no appends) run before the warmup steps, so clocks and "
                         "power settle")
    ap.add_argument("--config", type=int, default=3, choices=[1, 2, 3, 4, 5])
    ap.add_argument("--also", default="auto",
                    help="further workloads measured in the same run, reported under per_config: a comma list, "
                         "'none', or 'auto' (the other workloads of 2-5)")
    ap.add_argument("--layers", type=int, default=0, help="KV copies cycled by the steps (0: enough to exceed 1 GiB)")
    ap.add_argument("--ctx-scale", type=float, default=1.0,
                    help="scale every context length of the workload (1: the configured sizes)")
    ap.add_argument("--path", type=int, default=0, help="0 auto, 1 vector, 2 matrix cores")
    ap.add_argument("--splits", type=int, default=0, help="forced KV ranges per request (queue/grid schedules)")
    ap.add_argument("--schedule", type=int, default=0, help="0 balanced, 1 work queue, 2 one workgroup per unit")
    ap.add_argument("--unfused", action="store_true",
                    help="step as cp_kv_append + cp_attn_decode_ex instead of cp_attn_decode_step")
    ap.add_argument("--backing", type=int, default=0, choices=[0, 1],
                    help="pool memory: 0 one device buffer, 1 virtual ranges with chunks mapped on demand")
    ap.add_argument("--planes", action="store_true",
                    help="one pool whose models have one KV plane per layer, the steps moving each request's "
                         "layer cursor, instead of one pool per layer")
    ap.add_argument("--layer-launch", type=int, default=0, metavar="L",
                    help="also time steps that take every request through L KV layers in one "
                         "cp_attn_decode_layers call, against L per-layer cp_attn_decode_step calls on the same pool "
                         "(reported under layer_launch)")
    ap.add_argument("--device-pages", action="store_true",
                    help="pools with device free-page stacks: the steps pop new pages inside the launch")
    ap.add_argument("--no-inflight", action="store_true",
                    help="skip the two-batches-in-flight record (two pools stepping on two streams)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=12.0, help="target CPU time of the oracle sample")
    ap.add_argument("--copy-mib", type=int, default=0,
                    help="before timing, run one device copy of this many MiB (reference for HBM byte counters)")
    return ap.parse_args()


def kernel_source_hash() -> str:
    """Hash of the sources that decide what a decode launch does: the device
    code, the host code that plans and launches it, and the page allocator
    (placement). The pool planner and other host-only sources are left out."""
    import glob
    import hashlib

    csrc = os.path.join(ROOT, "paper_2606_24506_amd", "csrc")
    files = glob.glob(os.path.join(csrc, "*.hip")) + glob.glob(os.path.join(csrc, "*.h"))
    files += [os.path.join(csrc, f) for f in ("api.cpp", "pool.cpp", "pool.hpp")]
    h = hashlib.sha256()
    for fn in sorted(files):
        h.update(os.path.basename(fn).encode())
        h.update(open(fn, "rb").read())
    return h.hexdigest()


def measured_traffic(cfg: int):
    """(HBM bytes, algorithmic bytes) of one decode launch from the committed
    rocprofv3 counter summary of this workload (scaled FETCH_SIZE +
    WRITE_SIZE, and the algorithmic bytes of the counted launches), or
    (None, None) when there is none or the kernel sources changed since."""
    path = os.path.join(ROOT, "profiles", PROFILE_NAMES.get(cfg, "") + ".json")
    if not os.path.exists(path):
        return None, None
    try:
        d = json.load(open(path))
        if d.get("kernel_source_sha256") != kernel_source_hash() or d.get("workload_config") != cfg:
            return None, None
        k = d["decode_kernel"]
        return float(k["read_bytes"] + k["write_bytes"]), k.get("algorithmic_bytes_per_launch")
    except (OSError, ValueError, KeyError):
        return None, None


def algorithmic_bytes_decode(wl, ctx):
    from workloads import algorithmic_bytes

    return algorithmic_bytes([wl.model(r) for r in range(len(ctx))], ctx)


def algorithmic_flops_decode(wl, ctx):
    """Multiply-adds of the attention itself (QK^T and PV, two flops each)."""
    return sum(2 * c * wl.model(r).n_q_heads * (wl.model(r).d_k + wl.model(r).d_v) for r, c in enumerate(ctx))


def cpu_baseline(wl, budget_s: float):
    """The fp64 oracle, as it stands, on a bounded sample of the same batch:
    whole requests in batch order until about budget_s seconds of CPU work."""
    import oracle

    try:
        from threadpoolctl import threadpool_info

        threads = max([d.get("num_threads", 1) for d in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        threads = len(os.sched_getaffinity(0))
    # whole requests in batch order, cycling over the batch until the budget
    # is spent; rows are drawn outside the timed calls and kept (up to 2 GiB)
    # so that later cycles do not draw them again
    done, t_total = [], 0.0
    rows_cache, cached = {}, 0
    while t_total < budget_s:
        r = len(done) % len(wl.requests)
        rows = rows_cache.get(r)
        if rows is None:
            rows = wl.rows_bits(r)
            if cached + rows.nbytes <= (2 << 30):
                rows_cache[r] = rows
                cached += rows.nbytes
        t0 = time.perf_counter()
        oracle.decode(rows, wl.q_bits[r], wl.model(r))
        t_total += time.perf_counter() - t0
        done.append(r)
    from workloads import algorithmic_bytes

    nbytes = algorithmic_bytes([wl.model(r) for r in done], [wl.requests[r].ctx_len for r in done])
    cpu = "unknown"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                cpu = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return {
        "value": nbytes / t_total / 1e9,
        "unit": "GB/s",
        "cores": int(threads),
        "kind": "oracle",
        "sample": f"fp64 NumPy oracle, {len(done)} whole-request calls cycling over the {len(wl.requests)} requests "
                  f"of the same batch in order, {t_total:.1f} s of oracle time; host CPU: {cpu}",
        "req_tokens_per_s": len(done) / t_total,
    }


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def measure(cfg: int, args) -> dict:
    """Loads workload cfg, settles the clocks, runs the warmup steps, then
    the timed throughput pass and the kernel-timing pass; returns the
    record of this workload."""
    import torch

    from workloads import make_workload
    from workloads.harness import load, to_device_u16

    wl = make_workload(cfg, scale_ctx=args.ctx_scale)
    if args.ctx_scale != 1.0 and wl.filler_pages:
        wl.filler_pages = int(wl.filler_pages * args.ctx_scale)
    B = len(wl.requests)
    kv_bytes = sum(rq.ctx_len * wl.model(r).kappa for r, rq in enumerate(wl.requests))
    layers = args.layers or max(1, math.ceil((1 << 30) / kv_bytes))
    n_warm = args.warmup
    # appends each layer sees before its first timed step
    pre = [len(range(li, n_warm, layers)) for li in range(layers)]
    grow = -(-(n_warm + 2 * args.steps) // layers) + 2
    log(f"cfg{cfg}: {B} requests, {kv_bytes / 1e6:.1f} MB KV per layer, {layers} layers")

    rows_full = {r: wl.rows_bits(r) for r in range(B)}
    inter = 512 if cfg == 4 else (4096 if cfg == 5 else 0)
    if args.planes:
        if wl.filler_pages:
            sys.exit("--planes: the filler requests of this pool leave no room for more than one KV plane")
        # one pool, L planes: step i serves layer i % L of every request
        short = n_warm // layers + 1
        one = load(wl, reserve_extra=grow, interleave=inter,
                   rows_override={r: x[:max(1, x.shape[0] - short)] for r, x in rows_full.items()},
                   placement_seed=wl.placement_seed, backing=args.backing, n_layers=layers,
                   device_pages=int(args.device_pages))
        lds = [one] * layers
    else:
        lds = []
        for li in range(layers):
            # one token short of the configured context after this layer's warmup appends
            rows_li = {r: x[:max(1, x.shape[0] - pre[li] - 1)] for r, x in rows_full.items()}
            lds.append(load(wl, reserve_extra=grow, interleave=inter, rows_override=rows_li,
                            placement_seed=wl.placement_seed + 1000 * li, backing=args.backing,
                            device_pages=int(args.device_pages)))
    del rows_full
    # one new token per request per step: seeded rows, resident on the GPU before timing
    new_rows = to_device_u16(np.concatenate([wl.step_rows_bits(r, 0).reshape(-1) for r in range(B)]), "cuda")
    # request ids and append counts marshalled once (the steps repeat them)
    from paper_2606_24506_amd import crosspool as cpl
    ones = cpl.i32_array([1] * B)
    ids = [cpl.i32_array(ld.req_ids) for ld in lds]
    stream = torch.cuda.current_stream()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    for a, b in ev:
        a.record(stream)
        b.record(stream)
    torch.cuda.synchronize()
    opts = dict(num_splits=args.splits, path=args.path, schedule=args.schedule)

    # device pointers and the stream handle taken once, as a serving loop
    # would hold them
    ptrs = [(ld.q.data_ptr(), ld.out.data_ptr(), ld.lse.data_ptr()) for ld in lds]
    rows_p, stream_p = new_rows.data_ptr(), stream.cuda_stream

    def step(i, evs=None):
        ld, rid, (q_p, o_p, l_p) = lds[i % layers], ids[i % layers], ptrs[i % layers]
        o = opts
        if evs is not None:
            o = dict(opts, ev_begin=evs[0].cuda_event, ev_end=evs[1].cuda_event)
        if args.unfused:
            ld.pool.append(rid, ones, rows_p, stream_p)
            ld.pool.decode(rid, q_p, o_p, l_p, stream_p, **o)
        else:
            ld.pool.decode_step(rid, ones, rows_p, q_p, o_p, l_p, stream_p, **o)

    if args.copy_mib:
        src = torch.empty(args.copy_mib << 20, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        dst.copy_(src)
        del src, dst
    # Clock settling: the attention kernels of the 128-head batches draw
    # enough power that the clocks take tens of milliseconds of continuous
    # work to settle after an idle gap. Decode-only calls (no appends, so no
    # context grows) fill args.settle_seconds of GPU time.
    settle = 0
    if args.settle_seconds > 0:
        t0 = time.perf_counter()
        for i in range(10):
            ld = lds[i % layers]
            ld.pool.decode(ld.req_ids, ld.q, ld.out, ld.lse, stream, **opts)
        torch.cuda.synchronize()
        per = (time.perf_counter() - t0) / 10
        settle = 10 + max(0, min(MAX_SETTLE_CALLS, math.ceil(args.settle_seconds / per)) - 10)
        for i in range(10, settle):
            ld = lds[i % layers]
            ld.pool.decode(ld.req_ids, ld.q, ld.out, ld.lse, stream, **opts)
    for i in range(n_warm):
        step(i)
    torch.cuda.synchronize()
    ctx0 = [[ld.pool.ctx_len(r) for r in ld.req_ids] for ld in lds]
    if args.planes:  # tokens in flight through the planes count for the layers they reached
        ctx0 = [[c + (li < lds[0].pool.cursor(r)[0]) for c, r in zip(ctx0[li], lds[0].req_ids)]
                for li in range(layers)]
    # Throughput pass: K steps with nothing but the work in the stream.
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(n_warm + i)
    t_enq = time.perf_counter() - t0
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    # Kernel-timing pass: the next K steps, with HIP events taken by the
    # decode launches themselves on the launch stream (start of the first,
    # end of the last attention kernel of each call). Launching with events
    # costs the host tens of microseconds per call, enough to leave the GPU
    # waiting, so these steps are not part of the throughput figure.
    for i in range(args.steps):
        step(n_warm + args.steps + i, ev[i])
    torch.cuda.synchronize()
    kern_each = sorted(a.elapsed_time(b) for a, b in ev)
    kern_ms = sum(kern_each) / args.steps
    pct = lambda q: kern_each[min(len(kern_each) - 1, int(q * len(kern_each)))]
    # algorithmic bytes of the two timed passes (contexts grow by one per visit)
    dec_bytes, app_bytes, dec_bytes_timed, dec_flops_timed = 0, 0, 0, 0
    first_ctx = None
    visits = [0] * layers
    for i in range(2 * args.steps):
        li = (n_warm + i) % layers
        ctx = [c + visits[li] + 1 for c in ctx0[li]]
        if first_ctx is None:
            first_ctx = ctx
        visits[li] += 1
        if i < args.steps:
            dec_bytes += algorithmic_bytes_decode(wl, ctx)
            app_bytes += sum(2 * wl.model(r).kappa + 4 for r in range(B))
        else:
            dec_bytes_timed += algorithmic_bytes_decode(wl, ctx)
            dec_flops_timed += algorithmic_flops_decode(wl, ctx)
    configured = [rq.ctx_len for rq in wl.requests]

    value = (dec_bytes + app_bytes) / wall / 1e9
    ms_per_step = wall * 1e3 / args.steps
    achieved = dec_bytes_timed / args.steps / (kern_ms * 1e-3) / 1e9
    tflops = dec_flops_timed / args.steps / (kern_ms * 1e-3) / 1e12
    traffic, traffic_alg = measured_traffic(cfg)
    rec = {
        "value": round(value, 2),
        "ms_per_step": round(ms_per_step, 5),
        "config": {
            "workload": WORKLOAD_NAMES[cfg],
            "requests": B,
            "context_tokens_configured": int(sum(configured)),
            "context_tokens_first_timed_step": int(sum(first_ctx)),
            "first_timed_step_at_configured_lengths": (not args.planes) and list(first_ctx) == configured,
            "context_growth_per_timed_pass": -(-args.steps // layers),
            "kv_bytes_per_step": int(kv_bytes),
            "layers_cycled": layers,
            "step": ("cp_kv_append (1 token/request) + cp_attn_decode" if args.unfused
                     else "cp_attn_decode_step: 1 appended token/request + decode, append fused into the launch"),
            "path": ["auto", "vector", "matrix"][args.path],
            "schedule": ["balanced", "queue", "grid"][args.schedule],
            "backing": ["buffer", "virtual"][args.backing],
            "new_pages": "device free-page stacks" if args.device_pages else "host allocation",
            "layers_as": "KV planes of one pool (layer cursor)" if args.planes else "one pool per layer",
            "settle_calls": settle,
        },
        "req_tokens_per_s": round(B / (wall / args.steps), 1),
        "host_enqueue_ms_per_step": round(t_enq * 1e3 / args.steps, 5),
        "context_tokens_per_s": round(sum(ctx0[0]) / (wall / args.steps), 1),
        "roofline": {
            "bound": "hbm",
            "kernel": KERNEL_NAMES.get(cfg, "decode attention") + ": cp_attn_decode's attention launch, merge excluded",
            "achieved": round(achieved, 2),
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBS, 4),
            "traffic": traffic,
            "traffic_unit": "bytes per decode launch (rocprofv3 FETCH_SIZE + WRITE_SIZE, copy-calibrated)",
            "traffic_algorithmic_bytes": traffic_alg,  # of the launches the counters saw
            "algorithmic_bytes_per_launch": int(dec_bytes_timed / args.steps),
            "kernel_ms": round(kern_ms, 5),
            "kernel_ms_p10_p50_p90": [round(pct(0.1), 5), round(pct(0.5), 5), round(pct(0.9), 5)],
        },
        # the whole step (fused append, attention, split merge, launch gaps)
        # against the same roofline: decode bytes per step over the
        # throughput pass's wall time per step
        "whole_step": {
            "achieved": round(dec_bytes / args.steps / (ms_per_step * 1e-3) / 1e9, 2),
            "unit": "GB/s",
            "frac": round(dec_bytes / args.steps / (ms_per_step * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
        },
        # the same kernel's attention arithmetic against the dense bf16
        # matrix-core peak (the many-head MLA batches are the ones near it)
        "matrix": {
            "achieved": round(tflops, 2),
            "peak": MFMA_BF16_PEAK_TFLOPS,
            "unit": "TFLOP/s",
            "frac": round(tflops / MFMA_BF16_PEAK_TFLOPS, 4),
        },
    }
    log(f"cfg{cfg}: kernel {kern_ms * 1e3:.1f} us, {achieved:.0f} GB/s ({achieved / HBM_PEAK_GBS:.3f}), "
        f"step {ms_per_step * 1e3:.1f} us")
    for ld in (lds[:1] if args.planes else lds):
        ld.close()
    del lds
    torch.cuda.empty_cache()
    return rec


def measure_layer_launch(cfg: int, args) -> dict:
    """One pool whose models have L KV planes; a step takes one new token
    per request through all L layers, either as L per-layer
    cp_attn_decode_step calls (the host moving the layer cursors) or as one
    cp_attn_decode_layers call (the launch moving them). Same queries and
    rows for every layer (timing only). Returns both records."""
    import torch

    from workloads import make_workload
    from workloads.harness import load, to_device_u16

    L = args.layer_launch
    wl = make_workload(cfg, scale_ctx=args.ctx_scale)
    if wl.filler_pages:
        sys.exit("--layer-launch: the filler requests of this pool leave no room for more KV planes")
    B = len(wl.requests)
    steps, warm = args.steps, args.warmup
    ld = load(wl, reserve_extra=2 * (warm + 2 * steps) + 4, n_layers=L, device_pages=int(args.device_pages))
    hq = [wl.model(r).n_q_heads for r in range(B)]
    qd = [wl.model(r).d_k for r in range(B)]
    dv = [wl.model(r).d_v for r in range(B)]
    q1 = ld.q
    qL = torch.cat([q1[sum(h * d for h, d in zip(hq[:r], qd[:r])):][:hq[r] * qd[r]].repeat(L) for r in range(B)])
    outL = torch.empty(L * sum(h * d for h, d in zip(hq, dv)), dtype=torch.int16, device="cuda")
    lseL = torch.empty(L * sum(hq), dtype=torch.float32, device="cuda")
    row1 = [wl.step_rows_bits(r, 0).reshape(-1) for r in range(B)]
    rows1 = to_device_u16(np.concatenate(row1), "cuda")
    rowsL = to_device_u16(np.concatenate([np.tile(x, L) for x in row1]), "cuda")
    ones = [1] * B
    stream = torch.cuda.current_stream()

    def per_layer():
        for _ in range(L):
            ld.pool.decode_step(ld.req_ids, ones, rows1, q1, ld.out, ld.lse, stream)

    def one_call():
        ld.pool.decode_layers(ld.req_ids, ones, rowsL, qL, outL, lseL, stream)

    rec = {}
    for name, fn in (("per_layer_steps", per_layer), ("one_launch", one_call)):
        for _ in range(warm):
            fn()
        torch.cuda.synchronize()
        ctx = [ld.pool.ctx_len(r) for r in ld.req_ids]
        t0 = time.perf_counter()
        for _ in range(steps):
            fn()
        t_enq = time.perf_counter() - t0
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        by = sum(L * algorithmic_bytes_decode(wl, [c + 1 + i for c in ctx]) for i in range(steps))
        rec[name] = {"ms_per_token_step": round(wall * 1e3 / steps, 5),
                     "host_enqueue_ms_per_token_step": round(t_enq * 1e3 / steps, 5),
                     "decode_GBps": round(by / wall / 1e9, 2),
                     "frac_of_peak": round(by / wall / 1e9 / HBM_PEAK_GBS, 4)}
        log(f"cfg{cfg} x {L} layers, {name}: {rec[name]}")
    ld.close()
    torch.cuda.empty_cache()
    return {"workload": WORKLOAD_NAMES[cfg], "layers": L,
            "step": "one new token per request through every layer: L cp_attn_decode_step calls, or one "
                    "cp_attn_decode_layers call", **rec}


_STREAMS = []


def inflight_streams():
    """The two streams of the in-flight passes, made once per process (at
    the default priority) and reused by every workload: HIP maps streams
    onto a few hardware queues, and two streams that share one run their
    launches in turn."""
    import torch

    if not _STREAMS:
        _STREAMS.extend([torch.cuda.Stream(), torch.cuda.Stream()])
    return _STREAMS


def measure_inflight(cfg: int, args) -> dict:
    """Two batches in flight (the layer-wise pipeline keeps two batches,
    each with its own state, in flight; Section 3.2): two pools, each
    holding a copy of the workload, their decode steps issued alternately on
    two streams, against the same steps issued on one stream. Each pool
    stays on one stream; each batch cycles enough pools that the two
    together hold over 1 GiB of KV. Returns aggregate whole-step GB/s."""
    import torch

    from workloads import make_workload
    from workloads.harness import load, to_device_u16
    from paper_2606_24506_amd import crosspool as cpl

    wl = make_workload(cfg, scale_ctx=args.ctx_scale)
    if args.ctx_scale != 1.0 and wl.filler_pages:
        wl.filler_pages = int(wl.filler_pages * args.ctx_scale)
    B = len(wl.requests)
    kv_bytes = sum(rq.ctx_len * wl.model(r).kappa for r, rq in enumerate(wl.requests))
    lay = max(1, math.ceil((1 << 29) / kv_bytes))  # pools per batch
    K = max(2, args.steps)  # step pairs per timed pass
    warm = max(2, args.steps)
    visits_per_pool = -(-(2 * warm + 4 * K) // lay) + 2
    inter = 512 if cfg == 4 else (4096 if cfg == 5 else 0)
    pools = [[load(wl, reserve_extra=visits_per_pool, interleave=inter,
                   placement_seed=wl.placement_seed + 1000 * (b * lay + li) + 7) for li in range(lay)]
             for b in range(2)]
    new_rows = to_device_u16(np.concatenate([wl.step_rows_bits(r, 0).reshape(-1) for r in range(B)]), "cuda")
    ones = cpl.i32_array([1] * B)
    ids = [[cpl.i32_array(ld.req_ids) for ld in row] for row in pools]
    ptrs = [[(ld.q.data_ptr(), ld.out.data_ptr(), ld.lse.data_ptr()) for ld in row] for row in pools]
    streams = inflight_streams()
    sp = [st.cuda_stream for st in streams]
    rows_p = new_rows.data_ptr()
    visits = [[0] * lay for _ in range(2)]

    def pair(j, two, seen):
        for b in (0, 1):
            li = j % lay
            q_p, o_p, l_p = ptrs[b][li]
            pools[b][li].pool.decode_step(ids[b][li], ones, rows_p, q_p, o_p, l_p, sp[b] if two else sp[0])
            visits[b][li] += 1
            seen.append(visits[b][li])

    def bytes_of(seen):  # counted after the timed pass, off the host's issue path
        return sum(algorithmic_bytes_decode(wl, [rq.ctx_len + v for rq in wl.requests]) for v in seen)

    # clock settling as in measure(): decode-only calls (no context grows)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    n_settle = 0
    while time.perf_counter() - t0 < args.settle_seconds and n_settle < MAX_SETTLE_CALLS:
        for row in pools:
            for ld in row:
                ld.pool.decode(ld.req_ids, ld.q, ld.out, ld.lse, streams[0])
        n_settle += 1
        if n_settle % 8 == 0:
            streams[0].synchronize()
    # warmup, one pass in each mode: the first pass on two streams runs
    # slower than later ones (measured 5-10% on the V2-Lite batch), a one-time
    # cost of the second stream's first use
    j = 0
    for two in (False, True):
        for _ in range(warm):
            pair(j, two, [])
            j += 1
        torch.cuda.synchronize()
    rates = {1: [], 2: []}
    for two in (False, True, False, True):
        seen = []
        t0 = time.perf_counter()
        for _ in range(K):
            pair(j, two, seen)
            j += 1
        for st in streams:
            st.synchronize()
        dt = time.perf_counter() - t0
        rates[2 if two else 1].append(bytes_of(seen) / dt / 1e9)
        log(f"cfg{cfg}: in-flight pass on {'two streams' if two else 'one stream'}: {rates[2 if two else 1][-1]:.0f} GB/s")
    for row in pools:
        for ld in row:
            ld.close()
    torch.cuda.empty_cache()
    one, two = sum(rates[1]) / 2, sum(rates[2]) / 2
    log(f"cfg{cfg}: two batches in flight {two:.0f} GB/s against {one:.0f} GB/s on one stream")
    return {"workload": "two batches of " + WORKLOAD_NAMES[cfg],
            "step": "cp_attn_decode_step (1 appended token/request + decode) on each batch's pool in turn",
            "two_streams_GBps": round(two, 2), "one_stream_GBps": round(one, 2),
            "ratio": round(two / one, 4), "pools_per_batch": lay, "step_pairs_per_pass": K}


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only; --gpus {args.gpus} is not supported (the path does not shard).",
              file=sys.stderr)
        sys.exit(2)
    import torch

    from paper_2606_24506_amd import crosspool as cpl  # noqa: F401  (fails loudly without the built library)
    from workloads import make_workload

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    if args.also == "auto":
        also = [c for c in (2, 3, 4, 5) if c != args.config] if args.config in (2, 3, 4, 5) else []
    elif args.also in ("", "none"):
        also = []
    else:
        also = [int(x) for x in args.also.split(",") if x and int(x) != args.config]

    inflight_ok = not args.no_inflight and not (args.planes or args.unfused or args.device_pages or args.backing)
    if inflight_ok:
        inflight_streams()
    head = measure(args.config, args)
    if inflight_ok:
        head["two_batches_in_flight"] = measure_inflight(args.config, args)
    per_config = {}
    for c in also:
        r = measure(c, args)
        per_config[str(c)] = {"workload": WORKLOAD_NAMES[c], "value": r["value"], "unit": "GB/s",
                              "ms_per_step": r["ms_per_step"], "req_tokens_per_s": r["req_tokens_per_s"],
                              "host_enqueue_ms_per_step": r["host_enqueue_ms_per_step"],
                              "roofline": r["roofline"], "whole_step": r["whole_step"], "matrix": r["matrix"],
                              "config": r["config"]}
        if inflight_ok:
            per_config[str(c)]["two_batches_in_flight"] = measure_inflight(c, args)
    res = {
        "metric": "paged decode-attention achieved HBM GB/s and req-tokens/s on 1 MI355X",
        "value": head["value"],
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": head["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded draws shaped like the workload; no dataset)",
        "config": head["config"],
        "req_tokens_per_s": head["req_tokens_per_s"],
        "host_enqueue_ms_per_step": head["host_enqueue_ms_per_step"],
        "context_tokens_per_s": head["context_tokens_per_s"],
        "roofline": head["roofline"],
        "whole_step": head["whole_step"],
        "matrix": head["matrix"],
        "per_config": per_config,
    }
    if "two_batches_in_flight" in head:
        res["two_batches_in_flight"] = head["two_batches_in_flight"]
    if args.layer_launch:
        res["layer_launch"] = measure_layer_launch(2 if args.config == 3 else args.config, args)
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline(make_workload(args.config), args.cpu_seconds)
    print(json.dumps(res))


if __name__ == "__main__":
    main()
