"""GPU: two batches in flight. Two pools share no device state, so their
decode steps may run concurrently on two streams (the layer-wise pipeline's
two in-flight batches). Several fused decode steps per pool are issued on two
streams without synchronising between them, each step writing its own output
buffers; the same steps on a second pair of pools (same placement seeds)
issued on one stream must give the same bits, and the results meet the fp64
oracle's tolerance. Balanced and work-queue schedules (the queue schedule's
counters live in each pool)."""
import math

import numpy as np
import pytest
import torch

from parity import OUT_MAX_ABS, OUT_REL_L2, LSE_MAX_ABS
import oracle
from paper_2606_24506_amd import crosspool as cpl
from workloads import MODELS, RequestSpec, Workload
from workloads.gen import normal_bf16
from workloads.harness import load, to_device_u16

pytestmark = pytest.mark.gpu

BATCHES = [[("mla128", 700), ("mla16", 1500), ("mqa32", 300), ("gqa32x4", 64)],
           [("mla16", 63), ("mla128", 2100), ("gqa16x4d64", 900), ("mla32", 333)]]
STEPS = 6


def _bits(t):
    return t.cpu().numpy().view(np.uint16 if t.dtype == torch.int16 else np.uint32)


def _workload(specs, seed):
    rng = np.random.default_rng(seed)
    reqs = [RequestSpec(m, n) for m, n in specs]
    qs = [normal_bf16(rng, (MODELS[m].n_q_heads, MODELS[m].d_k), 1.0) for m, _ in specs]
    return Workload(f"inflight{seed}", seed, reqs, qs, math.sqrt(0.5), 256 << 20, 2 << 20, seed)


@pytest.mark.parametrize("schedule,splits", [(cpl.CP_SCHED_BALANCED, 0), (cpl.CP_SCHED_QUEUE, 3)])
def test_two_pools_on_two_streams(schedule, splits):
    print(f"[case] two batches in flight sched{schedule} s{splits}", flush=True)
    wls = [_workload(specs, 40 + b) for b, specs in enumerate(BATCHES)]
    rng = np.random.default_rng(9)
    new = [[[normal_bf16(rng, (1, wl.model(r).row_width), 0.7) for r in range(len(wl.requests))]
            for _ in range(STEPS)] for wl in wls]
    loads = {}
    try:
        for mode in ("two", "one"):
            loads[mode] = [load(wl, reserve_extra=STEPS + 1, interleave=11) for wl in wls]
        outs = {}
        for mode in ("two", "one"):
            streams = [torch.cuda.Stream(), torch.cuda.Stream()] if mode == "two" else [torch.cuda.Stream()] * 2
            res = []
            rows_dev = [[to_device_u16(np.concatenate([x.reshape(-1) for x in new[b][s]]), "cuda")
                         for s in range(STEPS)] for b in range(2)]
            bufs = [[(torch.empty_like(loads[mode][b].out), torch.empty_like(loads[mode][b].lse)) for _ in range(STEPS)]
                    for b in range(2)]
            torch.cuda.synchronize()
            for s in range(STEPS):
                for b in range(2):
                    ld = loads[mode][b]
                    o, l = bufs[b][s]
                    # q, rows and the output buffers were made on the default
                    # stream and synchronised above; every step of a pool stays
                    # on that pool's stream
                    ld.pool.decode_step(ld.req_ids, [1] * len(ld.req_ids), rows_dev[b][s], ld.q, o, l,
                                        streams[b], num_splits=splits, schedule=schedule)
            for st in streams:
                st.synchronize()
            outs[mode] = [[(_bits(o), _bits(l)) for o, l in bufs[b]] for b in range(2)]
        for b in range(2):
            for s in range(STEPS):
                assert np.array_equal(outs["two"][b][s][0], outs["one"][b][s][0]), f"batch {b} step {s}: out"
                assert np.array_equal(outs["two"][b][s][1], outs["one"][b][s][1]), f"batch {b} step {s}: lse"
        # the last step against the oracle
        for b, wl in enumerate(wls):
            ld = loads["two"][b]
            o_all, l_all = outs["two"][b][STEPS - 1]
            l_all = l_all.view(np.float32).astype(np.float64)
            oo = lo = 0
            for r in range(len(wl.requests)):
                m = wl.model(r)
                rows = np.concatenate([wl.rows_bits(r)] + [new[b][s][r] for s in range(STEPS)])
                assert ld.pool.ctx_len(ld.req_ids[r]) == rows.shape[0]
                o_ref, l_ref = oracle.decode(rows, wl.q_bits[r], m)
                o = oracle.bf16_bits_to_f64(o_all[oo:oo + m.n_q_heads * m.d_v].reshape(m.n_q_heads, m.d_v))
                d = o - o_ref
                assert np.abs(d).max() <= OUT_MAX_ABS
                assert np.sqrt((d * d).sum() / (o_ref * o_ref).sum()) <= OUT_REL_L2
                assert np.abs(l_all[lo:lo + m.n_q_heads] - l_ref).max() <= LSE_MAX_ABS
                oo += m.n_q_heads * m.d_v
                lo += m.n_q_heads
    finally:
        torch.cuda.synchronize()
        for lds in loads.values():
            for ld in lds:
                ld.close()
