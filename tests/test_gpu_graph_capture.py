"""GPU: cp_attn_decode_noalloc captured into a HIP graph (through torch's
graph capture) and replayed. The call allocates nothing and enqueues only
kernel launches, so a captured decode replays the same launches: every
replay must give the eager call's outputs and lse bit for bit, with the
program's own eager work (refilling the outputs with NaN) and
synchronizations between the replays, and meet the oracle's bars. Covered:
the balanced schedule (split requests, merge launch) and the work-queue
schedule, whose device counters the last workgroup of each launch resets.
A graph holds the kernel arguments of the moment it was captured (the
contexts attend at their lengths then), so this checks repeated decodes of
one batch state, not steps that grow it."""
import math

import numpy as np
import pytest
import torch

from parity import compare, expected_for
from paper_2606_24506_amd import crosspool as cpl
from workloads import MODELS, RequestSpec, Workload
from workloads.gen import normal_bf16
from workloads.harness import load

pytestmark = pytest.mark.gpu

LENS = [("mla128", 6000), ("mla16", 2500), ("gqa32x4", 1800), ("mqa32", 900), ("mla16", 130)]


def _workload():
    rng = np.random.default_rng(77)
    reqs = [RequestSpec(m, n) for m, n in LENS]
    qs = [normal_bf16(rng, (MODELS[m].n_q_heads, MODELS[m].d_k), 1.0) for m, _ in LENS]
    return Workload("graph", 77, reqs, qs, math.sqrt(0.5), 512 << 20, 2 << 20, 77)


def _fresh(ld):
    ld.out.fill_(0x7FC0)  # bf16 NaN: a result that is never written shows
    ld.lse.fill_(float("nan"))


def _snapshot(ld):
    torch.cuda.synchronize()
    return ld.out.cpu().numpy().view(np.uint16).copy(), ld.lse.cpu().numpy().view(np.uint32).copy()


@pytest.mark.parametrize("opts,label", [(dict(), "balanced"),
                                        (dict(schedule=cpl.CP_SCHED_QUEUE, num_splits=3), "queue x3")])
def test_captured_noalloc_decode_replays_bit_identically(opts, label):
    wl = _workload()
    print(f"[case] graph capture, {label}: loading", flush=True)
    ld = load(wl, interleave=37)
    try:
        ids = ld.req_ids
        exp = {r: expected_for(wl, r) for r in range(len(LENS))}
        # eager: the first call also resolves the fixed workspace's address
        # and loads the kernels' code objects, outside the capture
        ld.pool.decode_noalloc(ids, ld.q, ld.out, ld.lse, **opts)
        _fresh(ld)
        ld.pool.decode_noalloc(ids, ld.q, ld.out, ld.lse, **opts)
        want = _snapshot(ld)
        compare(ld, exp, f"eager noalloc {label}")

        print(f"[case] graph capture, {label}: capturing", flush=True)
        g = torch.cuda.CUDAGraph()
        _fresh(ld)
        torch.cuda.synchronize()
        with torch.cuda.graph(g):
            ld.pool.decode_noalloc(ids, ld.q, ld.out, ld.lse, **opts)  # on the capture stream
        torch.cuda.synchronize()
        for rep in range(4):
            _fresh(ld)  # eager work between the replays
            torch.cuda.synchronize()
            g.replay()
            got = _snapshot(ld)
            print(f"[case] graph capture, {label}: replay {rep}", flush=True)
            assert np.array_equal(got[0], want[0]), f"{label} replay {rep}: outputs differ from the eager call"
            assert np.array_equal(got[1], want[1]), f"{label} replay {rep}: lse differs from the eager call"
        compare(ld, exp, f"replayed noalloc {label}")
        # an eager call after the replays still agrees (the queue counters
        # were left at zero by every replay)
        _fresh(ld)
        ld.pool.decode_noalloc(ids, ld.q, ld.out, ld.lse, **opts)
        got = _snapshot(ld)
        assert np.array_equal(got[0], want[0]) and np.array_equal(got[1], want[1])
        del g
    finally:
        ld.close()
