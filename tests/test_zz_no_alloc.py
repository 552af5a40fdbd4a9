"""GPU: cp_attn_decode_noalloc, the decode entry point that allocates no
device memory (its split workspace is a fixed device array), against
cp_attn_decode_ex on the same pool: outputs and lse bit for bit, and both
within the oracle's bars, on two calls in a row, the second with a smaller
batch; the noalloc call leaves the device's free memory unchanged while the
pool's own path grows its workspace; and a split plan past the fixed
workspace is refused before anything is enqueued."""
import math

import numpy as np
import pytest
import torch

from parity import compare, expected_for
from paper_2606_24506_amd import crosspool as cpl
from workloads import MODELS, RequestSpec, Workload
from workloads.gen import normal_bf16
from workloads.harness import load, to_device_u16

pytestmark = pytest.mark.gpu

# two 128-head requests give the big call about 34 MB of partials (of the
# 40 MiB the fixed workspace holds) under the balanced schedule
LENS = [("mla128", 16384), ("mla128", 8192), ("mla16", 3000), ("gqa32x4", 2500), ("mqa32", 1500),
        ("gqa32x8", 1200)]
SUBSET = [2, 3, 5]


def _workload():
    rng = np.random.default_rng(91)
    reqs = [RequestSpec(m, n) for m, n in LENS]
    qs = [normal_bf16(rng, (MODELS[m].n_q_heads, MODELS[m].d_k), 1.0) for m, _ in LENS]
    return Workload("noalloc", 91, reqs, qs, math.sqrt(0.5), 512 << 20, 2 << 20, 91)


class _Call:
    """Packed q, out and lse of one call over a subset of the requests."""

    def __init__(self, wl, idx):
        self.wl, self.idx = wl, idx
        self.q = to_device_u16(np.concatenate([wl.q_bits[r].reshape(-1) for r in idx]), "cuda")
        n_out = sum(wl.model(r).n_q_heads * wl.model(r).d_v for r in idx)
        n_lse = sum(wl.model(r).n_q_heads for r in idx)
        self.out = torch.zeros(n_out, dtype=torch.int16, device="cuda")
        self.lse = torch.zeros(n_lse, dtype=torch.float32, device="cuda")

    def fresh(self):
        self.out.fill_(0x7FC0)  # bf16 NaN: a result that is never written shows
        self.lse.fill_(float("nan"))

    def snapshot(self):
        return (self.out.cpu().numpy().view(np.uint16).copy(), self.lse.cpu().numpy().view(np.uint32).copy())

    # the views compare() reads, by position in this call
    def out_bits(self, k):
        m = self.wl.model(self.idx[k])
        off = sum(self.wl.model(r).n_q_heads * self.wl.model(r).d_v for r in self.idx[:k])
        return self.out[off:off + m.n_q_heads * m.d_v].cpu().numpy().view(np.uint16).reshape(m.n_q_heads, m.d_v)

    def lse_of(self, k):
        off = sum(self.wl.model(r).n_q_heads for r in self.idx[:k])
        return self.lse[off:off + self.wl.model(self.idx[k]).n_q_heads].cpu().numpy().astype(np.float64)


def test_noalloc_matches_decode_ex_on_two_calls():
    wl = _workload()
    print("[case] noalloc: loading", flush=True)
    ld = load(wl, interleave=61)
    try:
        ids = ld.req_ids
        big, small = _Call(wl, list(range(len(LENS)))), _Call(wl, SUBSET)
        exp = {r: expected_for(wl, r) for r in range(len(LENS))}
        # The runtime loads a kernel's code object and sizes its private
        # segment at that kernel's first launch in the process: one unsplit
        # decode (one KV range per request, no split workspace on any path)
        # launches every kernel of these calls before anything is measured.
        for call in (big, small):
            ld.pool.decode([ids[r] for r in call.idx], call.q, call.out, call.lse, schedule=cpl.CP_SCHED_QUEUE,
                           num_splits=1)
        torch.cuda.synchronize()
        for call, opts, label in ((big, dict(), "balanced, all requests"),
                                  (small, dict(schedule=cpl.CP_SCHED_QUEUE, num_splits=5), "queue x5, 3 requests")):
            rids = [ids[r] for r in call.idx]
            print(f"[case] noalloc {label}", flush=True)
            free0 = torch.cuda.mem_get_info()[0]
            call.fresh()
            ld.pool.decode_noalloc(rids, call.q, call.out, call.lse, **opts)
            torch.cuda.synchronize()
            free1 = torch.cuda.mem_get_info()[0]
            got = call.snapshot()
            compare(call, {k: exp[r] for k, r in enumerate(call.idx)}, f"noalloc {label}")
            call.fresh()
            ld.pool.decode(rids, call.q, call.out, call.lse, **opts)
            torch.cuda.synchronize()
            free2 = torch.cuda.mem_get_info()[0]
            want = call.snapshot()
            assert np.array_equal(got[0], want[0]), f"{label}: outputs differ from cp_attn_decode_ex"
            assert np.array_equal(got[1], want[1]), f"{label}: lse differs from cp_attn_decode_ex"
            print(f"[mem] {label}: free memory change noalloc {free0 - free1} B, decode_ex {free1 - free2} B",
                  flush=True)
            assert free0 - free1 < (16 << 20), "the noalloc call took device memory"
            if call is big:  # the pool's own path allocates its (doubled) workspace on first use
                assert free1 - free2 >= (16 << 20)
        # a plan past the fixed workspace: every range of both 128-head
        # requests forced (384 ranges x 128 KiB of partials) is refused
        with pytest.raises(cpl.CrossPoolError) as e:
            ld.pool.decode_noalloc(ids, big.q, big.out, big.lse, schedule=cpl.CP_SCHED_QUEUE, num_splits=256)
        assert e.value.status == cpl.CP_EINVAL and "workspace" in e.value.message
    finally:
        ld.close()
