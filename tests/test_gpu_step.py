"""GPU: cp_attn_decode_step (append fused into the attention launch) against
cp_kv_append followed by cp_attn_decode_ex on an identical second pool:
outputs and lse bit for bit, pool contents bit for bit, and the final state
against the fp64 oracle. Contexts sit on and next to page boundaries, so the
steps allocate new pages whose entries travel with the launch."""
import numpy as np
import pytest
import torch

import oracle
from parity import compare, expected_for
from paper_2606_24506_amd import crosspool as cpl
from workloads import MODELS, RequestSpec, Workload
from workloads.gen import normal_bf16
from workloads.harness import load, to_device_u16

pytestmark = pytest.mark.gpu

def custom(models_lens, seed, pool_bytes=256 << 20, chunk=2 << 20, sigma_kv=0.7071):
    rng = np.random.default_rng(seed)
    reqs = [RequestSpec(m, n) for m, n in models_lens]
    qs = [normal_bf16(rng, (MODELS[m].n_q_heads, MODELS[m].d_k), 1.0) for m, _ in models_lens]
    return Workload(f"custom{seed}", seed, reqs, qs, sigma_kv, pool_bytes, chunk, seed)


STEP_MODELS = [("mla16", 63), ("mla16", 64), ("mla16", 1000), ("mla128", 127), ("mla128", 128),
               ("mqa32", 191), ("gqa32x4", 255), ("gqa32x8", 64), ("gqa16x4d64", 65), ("mqa128", 300),
               ("gqa128x2", 129), ("mla32", 2)]
STEPS = 3


def _bits(t):
    return t.cpu().numpy().view(np.uint16 if t.dtype == torch.int16 else np.uint32)


@pytest.mark.parametrize("schedule,splits,path", [
    (cpl.CP_SCHED_BALANCED, 0, cpl.CP_PATH_AUTO),
    (cpl.CP_SCHED_QUEUE, 4, cpl.CP_PATH_AUTO),
    (cpl.CP_SCHED_BALANCED, 0, cpl.CP_PATH_VALU),
])
def test_decode_step_matches_append_then_decode(schedule, splits, path):
    wl = custom(STEP_MODELS, seed=11)
    print(f"[case] decode_step sched{schedule} s{splits} path{path}", flush=True)
    a = load(wl, reserve_extra=STEPS, interleave=29)
    b = load(wl, reserve_extra=STEPS, interleave=29)
    rng = np.random.default_rng(5)
    rows_now = [wl.rows_bits(r) for r in range(len(STEP_MODELS))]
    try:
        opts = dict(num_splits=splits, schedule=schedule, path=path)
        for step in range(STEPS):
            # every request appends on the first step, about half later
            n_new = [1 if step == 0 else int(rng.integers(0, 2)) for _ in STEP_MODELS]
            new_rows = []
            for r, k in enumerate(n_new):
                if k:
                    m = wl.model(r)
                    new_rows.append(normal_bf16(rng, (1, m.row_width), 0.7))
                    rows_now[r] = np.concatenate([rows_now[r], new_rows[-1]])
            rows_dev = to_device_u16(np.concatenate([x.reshape(-1) for x in new_rows]), "cuda")
            a.pool.append(a.req_ids, n_new, rows_dev)
            a.pool.decode(a.req_ids, a.q, a.out, a.lse, **opts)
            b.pool.decode_step(b.req_ids, n_new, rows_dev, b.q, b.out, b.lse, **opts)
            torch.cuda.synchronize()
            assert np.array_equal(_bits(a.out), _bits(b.out)), f"step {step}: outputs differ"
            assert np.array_equal(_bits(a.lse), _bits(b.lse)), f"step {step}: lse differs"
        for r, rid in enumerate(b.req_ids):
            n = rows_now[r].shape[0]
            assert b.pool.ctx_len(rid) == n
            dst = torch.empty(rows_now[r].size, dtype=torch.int16, device="cuda")
            b.pool.gather(rid, 0, n, dst)
            torch.cuda.synchronize()
            assert np.array_equal(_bits(dst).reshape(rows_now[r].shape), oracle.gather_rows([rows_now[r]])), f"request {r}"
        compare(b, {r: expected_for(wl, r, rows=rows_now[r]) for r in range(len(STEP_MODELS))},
                f"decode_step sched{schedule} path{path}")
    finally:
        a.close()
        b.close()


def test_decode_step_without_appends_is_decode():
    wl = custom([("mla16", 300), ("mqa32", 77)], seed=12)
    a = load(wl)
    try:
        a.pool.decode_step(a.req_ids, [0, 0], None, a.q, a.out, a.lse)
        torch.cuda.synchronize()
        compare(a, {r: expected_for(wl, r) for r in range(2)}, "decode_step n_new=0")
        with pytest.raises(cpl.CrossPoolError):
            a.pool.decode_step(a.req_ids, [2, 0], a.q, a.q, a.out, a.lse)  # more than one row
        with pytest.raises(cpl.CrossPoolError):
            a.pool.decode_step(a.req_ids, [1, 0], None, a.q, a.out, a.lse)  # rows missing
        assert a.pool.ctx_len(a.req_ids[0]) == 300  # rejected calls change nothing
    finally:
        a.close()
