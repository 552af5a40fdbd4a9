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


def test_refused_step_changes_nothing():
    """A step whose split plan needs more workspace than the pool may hold
    (max_workspace_bytes) is refused with CP_ENOMEM before any page is
    allocated: context lengths, cursors, page tables and pool statistics
    stay as they were. The same step then runs unsplit (one KV range per
    request needs no workspace) and appends exactly once."""
    lens = [("mla16", 4096), ("mqa32", 1000)]  # 4096: the new token opens a page
    wl = custom(lens, seed=13)
    pool = cpl.Pool(page_tokens=64, pool_bytes=wl.pool_bytes, chunk_bytes=wl.chunk_bytes, placement_seed=3,
                    device=0, max_workspace_bytes=4096)
    mids = {m: pool.register_spec(MODELS[m]) for m in wl.models_used()}
    rids = [pool.open(mids[rq.model], rq.ctx_len + 8) for rq in wl.requests]
    rows = [wl.rows_bits(r) for r in range(len(lens))]
    for rid, rw in zip(rids, rows):
        pool.append([rid], [rw.shape[0]], to_device_u16(rw, "cuda"))
    q = to_device_u16(np.concatenate([x.reshape(-1) for x in wl.q_bits]), "cuda")
    out = torch.zeros(sum(MODELS[m].n_q_heads * MODELS[m].d_v for m, _ in lens), dtype=torch.int16, device="cuda")
    lse = torch.zeros(sum(MODELS[m].n_q_heads for m, _ in lens), dtype=torch.float32, device="cuda")
    rng = np.random.default_rng(14)
    new = [normal_bf16(rng, (1, wl.model(r).row_width), 0.7) for r in range(len(lens))]
    new_dev = to_device_u16(np.concatenate([x.reshape(-1) for x in new]), "cuda")

    def state():
        return ([pool.ctx_len(r) for r in rids], [pool.cursor(r) for r in rids],
                [pool.pages(r).tolist() for r in rids], pool.stats())

    try:
        torch.cuda.synchronize()
        before = state()
        for fn in (lambda: pool.decode_step(rids, [1, 1], new_dev, q, out, lse),  # balanced: splits
                   lambda: pool.decode_step(rids, [1, 1], new_dev, q, out, lse, schedule=cpl.CP_SCHED_QUEUE,
                                            num_splits=3),
                   lambda: pool.decode(rids, q, out, lse, schedule=cpl.CP_SCHED_GRID)):
            with pytest.raises(cpl.CrossPoolError) as e:
                fn()
            assert e.value.status == cpl.CP_ENOMEM
            assert state() == before
        pool.decode_step(rids, [1, 1], new_dev, q, out, lse, schedule=cpl.CP_SCHED_QUEUE, num_splits=1)
        torch.cuda.synchronize()
        assert [pool.ctx_len(r) for r in rids] == [n + 1 for _, n in lens]
        for r, rid in enumerate(rids):
            full = np.concatenate([rows[r], new[r]])
            dst = torch.empty(full.size, dtype=torch.int16, device="cuda")
            pool.gather(rid, 0, full.shape[0], dst)
            torch.cuda.synchronize()
            assert np.array_equal(_bits(dst).reshape(full.shape), full)

        class _View:
            def out_bits(self, r):
                off = sum(MODELS[m].n_q_heads * MODELS[m].d_v for m, _ in lens[:r])
                m = wl.model(r)
                return _bits(out)[off:off + m.n_q_heads * m.d_v].reshape(m.n_q_heads, m.d_v)

            def lse_of(self, r):
                off = sum(MODELS[m].n_q_heads for m, _ in lens[:r])
                return lse.cpu().numpy()[off:off + wl.model(r).n_q_heads].astype(np.float64)

        compare(_View(), {r: expected_for(wl, r, rows=np.concatenate([rows[r], new[r]])) for r in range(len(lens))},
                "refused then unsplit step")
    finally:
        torch.cuda.synchronize()
        for r in rids:
            pool.close(r)
        pool.destroy()
