"""GPU: decode steps on a pool with device free-page stacks. A new token
that opens a page takes it (in every KV plane) from its model's stack inside
the decode launch, and the host only refills stacks and reads the popped
page-table entries back at slow-path calls. Against the same steps on a pool
whose pages are allocated on the host: outputs and lse bit for bit at every
step, the same rows gathered back, the fp64 oracle's tolerance at the end;
the read-back entries are valid and distinct, a host-side append after the
read-back (which copies page-table ranges from the host's mirror to the
device) leaves every row in place, and closing every request returns every
chunk. Small chunks make the stacks refill often and pages cross chunk
boundaries; contexts start on and next to page boundaries."""
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

# (model, initial context): every page-table plane of these opens one or two
# pages over STEPS single-token steps
DP_MODELS = [("mla16", 63), ("mla16", 64), ("mla16", 1000), ("mla128", 127), ("mla128", 320),
             ("mqa32", 191), ("gqa32x4", 255), ("gqa32x4", 64), ("gqa16x4d64", 65), ("mla16", 1)]
STEPS = 70
CHUNK = 512 << 10  # 7 MLA pages per chunk: stacks refill every few steps


def _bits(t):
    return t.cpu().numpy().view(np.uint16 if t.dtype == torch.int16 else np.uint32)


def _workload(seed):
    rng = np.random.default_rng(seed)
    reqs = [RequestSpec(m, n) for m, n in DP_MODELS]
    qs = [normal_bf16(rng, (MODELS[m].n_q_heads, MODELS[m].d_k), 1.0) for m, _ in DP_MODELS]
    return Workload(f"devpages{seed}", seed, reqs, qs, 0.7071, 256 << 20, CHUNK, seed)


def _gather(ld, r, n, width):
    dst = torch.empty(n * width, dtype=torch.int16, device="cuda")
    ld.pool.gather(ld.req_ids[r], 0, n, dst)
    torch.cuda.synchronize()
    return _bits(dst).reshape(n, width)


@pytest.mark.parametrize("schedule,splits,path,backing", [
    (cpl.CP_SCHED_BALANCED, 0, cpl.CP_PATH_AUTO, cpl.CP_BACKING_BUFFER),
    (cpl.CP_SCHED_QUEUE, 4, cpl.CP_PATH_AUTO, cpl.CP_BACKING_BUFFER),
    (cpl.CP_SCHED_BALANCED, 0, cpl.CP_PATH_VALU, cpl.CP_BACKING_BUFFER),
    (cpl.CP_SCHED_BALANCED, 0, cpl.CP_PATH_AUTO, cpl.CP_BACKING_VIRTUAL),
])
def test_device_pages_match_host_allocation(schedule, splits, path, backing):
    print(f"[case] device pages sched{schedule} s{splits} path{path} backing{backing}", flush=True)
    wl = _workload(21)
    host = load(wl, reserve_extra=STEPS + 2, interleave=37, backing=backing)
    dev = load(wl, reserve_extra=STEPS + 2, interleave=37, backing=backing, device_pages=1)
    rng = np.random.default_rng(8)
    rows_now = [wl.rows_bits(r) for r in range(len(DP_MODELS))]
    try:
        opts = dict(num_splits=splits, schedule=schedule, path=path)
        for step in range(STEPS):
            # most requests append at most steps; the last one never does
            n_new = [int(rng.random() < 0.9) if r + 1 < len(DP_MODELS) else 0 for r in range(len(DP_MODELS))]
            new_rows = []
            for r, k in enumerate(n_new):
                if k:
                    new_rows.append(normal_bf16(rng, (1, wl.model(r).row_width), 0.7))
                    rows_now[r] = np.concatenate([rows_now[r], new_rows[-1]])
            rows_dev = to_device_u16(np.concatenate([x.reshape(-1) for x in new_rows]), "cuda")
            host.pool.decode_step(host.req_ids, n_new, rows_dev, host.q, host.out, host.lse, **opts)
            dev.pool.decode_step(dev.req_ids, n_new, rows_dev, dev.q, dev.out, dev.lse, **opts)
            torch.cuda.synchronize()
            assert np.array_equal(_bits(host.out), _bits(dev.out)), f"step {step}: outputs differ"
            assert np.array_equal(_bits(host.lse), _bits(dev.lse)), f"step {step}: lse differs"
        for r in range(len(DP_MODELS)):
            n, w = rows_now[r].shape
            assert dev.pool.ctx_len(dev.req_ids[r]) == n
            assert np.array_equal(_gather(dev, r, n, w), rows_now[r]), f"request {r}: gathered rows"
        compare(dev, {r: expected_for(wl, r, rows=rows_now[r]) for r in range(len(DP_MODELS))},
                f"device pages sched{schedule} path{path}")
        # read back: every entry valid, no page handed out twice
        ents = np.concatenate([dev.pool.pages(rid) for rid in dev.req_ids + dev.fillers])
        assert not np.any(ents == 0xFFFFFFFF)
        assert len(np.unique(ents)) == len(ents), "a page belongs to two requests"
        sd, sh = dev.pool.stats(), host.pool.stats()
        assert sd["pages_used"] == sh["pages_used"]
        # a host-side append after the read-back copies page-table ranges from
        # the mirror: every row must still be where the device put it
        extra = [normal_bf16(rng, (1, wl.model(r).row_width), 0.7) for r in range(len(DP_MODELS))]
        dev.pool.append(dev.req_ids, [1] * len(DP_MODELS),
                        to_device_u16(np.concatenate([x.reshape(-1) for x in extra]), "cuda"))
        for r in range(len(DP_MODELS)):
            rows_now[r] = np.concatenate([rows_now[r], extra[r]])
            n, w = rows_now[r].shape
            assert np.array_equal(_gather(dev, r, n, w), rows_now[r]), f"request {r}: rows after host append"
    finally:
        host.close()
        dev.close()


def test_device_pages_return_every_chunk():
    print("[case] device pages: stacks drained as requests close", flush=True)
    wl = _workload(22)
    dev = load(wl, reserve_extra=200, interleave=0, device_pages=1)
    ids, fillers = list(dev.req_ids), list(dev.fillers)
    try:
        rng = np.random.default_rng(3)
        n_req = len(ids)
        for step in range(40):
            rows = to_device_u16(np.concatenate([normal_bf16(rng, (1, wl.model(r).row_width), 0.7).reshape(-1)
                                                 for r in range(n_req)]), "cuda")
            dev.pool.decode_step(ids, [1] * n_req, rows, dev.q, dev.out, dev.lse)
        torch.cuda.synchronize()
        before = dev.pool.stats()
        assert before["chunks_used"] > 0
        # closing half the requests leaves the others able to grow to their
        # reservations; closing all returns every chunk (buffer backing)
        for rid in ids[::2]:
            dev.pool.close(rid)
        for rid in ids[1::2]:
            rows = to_device_u16(normal_bf16(rng, (1, MODELS[DP_MODELS[ids.index(rid)][0]].row_width), 0.7).reshape(-1),
                                 "cuda")
            n = dev.pool.ctx_len(rid)
            dev.pool.append([rid], [1], rows)
            assert dev.pool.ctx_len(rid) == n + 1
        for rid in ids[1::2] + fillers:
            dev.pool.close(rid)
        s = dev.pool.stats()
        assert s["requests_open"] == 0 and s["pages_used"] == 0
        assert s["chunks_used"] == 0, f"{s['chunks_used']} chunks still held after every request closed"
    finally:
        torch.cuda.synchronize()
        dev.pool.destroy()


def test_device_pages_multi_layer_steps():
    """Per-layer steps of 3- and 2-layer models: the layer-0 step pops one
    page per plane; later layers find their entry in the device table."""
    print("[case] device pages, multi-layer steps", flush=True)
    reqs = [("mla16", 3, 63), ("gqa32x4", 2, 128), ("mla16", 3, 200)]
    rng = np.random.default_rng(41)
    pools = [cpl.Pool(page_tokens=64, pool_bytes=128 << 20, chunk_bytes=CHUNK, placement_seed=5, device=0,
                      device_pages=d) for d in (0, 1)]
    rids = []
    try:
        mids = [{(m, L): P.register_spec(MODELS[m], n_layers=L) for m, L, _ in reqs} for P in pools]
        rows = [[normal_bf16(rng, (n, MODELS[m].row_width), 0.7071) for _ in range(L)] for m, L, n in reqs]
        for P, mid in zip(pools, mids):
            ids = [P.open(mid[(m, L)], n + 120) for m, L, n in reqs]
            P.append(ids, [n for _, _, n in reqs],
                     to_device_u16(np.concatenate([np.stack(r).reshape(-1) for r in rows]), "cuda"))
            rids.append(ids)
        specs = [MODELS[m] for m, _, _ in reqs]
        hq = [s.n_q_heads for s in specs]
        outs = [torch.empty(sum(h * s.d_v for h, s in zip(hq, specs)), dtype=torch.int16, device="cuda")
                for _ in pools]
        lses = [torch.empty(sum(hq), dtype=torch.float32, device="cuda") for _ in pools]
        for step in range(3 * 70):
            n_new, new_rows = [], []
            for i, (m, L, n) in enumerate(reqs):
                layer, inflight = pools[0].cursor(rids[0][i])
                k = 1 if layer == 0 and step % 5 != 4 else inflight
                n_new.append(k)
                if k:
                    row = normal_bf16(rng, (1, MODELS[m].row_width), 0.7)
                    new_rows.append(row)
                    rows[i][layer] = np.concatenate([rows[i][layer], row])
            q = to_device_u16(np.concatenate([normal_bf16(rng, (s.n_q_heads, s.d_k), 1.0).reshape(-1)
                                              for s in specs]), "cuda")
            rows_dev = to_device_u16(np.concatenate([x.reshape(-1) for x in new_rows]), "cuda") if new_rows else None
            for P, ids, o, l in zip(pools, rids, outs, lses):
                P.decode_step(ids, n_new, rows_dev, q, o, l)
            torch.cuda.synchronize()
            assert np.array_equal(_bits(outs[0]), _bits(outs[1])), f"step {step}: outputs differ"
            assert np.array_equal(_bits(lses[0]), _bits(lses[1])), f"step {step}: lse differs"
            assert [pools[1].cursor(r) for r in rids[1]] == [pools[0].cursor(r) for r in rids[0]]
        for i, (m, L, n) in enumerate(reqs):
            ctx = pools[1].ctx_len(rids[1][i])
            assert ctx == pools[0].ctx_len(rids[0][i])
            dst = torch.empty(L * ctx * MODELS[m].row_width, dtype=torch.int16, device="cuda")
            pools[1].gather(rids[1][i], 0, ctx, dst)
            torch.cuda.synchronize()
            got = _bits(dst).reshape(L, ctx, -1)
            # committed rows of every plane (a token in flight is not gathered)
            assert np.array_equal(got, np.stack([r[:ctx] for r in rows[i]])), f"request {i}"
            ents = pools[1].pages(rids[1][i], layers=L)
            assert not np.any(np.asarray(ents) == 0xFFFFFFFF)
    finally:
        torch.cuda.synchronize()
        for k, P in enumerate(pools):
            for r in (rids[k] if k < len(rids) else []):
                P.close(r)
            P.destroy()
