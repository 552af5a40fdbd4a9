"""GPU: the virtual backing (an address range per model, physical chunks
mapped at admission and unmapped at close) against the one-buffer backing
on identical inputs: decode outputs and lse bit for bit (plans never depend
on placement), appended rows gathered back bit-exact, the fp64 oracle's
tolerance, decode steps that grow into chunks mapped at admission, and
device memory taken and returned with the requests."""
import math

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


def custom(models_lens, seed, pool_bytes=256 << 20, chunk=2 << 20, sigma_kv=math.sqrt(0.5)):
    rng = np.random.default_rng(seed)
    reqs = [RequestSpec(m, n) for m, n in models_lens]
    qs = [normal_bf16(rng, (MODELS[m].n_q_heads, MODELS[m].d_k), 1.0) for m, _ in models_lens]
    return Workload(f"custom{seed}", seed, reqs, qs, sigma_kv, pool_bytes, chunk, seed)


def _bits(t):
    return t.cpu().numpy().view(np.uint16 if t.dtype == torch.int16 else np.uint32)


# one full chunk of each layout (mla16 28 pages, mqa32 64, gqa32x4 16), one
# token past it, ragged tails and the 128-head MLA kernel
VIRT_MODELS = [("mla16", 1792), ("mla16", 1793), ("mla128", 700), ("mqa32", 4096), ("mqa32", 97),
               ("gqa32x4", 1024), ("gqa32x4", 1), ("gqa16x4d64", 65), ("mqa128", 300)]


@pytest.mark.parametrize("schedule,splits", [(cpl.CP_SCHED_BALANCED, 0), (cpl.CP_SCHED_QUEUE, 4)])
def test_virtual_backing_matches_buffer(schedule, splits):
    wl = custom(VIRT_MODELS, seed=21)
    print(f"[case] virtual vs buffer sched{schedule} s{splits}", flush=True)
    a = load(wl, interleave=100)
    b = load(wl, interleave=100, backing=cpl.CP_BACKING_VIRTUAL)
    try:
        s = b.pool.stats()
        assert s["backing"] == cpl.CP_BACKING_VIRTUAL and s["chunks_used"] >= len(set(m for m, _ in VIRT_MODELS))
        opts = dict(num_splits=splits, schedule=schedule)
        a.pool.decode(a.req_ids, a.q, a.out, a.lse, **opts)
        b.pool.decode(b.req_ids, b.q, b.out, b.lse, **opts)
        torch.cuda.synchronize()
        assert np.array_equal(_bits(a.out), _bits(b.out))
        assert np.array_equal(_bits(a.lse), _bits(b.lse))
        compare(b, {r: expected_for(wl, r) for r in range(len(VIRT_MODELS))}, f"virtual sched{schedule}")
        for r, rid in enumerate(b.req_ids):
            rows = wl.rows_bits(r)
            dst = torch.empty(rows.size, dtype=torch.int16, device="cuda")
            b.pool.gather(rid, 0, rows.shape[0], dst)
            torch.cuda.synchronize()
            assert np.array_equal(_bits(dst).reshape(rows.shape), oracle.gather_rows([rows])), f"request {r}"
    finally:
        a.close()
        b.close()


def test_virtual_decode_step_grows_into_chunks_mapped_at_admission():
    # each request fills exactly one chunk of its model; its reservation
    # (4 more tokens) took a second chunk at admission, which the first
    # step's new token starts
    lens = [("mla16", 1792), ("mqa32", 4096), ("gqa32x4", 1024)]
    wl = custom(lens, seed=22)
    print("[case] virtual decode_step at chunk boundaries", flush=True)
    a = load(wl, reserve_extra=4)
    b = load(wl, reserve_extra=4, backing=cpl.CP_BACKING_VIRTUAL)
    rng = np.random.default_rng(8)
    rows_now = [wl.rows_bits(r) for r in range(len(lens))]
    try:
        assert b.pool.stats()["chunks_used"] == 6
        for step in range(3):
            new_rows = []
            for r in range(len(lens)):
                new_rows.append(normal_bf16(rng, (1, wl.model(r).row_width), 0.7))
                rows_now[r] = np.concatenate([rows_now[r], new_rows[-1]])
            rows_dev = to_device_u16(np.concatenate([x.reshape(-1) for x in new_rows]), "cuda")
            a.pool.decode_step(a.req_ids, [1] * len(lens), rows_dev, a.q, a.out, a.lse)
            b.pool.decode_step(b.req_ids, [1] * len(lens), rows_dev, b.q, b.out, b.lse)
            torch.cuda.synchronize()
            assert np.array_equal(_bits(a.out), _bits(b.out)), f"step {step}"
            assert np.array_equal(_bits(a.lse), _bits(b.lse)), f"step {step}"
            assert b.pool.stats()["chunks_used"] == 6
        compare(b, {r: expected_for(wl, r, rows=rows_now[r]) for r in range(len(lens))}, "virtual decode_step")
    finally:
        a.close()
        b.close()


def test_virtual_pool_takes_and_returns_device_memory():
    spec = MODELS["gqa32x4"]  # 2048 bytes per token, 16 pages per 2 MiB chunk
    chunk, n_tok = 2 << 20, 65536  # 64 chunks = 128 MiB
    p = cpl.Pool(page_tokens=64, pool_bytes=1 << 30, chunk_bytes=chunk, device=0, backing=cpl.CP_BACKING_VIRTUAL)
    rows = torch.randint(-30000, 30000, (n_tok * spec.row_width,), dtype=torch.int16, device="cuda")
    rows_host = rows.cpu().numpy()
    # every device tensor exists before memory is measured; comparisons run
    # on the host so that torch allocates nothing on the device in between
    dst = torch.empty_like(rows)
    try:
        m = p.register_spec(spec)
        torch.cuda.synchronize()
        free0 = torch.cuda.mem_get_info()[0]
        print(f"[case] virtual memory: free {free0}", flush=True)
        r1 = p.open(m, n_tok)
        free1 = torch.cuda.mem_get_info()[0]
        assert p.stats()["chunks_used"] == 64
        assert free0 - free1 >= 0.9 * 64 * chunk, (free0, free1)
        p.append([r1], [n_tok], rows)
        p.gather(r1, 0, n_tok, dst)
        torch.cuda.synchronize()
        assert p.stats()["chunks_used"] == 64
        assert np.array_equal(dst.cpu().numpy(), rows_host)
        p.close(r1)
        free2 = torch.cuda.mem_get_info()[0]
        assert p.stats()["chunks_used"] == 0
        assert free2 - free1 >= 0.9 * 64 * chunk, (free1, free2)
        # the range is mapped again on demand
        r2 = p.open(m, 4096)
        assert p.stats()["chunks_used"] == 4
        p.append([r2], [4096], rows[:4096 * spec.row_width])
        p.gather(r2, 0, 4096, dst[:4096 * spec.row_width])
        torch.cuda.synchronize()
        assert np.array_equal(dst[:4096 * spec.row_width].cpu().numpy(), rows_host[:4096 * spec.row_width])
        p.close(r2)
    finally:
        torch.cuda.synchronize()
        p.destroy()
