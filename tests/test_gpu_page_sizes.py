"""GPU parity at page sizes other than 64 tokens. The page size decides how
the decode kernels walk a piece: the 128-head MLA kernel takes pages of a
multiple of 32 tokens in 32-token tiles (one, four or eight tiles per page
here) and the narrow and small-group kernels pages of a multiple of 16;
other sizes go to the generic vector kernel. Each size runs a ragged batch
of every kernel family (contexts of one token, one short of and one past a
page or tile boundary, several pages) under the balanced schedule and under
forced splits, fused decode steps that open new pages, and unsplit pieces
long enough to reload the page-table entries several times, all against
the fp64 oracle at the usual bars."""
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

PAGE_SIZES = [16, 32, 48, 128, 256]
BATCH = [("mla128", 1), ("mla128", 31), ("mla128", 33), ("mla128", 700), ("mla16", 15), ("mla16", 257),
         ("mla32", 90), ("mqa32", 300), ("mqa128", 200), ("gqa32x4", 129), ("gqa16x4d64", 77), ("gqa32x8", 47)]


def _workload(seed):
    rng = np.random.default_rng(seed)
    reqs = [RequestSpec(m, n) for m, n in BATCH]
    qs = [normal_bf16(rng, (MODELS[m].n_q_heads, MODELS[m].d_k), 1.0) for m, _ in BATCH]
    return Workload(f"pages{seed}", seed, reqs, qs, math.sqrt(0.5), 256 << 20, 2 << 20, seed)


@pytest.mark.parametrize("page_tokens", PAGE_SIZES)
@pytest.mark.parametrize("schedule,splits", [(cpl.CP_SCHED_BALANCED, 0), (cpl.CP_SCHED_QUEUE, 3)])
def test_decode_at_page_size(page_tokens, schedule, splits):
    print(f"[case] page size {page_tokens} sched{schedule} s{splits}", flush=True)
    wl = _workload(31)
    ld = load(wl, interleave=19, page_tokens=page_tokens)
    try:
        ld.decode(num_splits=splits, schedule=schedule)
        torch.cuda.synchronize()
        compare(ld, {r: expected_for(wl, r) for r in range(len(BATCH))},
                f"page size {page_tokens} sched{schedule} s{splits}")
    finally:
        ld.close()


@pytest.mark.parametrize("page_tokens", [32, 128])
def test_fused_steps_at_page_size(page_tokens):
    """Decode steps whose new tokens open pages (contexts start one short of
    a page boundary), fused append included."""
    print(f"[case] fused steps at page size {page_tokens}", flush=True)
    specs = [("mla128", page_tokens - 1), ("mla16", 2 * page_tokens - 1), ("mqa32", page_tokens), ("gqa32x4", 5)]
    rng = np.random.default_rng(page_tokens)
    reqs = [RequestSpec(m, n) for m, n in specs]
    qs = [normal_bf16(rng, (MODELS[m].n_q_heads, MODELS[m].d_k), 1.0) for m, _ in specs]
    wl = Workload(f"steps{page_tokens}", 5, reqs, qs, math.sqrt(0.5), 256 << 20, 2 << 20, 5)
    steps = 3
    ld = load(wl, reserve_extra=steps + 1, interleave=7, page_tokens=page_tokens)
    rows_now = [wl.rows_bits(r) for r in range(len(specs))]
    try:
        for _ in range(steps):
            new = [normal_bf16(rng, (1, wl.model(r).row_width), 0.7) for r in range(len(specs))]
            for r in range(len(specs)):
                rows_now[r] = np.concatenate([rows_now[r], new[r]])
            rows_dev = to_device_u16(np.concatenate([x.reshape(-1) for x in new]), "cuda")
            ld.pool.decode_step(ld.req_ids, [1] * len(specs), rows_dev, ld.q, ld.out, ld.lse)
            torch.cuda.synchronize()
            compare(ld, {r: expected_for(wl, r, rows=rows_now[r]) for r in range(len(specs))},
                    f"step at page size {page_tokens}")
        for r, rid in enumerate(ld.req_ids):
            assert ld.pool.ctx_len(rid) == rows_now[r].shape[0]
    finally:
        ld.close()


@pytest.mark.parametrize("page_tokens", [32, 64])
def test_long_unsplit_pieces(page_tokens):
    """One piece per request (one forced KV range) over 70 to 290 pages:
    every kernel family reloads its batch of 64 page-table entries several
    times inside one piece."""
    print(f"[case] long unsplit pieces at page size {page_tokens}", flush=True)
    specs = [("mla128", 9000), ("mla16", 9001), ("mqa32", 5000), ("gqa32x4", 4500), ("gqa16x4d64", 4200),
             ("mqa128", 4300)]
    rng = np.random.default_rng(77)
    reqs = [RequestSpec(m, n) for m, n in specs]
    qs = [normal_bf16(rng, (MODELS[m].n_q_heads, MODELS[m].d_k), 1.0) for m, _ in specs]
    wl = Workload(f"long{page_tokens}", 13, reqs, qs, math.sqrt(0.5), 512 << 20, 2 << 20, 13)
    ld = load(wl, interleave=97, page_tokens=page_tokens)
    try:
        ld.decode(num_splits=1, schedule=cpl.CP_SCHED_QUEUE)
        torch.cuda.synchronize()
        compare(ld, {r: expected_for(wl, r) for r in range(len(specs))}, f"long unsplit pieces P{page_tokens}")
    finally:
        ld.close()
