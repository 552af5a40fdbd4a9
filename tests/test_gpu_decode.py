"""GPU parity: the HIP path (through the C ABI) against the fp64 oracle on
identical seeded inputs. Small cases span several pages, ragged tails and
all three KV layouts; full-size cases use the five workloads (the oracle
checks every request where it finishes in seconds, sampled requests
otherwise)."""
import math

import numpy as np
import pytest
import torch

import oracle
from parity import compare, expected_for
from paper_2606_24506_amd import crosspool as cpl
from workloads import MODELS, RequestSpec, Workload, make_workload
from workloads.gen import normal_bf16
from workloads.harness import load, to_device_u16

pytestmark = pytest.mark.gpu


def custom(models_lens, seed=1, pool_bytes=256 << 20, chunk=2 << 20, sigma_kv=math.sqrt(0.5)):
    rng = np.random.default_rng(seed)
    reqs = [RequestSpec(m, n) for m, n in models_lens]
    qs = [normal_bf16(rng, (MODELS[m].n_q_heads, MODELS[m].d_k), 1.0) for m, _ in models_lens]
    return Workload(f"custom{seed}", seed, reqs, qs, sigma_kv, pool_bytes, chunk, seed)


RAGGED = [("mla16", 1), ("mla16", 63), ("mla16", 64), ("mla16", 65), ("mla16", 700),
          ("mqa32", 2), ("mqa32", 129), ("mqa32", 1000),
          ("gqa32x4", 1), ("gqa32x4", 127), ("gqa32x4", 128), ("gqa32x4", 777),
          ("mla128", 5), ("mla128", 300)]


# ---------------------------------------------------------- scatter/gather

@pytest.mark.parametrize("seed", [0, 5])
def test_append_gather_bit_exact(seed):
    wl = custom(RAGGED, seed=3)
    wl.placement_seed = seed
    ld = load(wl, interleave=17)
    try:
        for r, rid in enumerate(ld.req_ids):
            rows = wl.rows_bits(r)
            n = rows.shape[0]
            dst = torch.empty(rows.size, dtype=torch.int16, device="cuda")
            ld.pool.gather(rid, 0, n, dst)
            got = dst.cpu().numpy().view(np.uint16).reshape(rows.shape)
            assert np.array_equal(got, oracle.gather_rows([rows])), f"request {r}"
            if n > 3:
                a, b = n // 3, n - 1
                part = torch.empty((b - a) * rows.shape[1], dtype=torch.int16, device="cuda")
                ld.pool.gather(rid, a, b - a, part)
                assert np.array_equal(part.cpu().numpy().view(np.uint16).reshape(b - a, -1), rows[a:b])
        with pytest.raises(cpl.CrossPoolError):
            ld.pool.gather(ld.req_ids[0], 0, 2, dst)  # past the 1-token context
    finally:
        ld.close()


def test_append_in_many_calls_matches_concatenation():
    wl = custom([("gqa32x4", 300), ("mla16", 260), ("mqa32", 190)], seed=4)
    pool = cpl.Pool(page_tokens=64, pool_bytes=wl.pool_bytes, chunk_bytes=wl.chunk_bytes, placement_seed=11, device=0)
    mids = {m: pool.register_spec(MODELS[m]) for m in wl.models_used()}
    rids = [pool.open(mids[rq.model], rq.ctx_len) for rq in wl.requests]
    rows = [wl.rows_bits(r) for r in range(3)]
    pos = [0, 0, 0]
    rng = np.random.default_rng(0)
    blocks = [[], [], []]
    while any(pos[r] < rows[r].shape[0] for r in range(3)):
        ids, nn, flat = [], [], []
        for r in range(3):
            k = int(min(rng.integers(0, 90), rows[r].shape[0] - pos[r]))
            ids.append(rids[r])
            nn.append(k)
            flat.append(rows[r][pos[r]:pos[r] + k].reshape(-1))
            blocks[r].append(rows[r][pos[r]:pos[r] + k])
            pos[r] += k
        pool.append(ids, nn, to_device_u16(np.concatenate(flat), "cuda"))
    for r in range(3):
        dst = torch.empty(rows[r].size, dtype=torch.int16, device="cuda")
        pool.gather(rids[r], 0, rows[r].shape[0], dst)
        assert np.array_equal(dst.cpu().numpy().view(np.uint16).reshape(rows[r].shape), oracle.gather_rows(blocks[r]))
    for r in rids:
        pool.close(r)
    pool.destroy()


# ------------------------------------------------------------ decode parity

BAL, QUE, GRD = cpl.CP_SCHED_BALANCED, cpl.CP_SCHED_QUEUE, cpl.CP_SCHED_GRID
SCHEDULES = [(BAL, 0), (QUE, 0), (QUE, 1), (QUE, 3), (GRD, 0), (GRD, 5)]


@pytest.mark.parametrize("schedule,splits", SCHEDULES)
@pytest.mark.parametrize("path", [cpl.CP_PATH_AUTO, cpl.CP_PATH_VALU])
def test_tiny_mla_workload(schedule, splits, path):
    wl = make_workload(1)
    ld = load(wl)
    try:
        ld.decode(num_splits=splits, schedule=schedule, path=path)
        torch.cuda.synchronize()
        compare(ld, {r: expected_for(wl, r) for r in range(4)}, f"cfg1 sched{schedule} s{splits} path{path}")
    finally:
        ld.close()


@pytest.mark.parametrize("schedule,splits", [(BAL, 0), (QUE, 0), (QUE, 1), (QUE, 4), (QUE, 64), (GRD, 4)])
@pytest.mark.parametrize("path", [cpl.CP_PATH_AUTO, cpl.CP_PATH_VALU])
def test_ragged_mixed_batch(schedule, splits, path):
    wl = custom(RAGGED, seed=7)
    ld = load(wl, interleave=23)
    try:
        ld.decode(num_splits=splits, schedule=schedule, path=path)
        torch.cuda.synchronize()
        compare(ld, {r: expected_for(wl, r) for r in range(len(RAGGED))}, f"ragged sched{schedule} s{splits} path{path}")
    finally:
        ld.close()


def test_balanced_schedule_rejects_forced_splits():
    wl = custom([("mla16", 100)], seed=2)
    ld = load(wl)
    try:
        with pytest.raises(cpl.CrossPoolError) as e:
            ld.decode(num_splits=2, schedule=BAL)
        assert e.value.status == cpl.CP_EINVAL
    finally:
        ld.close()


VARIANT_MODELS = [("mla16", 700), ("mla32", 333), ("mla128", 290), ("mqa16", 515), ("mqa32", 190),
                  ("gqa128x2", 257), ("mqa128", 129), ("gqa32x4", 450), ("gqa8x8d64", 97),
                  ("gqa32x8", 611), ("gqa16x8", 77), ("gqa24x8", 301), ("gqa16x4d64", 1043)]


@pytest.mark.parametrize("schedule,splits", SCHEDULES)
def test_every_kernel_variant(schedule, splits):
    """One request per geometry, so every matrix-core and vector variant runs
    (workgroups of 2, 4 and 8 waves in separate launches of one call)."""
    wl = custom(VARIANT_MODELS, seed=41)
    ld = load(wl, interleave=31)
    try:
        ld.decode(num_splits=splits, schedule=schedule)
        torch.cuda.synchronize()
        compare(ld, {r: expected_for(wl, r) for r in range(len(VARIANT_MODELS))}, f"variants sched{schedule} s{splits}")
        # the vector path on the same data agrees too
        ld.decode(num_splits=splits, schedule=schedule, path=cpl.CP_PATH_VALU)
        torch.cuda.synchronize()
        compare(ld, {r: expected_for(wl, r) for r in range(len(VARIANT_MODELS))}, f"variants vector sched{schedule}")
    finally:
        ld.close()


@pytest.mark.parametrize("schedule,splits", [(BAL, 0), (QUE, 0), (GRD, 2)])
def test_many_requests_in_one_call(schedule, splits):
    """150 requests of six models in one call: more requests than one launch
    takes (64) and more models than one launch holds (4), so the call runs
    several launch groups and several merge launches."""
    rng = np.random.default_rng(77)
    names = ["mla16", "mqa32", "gqa32x4", "gqa16x4d64", "mla128", "mqa128"]
    lens = [(names[int(rng.integers(0, len(names)))], int(np.exp(rng.uniform(0, np.log(2000))))) for _ in range(150)]
    wl = custom(lens, seed=78, pool_bytes=1 << 30)
    print(f"[case] 150 requests sched{schedule} s{splits}", flush=True)
    ld = load(wl, interleave=50)
    try:
        ld.decode(num_splits=splits, schedule=schedule)
        torch.cuda.synchronize()
        compare(ld, {r: expected_for(wl, r) for r in range(len(lens))}, f"150 requests sched{schedule}")
    finally:
        ld.close()


def test_forced_matrix_path_rejects_narrow_groups():
    """One query head per KV head has no matrix-core variant."""
    wl = custom([("gqa8x8d64", 10)], seed=3)
    ld = load(wl)
    try:
        with pytest.raises(cpl.CrossPoolError) as e:
            ld.decode(path=cpl.CP_PATH_MFMA)
        assert e.value.status == cpl.CP_EINVAL
    finally:
        ld.close()


def test_single_token_returns_v_exactly():
    """n = 1: the softmax weight is exactly 1, so every head's output is its
    KV head's V row, bit for bit, and lse is the scaled score."""
    wl = custom([("mla16", 1), ("mqa32", 1), ("gqa32x4", 1), ("mla128", 1), ("mla32", 1), ("mqa128", 1),
                 ("mla16", 40)], seed=9)
    ld = load(wl)
    try:
        ld.decode()
        torch.cuda.synchronize()
        for r in range(6):
            m = wl.model(r)
            row = wl.rows_bits(r)[0]
            got = ld.out_bits(r)
            for h in range(m.n_q_heads):
                if m.kind == "mla":
                    v = row[: m.latent_dim]
                else:
                    kv = h // (m.n_q_heads // m.n_kv_heads)
                    d = m.head_dim
                    v = row[m.n_kv_heads * d + kv * d: m.n_kv_heads * d + (kv + 1) * d]
                assert np.array_equal(got[h], v), f"request {r} head {h}"
        compare(ld, {r: expected_for(wl, r) for r in range(7)}, "single-token")
    finally:
        ld.close()


def test_uniform_scores_give_mean_and_ln_n():
    """q = 0: output = mean of V, lse = ln n."""
    lens = [("mla16", 3000), ("mqa32", 1234), ("gqa32x4", 999)]
    wl = custom(lens, seed=12)
    zq = [np.zeros_like(q) for q in wl.q_bits]
    ld = load(wl, q_override=zq)
    try:
        ld.decode()
        torch.cuda.synchronize()
        for r, (_, n) in enumerate(lens):
            assert np.allclose(ld.lse_of(r), math.log(n), atol=1e-5, rtol=0)
        compare(ld, {r: oracle.decode(wl.rows_bits(r), zq[r], wl.model(r)) for r in range(3)}, "uniform")
    finally:
        ld.close()


def test_placement_does_not_change_a_single_bit():
    wl = custom(RAGGED, seed=21)
    outs = []
    for seed, inter in ((0, 0), (77, 9), (12345, 64)):
        ld = load(wl, placement_seed=seed, interleave=inter)
        try:
            ld.decode()
            torch.cuda.synchronize()
            outs.append((ld.out.cpu().numpy().copy(), ld.lse.cpu().numpy().copy()))
        finally:
            ld.close()
    for o, l in outs[1:]:
        assert np.array_equal(o, outs[0][0]) and np.array_equal(l.view(np.uint32), outs[0][1].view(np.uint32))


def test_split_and_unsplit_agree():
    wl = custom([("mla16", 5000), ("gqa32x4", 4100), ("mqa32", 2300)], seed=31)
    ld = load(wl)
    try:
        ld.decode(num_splits=1, schedule=QUE)
        torch.cuda.synchronize()
        a = ld.out.clone()
        exp = {r: expected_for(wl, r) for r in range(3)}
        compare(ld, exp, "unsplit")
        for k in (2, 7, 40):
            ld.decode(num_splits=k, schedule=QUE)
            torch.cuda.synchronize()
            compare(ld, exp, f"split{k}")
        d = (a.view(torch.bfloat16).float() - ld.out.view(torch.bfloat16).float()).abs().max().item()
        assert d <= 1e-2
    finally:
        ld.close()


def test_decode_errors():
    wl = custom([("mla16", 10)], seed=2)
    ld = load(wl)
    try:
        empty = ld.pool.open(ld.model_ids["mla16"], 100)
        with pytest.raises(cpl.CrossPoolError) as e:
            ld.pool.decode([empty], ld.q, ld.out, ld.lse)
        assert e.value.status == cpl.CP_EINVAL
        with pytest.raises(cpl.CrossPoolError):
            ld.pool.decode([ld.req_ids[0], ld.req_ids[0]], ld.q, ld.out, ld.lse)
        ld.pool.close(empty)
    finally:
        ld.close()


# ---------------------------------------------------------- full-size runs

def test_full_v2lite_batch():
    wl = make_workload(2)
    ld = load(wl)
    try:
        ld.decode()
        torch.cuda.synchronize()
        compare(ld, {r: expected_for(wl, r) for r in range(len(wl.requests))}, "cfg2 full")
    finally:
        ld.close()


def test_full_mixed_batch():
    wl = make_workload(4)
    ld = load(wl, interleave=512)
    try:
        ld.decode()
        torch.cuda.synchronize()
        compare(ld, {r: expected_for(wl, r) for r in range(len(wl.requests))}, "cfg4 full")
    finally:
        ld.close()


def test_full_v3_long_batch():
    """All 8 requests of 128K tokens at 128 heads, in the launch
    configuration the benchmark times (balanced schedule, automatic path)."""
    wl = make_workload(3)
    ld = load(wl)
    try:
        ld.decode()
        torch.cuda.synchronize()
        exp = {}
        for r in range(len(wl.requests)):
            exp[r] = expected_for(wl, r)
            print(f"[oracle] cfg3 request {r} done", flush=True)
        compare(ld, exp, "cfg3 full (all 8 requests)")
    finally:
        ld.close()


def test_full_burst_append_then_decode():
    """512K-token request in a pool 90% full: each step appends one token,
    then decodes; step rows come from the seeded per-step stream."""
    wl = make_workload(5)
    ld = load(wl, reserve_extra=256, interleave=4096)
    try:
        rows = wl.rows_bits(0)
        steps = 3
        for t in range(steps):
            new = wl.step_rows_bits(0, t)
            ld.pool.append([ld.req_ids[0]], [1], to_device_u16(new, "cuda"))
            rows = np.concatenate([rows, new])
            ld.decode()
        torch.cuda.synchronize()
        assert ld.pool.ctx_len(ld.req_ids[0]) == 524288 + steps
        s = ld.pool.stats()
        assert s["pages_used"] >= 25804
        compare(ld, {0: expected_for(wl, 0, rows=rows)}, "cfg5 burst")
    finally:
        ld.close()
