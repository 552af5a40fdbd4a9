"""GPU parity on inputs that move the online-softmax maximum.

Every decode kernel keeps a running reference maximum per query head and
moves it lazily: only when a new tile's maximum exceeds it by more than 8
log2 units does it rescale the accumulated outputs and row sums by
alpha = 2^(m_old - m_new). With i.i.d. normal inputs the first tile's
maximum is never beaten by that margin, so the only rescale that runs is the
first tile's, where alpha multiplies zeros. These tests build inputs whose
scores climb in steps, so the rescale runs many times inside one piece with
non-zero accumulators, with a different pattern for every query head, and
so that split partials with lse values tens of units apart meet in the
merge. Each run is compared with the fp64 oracle at the usual bars.

Input structure (checked by `_assert_mid_piece_rescales` before any GPU
work): one K coordinate per KV head (the last rotary dimension for MLA, the
last dimension of each K head for GQA/MQA) carries a "level" L_j that is
constant over contiguous spans of 37-150 tokens and steps up by one at each
span boundary; query head h carries 2 f_h on the matching coordinate, with
f_h drawn per head from {2, 1.5, 1, 0.5, 0, -1}. A level step then moves
head h's scores by about 10 f_h log2 units: heads with f_h >= 1 rescale at
every step, f_h = 0.5 every other step, f_h <= 0 never after the first tile.
The "dominant" inputs instead plant three single tokens (one a third of
the way in, one two thirds in, and the request's last token, in its last
page), each 15 f_h log2 units above the previous one.
"""
import math

import numpy as np
import pytest
import torch

import oracle
from parity import compare
from paper_2606_24506_amd import crosspool as cpl
from workloads import MODELS, RequestSpec, Workload
from workloads.gen import f32_to_bf16_bits
from workloads.harness import load

pytestmark = pytest.mark.gpu

BAL, QUE, GRD = cpl.CP_SCHED_BALANCED, cpl.CP_SCHED_QUEUE, cpl.CP_SCHED_GRID

# One request per kernel geometry: narrow matrix (MLA-16, MLA-32, MQA-16,
# MQA-32, GQA-32:4 padded to 16), wide matrix (MLA-128, GQA-128:2,
# MQA-128), small-group vector (groups of 1-4, head_dim 64 and 128).
MODELS_LENS = [("mla16", 1999), ("mla32", 2111), ("mla128", 2300), ("mqa16", 1537), ("mqa32", 2049),
               ("gqa128x2", 1201), ("mqa128", 1800), ("gqa32x4", 2222), ("gqa8x8d64", 1500),
               ("gqa32x8", 1750), ("gqa16x8", 1303), ("gqa24x8", 2400), ("gqa16x4d64", 1650)]

Q0 = 2.0             # query weight of the level coordinate, times f_h
STEP_LOG2 = 10.0     # score step of one level for f_h = 1, in log2 units (above the lazy threshold of 8)
FACTORS = np.array([2.0, 1.5, 1.0, 0.5, 0.0, -1.0])
LAZY_LOG2 = 8.0
TILE = 32


def _level_dims(m):
    """(K coordinates carrying the level, one per KV head; the query coordinate)."""
    if m.kind == "mla":
        return [m.d_k - 1], m.d_k - 1
    d = m.head_dim
    return [kv * d + d - 1 for kv in range(m.n_kv_heads)], d - 1


def _inputs(m, n, seed, kind):
    """bf16 bits (rows [n, row_width], q [Hq, d_k]) and the per-head factors."""
    rng = np.random.default_rng(seed)
    q = rng.standard_normal((m.n_q_heads, m.d_k), dtype=np.float32)
    rows = rng.standard_normal((n, m.row_width), dtype=np.float32) * np.float32(math.sqrt(0.5))
    f = rng.choice(FACTORS, size=m.n_q_heads)
    f[:len(FACTORS)] = FACTORS  # every factor appears at least once
    kdims, qdim = _level_dims(m)
    q[:, qdim] = Q0 * f
    # K value of one level step, so that a step moves an f = 1 head by STEP_LOG2
    c = STEP_LOG2 * math.log(2.0) / (m.scale * Q0)
    level = np.zeros(n)
    if kind == "staircase":
        j, lv = 0, 0
        while j < n:
            span = int(rng.integers(37, 151))
            level[j:j + span] = lv
            j += span
            lv += 1
    else:  # three planted tokens, 1.5 steps apart
        for k, pos in enumerate((n // 3 + 5, 2 * n // 3 + 11, n - 1)):
            level[pos] = 1.5 * (k + 1)
    for kd in kdims:
        rows[:, kd] = level * c
    return f32_to_bf16_bits(rows), f32_to_bf16_bits(q), f


def _assert_mid_piece_rescales(m, rows, q, f, kind):
    """The inputs do what the module docstring says: over 32-token tiles of
    the whole request (the unsplit piece), the running maximum of the scaled
    scores (log2 units) is beaten by more than the lazy threshold at least
    twice after the first tile, for every head with f_h >= 1."""
    K, _ = oracle.kv_views(rows, m)
    qq = oracle.bf16_bits_to_f64(q)
    g = m.n_q_heads // m.n_kv_heads
    n = rows.shape[0]
    counts = []
    for h in range(m.n_q_heads):
        s = (K[h // g] @ qq[h]) * m.scale / math.log(2.0)
        tmax = [s[t:t + TILE].max() for t in range(0, n, TILE)]
        ref, bumps = tmax[0], 0
        for x in tmax[1:]:
            if x > ref + LAZY_LOG2:
                bumps += 1
                ref = x
        counts.append(bumps)
    counts = np.array(counts)
    need = 2 if kind == "dominant" else 5
    assert (counts[f >= 1.0] >= need).all(), (m.name, kind, counts[f >= 1.0].min())
    if kind == "staircase":
        assert (counts[f <= 0.0] == 0).all()
    return counts


def _workload(kind, seed, models_lens=MODELS_LENS):
    reqs, qs, rows, facs = [], [], {}, []
    for r, (name, n) in enumerate(models_lens):
        m = MODELS[name]
        rw, qb, f = _inputs(m, n, seed * 1000 + r, kind)
        counts = _assert_mid_piece_rescales(m, rw, qb, f, kind)
        print(f"[inputs] {kind} {name} n={n}: tile-max bumps > {LAZY_LOG2:g} log2 per head "
              f"min/median/max {counts.min()}/{int(np.median(counts))}/{counts.max()}", flush=True)
        reqs.append(RequestSpec(name, n))
        qs.append(qb)
        rows[r] = rw
        facs.append(f)
    wl = Workload(f"rescale-{kind}", seed, reqs, qs, math.sqrt(0.5), 512 << 20, 2 << 20, seed)
    return wl, rows


@pytest.fixture(scope="module", params=["staircase", "dominant"])
def loaded(request):
    kind = request.param
    wl, rows = _workload(kind, seed=5 if kind == "staircase" else 6)
    ld = load(wl, rows_override=rows, interleave=29)
    exp = {r: oracle.decode(rows[r], wl.q_bits[r], wl.model(r)) for r in range(len(wl.requests))}
    yield kind, ld, exp
    ld.close()


# (schedule, forced splits): balanced; one piece per request (every rescale
# inside one piece); a few long pieces; the planner's ranges; many short ones
@pytest.mark.parametrize("schedule,splits", [(BAL, 0), (QUE, 1), (QUE, 4), (GRD, 0), (GRD, 9)])
@pytest.mark.parametrize("path", [cpl.CP_PATH_AUTO, cpl.CP_PATH_VALU])
def test_rescales_match_oracle(loaded, schedule, splits, path):
    kind, ld, exp = loaded
    label = f"{kind} sched{schedule} s{splits} path{path}"
    print(f"[case] {label}", flush=True)
    ld.out.zero_()
    ld.lse.zero_()
    ld.decode(num_splits=splits, schedule=schedule, path=path)
    torch.cuda.synchronize()
    compare(ld, exp, label)


def test_dominant_token_output_is_its_value_row():
    """One token whose score is far above every other (by more than 100
    log2 units) takes all the weight: the output is that token's V row to
    within the bf16 rounding of the output, and lse is its scaled score."""
    lens = [("mla128", 777), ("mla16", 640), ("mqa32", 1025), ("gqa32x4", 333), ("gqa32x8", 500)]
    rng = np.random.default_rng(8)
    reqs, qs, rows, pos_of = [], [], {}, []
    for r, (name, n) in enumerate(lens):
        m = MODELS[name]
        q = rng.standard_normal((m.n_q_heads, m.d_k), dtype=np.float32)
        rw = rng.standard_normal((n, m.row_width), dtype=np.float32) * np.float32(math.sqrt(0.5))
        kdims, qdim = _level_dims(m)
        q[:, qdim] = Q0
        pos = int(rng.integers(n // 2, n))
        for kd in kdims:
            rw[pos, kd] = 120.0 * math.log(2.0) / (m.scale * Q0)
        reqs.append(RequestSpec(name, n))
        qs.append(f32_to_bf16_bits(q))
        rows[r] = f32_to_bf16_bits(rw)
        pos_of.append(pos)
    wl = Workload("dominant1", 8, reqs, qs, math.sqrt(0.5), 256 << 20, 2 << 20, 8)
    ld = load(wl, rows_override=rows)
    try:
        for sched, splits in ((BAL, 0), (QUE, 1), (GRD, 5)):
            ld.decode(num_splits=splits, schedule=sched)
            torch.cuda.synchronize()
            for r in range(len(lens)):
                m = wl.model(r)
                _, V = oracle.kv_views(rows[r], m)
                g = m.n_q_heads // m.n_kv_heads
                got = oracle.bf16_bits_to_f64(ld.out_bits(r))
                for h in range(m.n_q_heads):
                    v = V[h // g][pos_of[r]]
                    # the other tokens' weights sum to less than 2^-100 of it
                    assert np.allclose(got[h], v, rtol=2.0 ** -8, atol=1e-30), (lens[r], h, sched)
            compare(ld, {r: oracle.decode(rows[r], wl.q_bits[r], wl.model(r)) for r in range(len(lens))},
                    f"dominant1 sched{sched}")
    finally:
        ld.close()
