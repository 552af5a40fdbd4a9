"""GPU: all-layer launches (cp_attn_decode_layers). One call takes each
request's token step through every KV layer of its model; the launch itself
moves each request's device layer cursor as its layers complete. Against the
host-driven per-layer steps (cp_attn_decode_step once per layer, the host
moving the cursors) on a second pool: every (request, layer) output and lse
bit for bit, at every token step, with host page allocation and with device
page stacks, under the schedules whose split plan depends only on each
request's own length (queue and grid with forced splits; the balanced
schedule shares the cost line of the whole launch, so its splits, and the
rounding of split partials, depend on what else the launch holds: there the
outputs are held to the fp64 oracle's tolerance at every step). The device
cursor is back at layer 0 after every call with one token counted per new
token, and every plane's rows gather back."""
import numpy as np
import pytest
import torch

import oracle
from paper_2606_24506_amd import crosspool as cpl
from workloads import MODELS
from workloads.gen import normal_bf16
from workloads.harness import to_device_u16

pytestmark = pytest.mark.gpu

# (model, layers, initial context): contexts on and next to page boundaries
REQS = [("mla16", 3, 300), ("mla16", 3, 63), ("gqa32x4", 2, 129), ("mqa32", 1, 64), ("mla128", 2, 192),
        ("gqa16x4d64", 4, 1)]
TOKENS = 70


def _bits(t):
    return t.cpu().numpy().view(np.uint16 if t.dtype == torch.int16 else np.uint32)


def _dev(a):
    return to_device_u16(np.ascontiguousarray(a).reshape(-1), "cuda")


@pytest.mark.parametrize("schedule,splits,path,device_pages", [
    (cpl.CP_SCHED_QUEUE, 1, cpl.CP_PATH_AUTO, 0),
    (cpl.CP_SCHED_QUEUE, 3, cpl.CP_PATH_AUTO, 1),
    (cpl.CP_SCHED_GRID, 2, cpl.CP_PATH_VALU, 0),
    (cpl.CP_SCHED_BALANCED, 0, cpl.CP_PATH_AUTO, 1),
])
def test_layer_launch_matches_per_layer_steps(schedule, splits, path, device_pages):
    print(f"[case] all-layer launch sched{schedule} s{splits} path{path} device_pages{device_pages}", flush=True)
    rng = np.random.default_rng(77)
    specs = [MODELS[m] for m, _, _ in REQS]
    X = cpl.Pool(page_tokens=64, pool_bytes=256 << 20, chunk_bytes=1 << 20, placement_seed=4, device=0)
    Y = cpl.Pool(page_tokens=64, pool_bytes=256 << 20, chunk_bytes=1 << 20, placement_seed=6, device=0,
                 device_pages=device_pages)
    xr, yr = [], []
    try:
        rows = [[normal_bf16(rng, (n, MODELS[m].row_width), 0.7071) for _ in range(L)] for m, L, n in REQS]
        for P, ids in ((X, xr), (Y, yr)):
            mids = {(m, L): P.register_spec(MODELS[m], n_layers=L) for m, L, _ in REQS}
            ids += [P.open(mids[(m, L)], n + TOKENS + 1) for m, L, n in REQS]
            P.append(ids, [n for _, _, n in REQS], _dev(np.concatenate([np.stack(r).reshape(-1) for r in rows])))
        B = len(REQS)
        opts = dict(num_splits=splits, schedule=schedule, path=path)
        L_of = [L for _, L, _ in REQS]
        ho = [s.n_q_heads * s.d_v for s in specs]
        hl = [s.n_q_heads for s in specs]
        y_out = torch.empty(sum(L * o for L, o in zip(L_of, ho)), dtype=torch.int16, device="cuda")
        y_lse = torch.empty(sum(L * h for L, h in zip(L_of, hl)), dtype=torch.float32, device="cuda")
        tokens = [0] * B
        for step in range(TOKENS):
            n_new = [0 if (step + i) % 9 == 8 else 1 for i in range(B)]
            q = [[normal_bf16(rng, (s.n_q_heads, s.d_k), 1.0) for _ in range(L)] for s, L in zip(specs, L_of)]
            new = [[normal_bf16(rng, (1, s.row_width), 0.7) for _ in range(L)] if k else None
                   for s, L, k in zip(specs, L_of, n_new)]
            for i in range(B):
                if n_new[i]:
                    tokens[i] += 1
                    for l in range(L_of[i]):
                        rows[i][l] = np.concatenate([rows[i][l], new[i][l]])
            # all layers in one call
            y_rows = [new[i][l].reshape(-1) for i in range(B) if n_new[i] for l in range(L_of[i])]
            Y.decode_layers(yr, n_new, _dev(np.concatenate(y_rows)) if y_rows else None,
                            _dev(np.concatenate([q[i][l].reshape(-1) for i in range(B) for l in range(L_of[i])])),
                            y_out, y_lse, **opts)
            # reference: one host-driven step per layer
            ref_o = [[None] * L for L in L_of]
            ref_l = [[None] * L for L in L_of]
            for l in range(max(L_of)):
                act = [i for i in range(B) if L_of[i] > l]
                xo = torch.empty(sum(ho[i] for i in act), dtype=torch.int16, device="cuda")
                xl = torch.empty(sum(hl[i] for i in act), dtype=torch.float32, device="cuda")
                x_rows = [new[i][l].reshape(-1) for i in act if n_new[i]]
                X.decode_step([xr[i] for i in act], [n_new[i] for i in act],
                              _dev(np.concatenate(x_rows)) if x_rows else None,
                              _dev(np.concatenate([q[i][l].reshape(-1) for i in act])), xo, xl, **opts)
                torch.cuda.synchronize()
                ob, lb = _bits(xo), _bits(xl)
                oo = lo = 0
                for i in act:
                    ref_o[i][l], ref_l[i][l] = ob[oo:oo + ho[i]], lb[lo:lo + hl[i]]
                    oo += ho[i]
                    lo += hl[i]
            torch.cuda.synchronize()
            yo, yl = _bits(y_out), _bits(y_lse)
            yf = y_lse.cpu().numpy().astype(np.float64)
            exact = schedule != cpl.CP_SCHED_BALANCED
            oo = lo = 0
            for i in range(B):
                for l in range(L_of[i]):
                    if exact:
                        assert np.array_equal(yo[oo:oo + ho[i]], ref_o[i][l]), f"step {step} request {i} layer {l}: out"
                        assert np.array_equal(yl[lo:lo + hl[i]], ref_l[i][l]), f"step {step} request {i} layer {l}: lse"
                    if step % 23 == 0 or not exact:
                        o_ref, l_ref = oracle.decode(rows[i][l], q[i][l], specs[i])
                        o = oracle.bf16_bits_to_f64(yo[oo:oo + ho[i]].reshape(specs[i].n_q_heads, -1))
                        d = o - o_ref
                        assert np.abs(d).max() <= 2e-2 and np.sqrt((d * d).sum() / (o_ref * o_ref).sum()) <= 1e-2
                        assert np.abs(yf[lo:lo + hl[i]] - l_ref).max() <= 1e-3
                    oo += ho[i]
                    lo += hl[i]
            if step % 10 == 0 or step == TOKENS - 1:
                for i in range(B):
                    assert Y.layer_state(yr[i]) == (0, tokens[i]), f"step {step} request {i}: device cursor"
                    assert Y.cursor(yr[i]) == (0, 0)
                    assert Y.ctx_len(yr[i]) == X.ctx_len(xr[i]) == REQS[i][2] + tokens[i]
        for i, (m, L, n) in enumerate(REQS):
            ctx = Y.ctx_len(yr[i])
            dst = torch.empty(L * ctx * MODELS[m].row_width, dtype=torch.int16, device="cuda")
            Y.gather(yr[i], 0, ctx, dst)
            torch.cuda.synchronize()
            assert np.array_equal(_bits(dst).reshape(L, ctx, -1), np.stack(rows[i])), f"request {i}: planes"
    finally:
        torch.cuda.synchronize()
        for P, ids in ((X, xr), (Y, yr)):
            for r in ids:
                P.close(r)
            P.destroy()


def test_layer_launch_refuses_a_token_in_flight():
    print("[case] all-layer launch refused mid-token", flush=True)
    rng = np.random.default_rng(3)
    P = cpl.Pool(page_tokens=64, pool_bytes=64 << 20, chunk_bytes=1 << 20, placement_seed=1, device=0)
    rid = None
    try:
        mid = P.register_spec(MODELS["mla16"], n_layers=2)
        rid = P.open(mid, 200)
        P.append([rid], [10], _dev(normal_bf16(rng, (2, 10, MODELS["mla16"].row_width), 0.7)))
        spec = MODELS["mla16"]
        out = torch.empty(2 * spec.n_q_heads * spec.d_v, dtype=torch.int16, device="cuda")
        lse = torch.empty(2 * spec.n_q_heads, dtype=torch.float32, device="cuda")
        q1 = _dev(normal_bf16(rng, (spec.n_q_heads, spec.d_k), 1.0))
        P.decode_step([rid], [1], _dev(normal_bf16(rng, (1, spec.row_width), 0.7)), q1, out, lse)
        assert P.cursor(rid) == (1, 1)
        q2 = _dev(normal_bf16(rng, (2, spec.n_q_heads, spec.d_k), 1.0))
        with pytest.raises(cpl.CrossPoolError) as e:
            P.decode_layers([rid], [1], _dev(normal_bf16(rng, (2, spec.row_width), 0.7)), q2, out, lse)
        assert e.value.status == cpl.CP_ESTATE
        assert P.cursor(rid) == (1, 1) and P.ctx_len(rid) == 10
        torch.cuda.synchronize()
    finally:
        torch.cuda.synchronize()
        if rid is not None:
            P.close(rid)
        P.destroy()
