"""GPU: multi-layer models (one KV plane per layer, a layer cursor per
request). A pool holding models of 3, 2 and 1 layers runs decode steps in
which requests of different models sit at different layers of one launch;
every call must give, bit for bit, what single-layer requests holding each
(request, layer) pair's rows give in a second pool, and meet the fp64
oracle's tolerance. Gathers return every layer's rows; the cursor rules
(tokens in flight, commits, rejected calls) hold."""
import numpy as np
import pytest
import torch

import oracle
from paper_2606_24506_amd import crosspool as cpl
from workloads import MODELS
from workloads.gen import normal_bf16
from workloads.harness import to_device_u16

pytestmark = pytest.mark.gpu

# (model, layers, initial context)
REQS = [("mla16", 3, 300), ("mla16", 3, 63), ("gqa32x4", 2, 129), ("mqa32", 1, 64), ("mla128", 2, 200)]
TOKENS = 3  # new tokens per request over the test
SIGMA = 0.7071


def _bits(t):
    return t.cpu().numpy().view(np.uint16 if t.dtype == torch.int16 else np.uint32)


def _dev(a):
    return to_device_u16(np.ascontiguousarray(a).reshape(-1), "cuda")


def _check_oracle(rows, q_bits, spec, out_bits, lse, label):
    o_ref, l_ref = oracle.decode(rows, q_bits, spec)
    o = oracle.bf16_bits_to_f64(out_bits)
    d = o - o_ref
    assert np.abs(d).max() <= 2e-2, label
    assert np.sqrt((d * d).sum() / (o_ref * o_ref).sum()) <= 1e-2, label
    assert np.abs(lse - l_ref).max() <= 1e-3, label


@pytest.mark.parametrize("backing", [cpl.CP_BACKING_BUFFER, cpl.CP_BACKING_VIRTUAL])
def test_layer_cursors_match_single_layer_requests(backing):
    print(f"[case] multi-layer decode steps, backing {backing}", flush=True)
    rng = np.random.default_rng(31)
    X = cpl.Pool(page_tokens=64, pool_bytes=256 << 20, chunk_bytes=2 << 20, placement_seed=3, device=0,
                 backing=backing)
    Y = cpl.Pool(page_tokens=64, pool_bytes=256 << 20, chunk_bytes=2 << 20, placement_seed=9, device=0)
    specs = [MODELS[m] for m, _, _ in REQS]
    try:
        xm = {(m, L): X.register_spec(MODELS[m], n_layers=L) for m, L, _ in REQS}
        ym = {m: Y.register_spec(MODELS[m]) for m, _, _ in REQS}
        # rows[i][l]: the logical rows of request i at layer l
        rows = [[normal_bf16(rng, (n, MODELS[m].row_width), SIGMA) for _ in range(L)] for m, L, n in REQS]
        xr = [X.open(xm[(m, L)], n + TOKENS) for m, L, n in REQS]
        yr = [[Y.open(ym[m], n + TOKENS) for _ in range(L)] for m, L, n in REQS]
        X.append(xr, [n for _, _, n in REQS], _dev(np.concatenate([np.stack(r).reshape(-1) for r in rows])))
        for i, (m, L, n) in enumerate(REQS):
            for l in range(L):
                Y.append([yr[i][l]], [n], _dev(rows[i][l]))
        for i, (m, L, n) in enumerate(REQS):
            assert X.pages(xr[i], layers=L).shape == ((L, -(-n // 64)) if L > 1 else (-(-n // 64),))
        torch.cuda.synchronize()

        B = len(REQS)
        hq = [s.n_q_heads for s in specs]
        q_len = sum(h * s.d_k for h, s in zip(hq, specs))
        o_len = sum(h * s.d_v for h, s in zip(hq, specs))
        xo = torch.empty(o_len, dtype=torch.int16, device="cuda")
        yo = torch.empty_like(xo)
        xl = torch.empty(sum(hq), dtype=torch.float32, device="cuda")
        yl = torch.empty_like(xl)
        tokens_left = [TOKENS] * B
        step = 0
        while any(tokens_left) or any(X.cursor(r) != (0, 0) for r in xr):
            assert step < 40
            n_new, new_rows, yids = [], [], []
            for i, (m, L, n) in enumerate(REQS):
                layer, inflight = X.cursor(xr[i])
                k = inflight
                if layer == 0 and tokens_left[i] > 0 and step % 4 != 3:  # some steps place no token
                    k = 1
                    tokens_left[i] -= 1
                n_new.append(k)
                if k:
                    row = normal_bf16(rng, (1, MODELS[m].row_width), SIGMA)
                    new_rows.append(row)
                    rows[i][layer] = np.concatenate([rows[i][layer], row])
                yids.append(yr[i][layer])
            q = [normal_bf16(rng, (s.n_q_heads, s.d_k), 1.0) for s in specs]
            q_dev = _dev(np.concatenate([x.reshape(-1) for x in q]))
            rows_dev = _dev(np.concatenate([x.reshape(-1) for x in new_rows])) if new_rows else None
            cursors = [X.cursor(r)[0] for r in xr]
            X.decode_step(xr, n_new, rows_dev, q_dev, xo, xl)
            Y.decode_step(yids, n_new, rows_dev, q_dev, yo, yl)
            torch.cuda.synchronize()
            assert np.array_equal(_bits(xo), _bits(yo)), f"step {step}: outputs differ"
            assert np.array_equal(_bits(xl), _bits(yl)), f"step {step}: lse differs"
            if step % 3 == 0:
                ob, lv = _bits(xo), xl.cpu().numpy().astype(np.float64)
                oo = lo = 0
                for i, s in enumerate(specs):
                    nq = s.n_q_heads
                    _check_oracle(rows[i][cursors[i]], q[i], s, ob[oo:oo + nq * s.d_v].reshape(nq, s.d_v),
                                  lv[lo:lo + nq], f"step {step} request {i} layer {cursors[i]}")
                    oo += nq * s.d_v
                    lo += nq
            step += 1
        # every token went through every layer: all committed, cursors back at 0
        for i, (m, L, n) in enumerate(REQS):
            assert X.cursor(xr[i]) == (0, 0)
            assert X.ctx_len(xr[i]) == n + TOKENS - tokens_left[i]
            ctx = X.ctx_len(xr[i])
            dst = torch.empty(L * ctx * MODELS[m].row_width, dtype=torch.int16, device="cuda")
            X.gather(xr[i], 0, ctx, dst)
            torch.cuda.synchronize()
            assert np.array_equal(_bits(dst).reshape(L, ctx, -1), np.stack(rows[i])), f"request {i}"
    finally:
        torch.cuda.synchronize()
        for pool in (X, Y):
            for r in range(64):
                try:
                    pool.close(r)
                except cpl.CrossPoolError:
                    pass
            pool.destroy()


def test_layer_cursor_rules():
    print("[case] layer cursor rules", flush=True)
    rng = np.random.default_rng(5)
    p = cpl.Pool(page_tokens=64, pool_bytes=64 << 20, chunk_bytes=2 << 20, device=0)
    spec = MODELS["mqa32"]
    try:
        m = p.register_spec(spec, n_layers=2)
        assert p.info(m)["n_layers"] == 2
        r = p.open(m, 200)
        p.append([r], [64], _dev(normal_bf16(rng, (2, 64, spec.row_width), SIGMA)))
        q = _dev(normal_bf16(rng, (spec.n_q_heads, spec.d_k), 1.0))
        out = torch.empty(spec.n_q_heads * spec.d_v, dtype=torch.int16, device="cuda")
        lse = torch.empty(spec.n_q_heads, dtype=torch.float32, device="cuda")
        row = _dev(normal_bf16(rng, (1, spec.row_width), SIGMA))
        p.decode_step([r], [1], row, q, out, lse)  # layer 0 places token 64 (a new page in both planes)
        assert p.cursor(r) == (1, 1) and p.ctx_len(r) == 64
        assert p.pages(r, count=2, layers=2).shape == (2, 2)
        with pytest.raises(cpl.CrossPoolError, match="in flight"):
            p.append([r], [1], row)  # no bulk append mid-token
        with pytest.raises(cpl.CrossPoolError, match="n_new must be 1"):
            p.decode_step([r], [0], None, q, out, lse)  # layer 1 owes the token's row
        assert p.cursor(r) == (1, 1)
        p.decode([r], q, out, lse)  # a plain decode reads layer 1 and leaves the cursor alone
        assert p.cursor(r) == (1, 1)
        p.decode_step([r], [1], row, q, out, lse)
        assert p.cursor(r) == (0, 0) and p.ctx_len(r) == 65
        p.decode_step([r], [0], None, q, out, lse)  # a step without a new token
        assert p.cursor(r) == (1, 0)
        with pytest.raises(cpl.CrossPoolError, match="n_new must be 0"):
            p.decode_step([r], [1], row, q, out, lse)
        p.decode_step([r], [0], None, q, out, lse)
        assert p.cursor(r) == (0, 0) and p.ctx_len(r) == 65
        torch.cuda.synchronize()
        p.close(r)
    finally:
        torch.cuda.synchronize()
        p.destroy()
