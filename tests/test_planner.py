"""KV-cache planner (Section 3.1, Eq. 1-2; the pool budget of cp_pool_create).

Oracle pins: published SplitMix64 outputs; Eq. 1 for one request (a ramp
from the prompt to prompt + output, released at T); Eq. 2 for periodic
arrivals (an exact sum); the Monte Carlo mean against Campbell's theorem
(mean active KV = lambda * kappa * E[T (O_p + O_d / 2)]); the quantile
against the Poisson law of the number of active requests; and whole-record
sampling against the product of marginals it must not reduce to. Then the
library's cp_plan_pool against the oracle on the same SplitMix64 draws."""
import json
import math
import os

import numpy as np
import pytest
from scipy.stats import poisson

import oracle
from oracle.planner import SplitMix64, active_tokens, plan_pool, pool_demand, quantile_rank

HERE = os.path.dirname(os.path.abspath(__file__))


def test_splitmix64_published_vectors():
    g = json.load(open(os.path.join(HERE, "golden", "splitmix64.json")))
    for v in g["vectors"]:
        r = SplitMix64(v["seed"])
        want = [int(x, 16) for x in v.get("outputs_hex", [])] or [int(x) for x in v["outputs_dec"]]
        assert [r.next_u64() for _ in want] == want


def test_eq1_single_request_ramp():
    # O_p = 100, O_d = 50, T = 10: 100 + 5u on [0, 10), nothing before or after
    for u, want in [(-1.0, 0.0), (0.0, 100.0), (5.0, 125.0), (9.5, 147.5), (10.0, 0.0), (12.0, 0.0)]:
        assert float(active_tokens(u, 100.0, 50.0, 10.0)) == want
    assert pool_demand(5.0, [(0.0, 2.0, 100.0, 50.0, 10.0)]) == 250.0  # kappa scales bytes


def test_eq2_periodic_arrivals_steady_state():
    # one arrival per second, T = 10: at t = 20.5 the ten requests of ages
    # 0.5 .. 9.5 are active: sum (100 + 5 u) = 1000 + 5 * 50
    arr = [(float(k), 1.0, 100.0, 50.0, 10.0) for k in range(30)]
    assert pool_demand(20.5, arr) == 1250.0
    # two models add (Eq. 2): a second model of kappa 3 with the same arrivals
    arr2 = arr + [(float(k), 3.0, 10.0, 0.0, 4.0) for k in range(30)]
    assert pool_demand(20.5, arr2) == 1250.0 + 3.0 * 10.0 * 4


def test_quantile_rank_is_the_inverse_empirical_cdf():
    v = [5.0, 1.0, 4.0, 2.0, 3.0]
    assert quantile_rank(v, 0.2) == 1.0 and quantile_rank(v, 0.21) == 2.0
    assert quantile_rank(v, 0.99) == 5.0 and quantile_rank(v, 1.0) == 5.0


def _model(kappa, rate, recs):
    op, od, tr = (np.array([r[i] for r in recs], dtype=np.float64) for i in range(3))
    return dict(kappa=kappa, rate=rate, prompt=op, output=od, residence=tr)


def test_monte_carlo_mean_follows_campbell():
    # lambda = 20/s, records of T in {1, 3}, mean active bytes =
    # lambda * kappa * E[T (O_p + O_d / 2)]
    recs = [(200, 100, 1.0), (50, 400, 3.0)]
    m = _model(64.0, 20.0, recs)
    want = 20.0 * 64.0 * np.mean([t * (p + d / 2) for p, d, t in recs])
    _, mean, _, _, _ = plan_pool([m], 4000.0, 20000, 0.99, 3, 1 << 20)
    assert abs(mean / want - 1) < 0.02


def test_quantile_follows_poisson_count():
    # no output growth and one residence time: the demand is kappa * O_p
    # times a Poisson(lambda T) count
    m = _model(1152.0, 10.0, [(1000, 0, 10.0)])
    for q in (0.95, 0.99):
        qb, _, _, pool, _ = plan_pool([m], 5000.0, 4000, q, 7, 2 << 20)
        n_emp = qb / (1152.0 * 1000)
        assert abs(n_emp - poisson.ppf(q, 100)) <= 3
        assert pool % (2 << 20) == 0 and qb <= pool < qb + (2 << 20)


def test_whole_records_keep_correlations():
    # long prompts stay briefly, short ones long: E[O_p T] = 1000, while
    # independent draws of the two would give E[O_p] E[T] = 505 * 50.5
    m = _model(1.0, 5.0, [(1000, 0, 1.0), (10, 0, 100.0)])
    _, mean, _, _, _ = plan_pool([m], 20000.0, 20000, 0.99, 11, 1 << 20)
    assert abs(mean / (5.0 * 1000.0) - 1) < 0.05
    assert mean < 0.1 * 5.0 * 505 * 50.5


# ------------------------------------------------------------- library

def _lib():
    from paper_2606_24506_amd import crosspool as cpl
    return cpl


def _trace(rng, n, p_scale, d_scale, t_scale):
    op = rng.integers(1, p_scale, n)
    od = rng.integers(0, d_scale, n)
    tr = t_scale * (0.2 + rng.random(n)) * (1 + od / d_scale)  # residence grows with output length
    return op, od, tr


def test_library_matches_oracle():
    cpl = _lib()
    rng = np.random.default_rng(4)
    specs = [(1152.0, 0.8, *_trace(rng, 37, 32768, 2048, 60.0)),   # MLA latent rows
             (512.0, 1.5, *_trace(rng, 23, 8192, 1024, 30.0)),     # MQA
             (2048.0, 0.3, *_trace(rng, 11, 65536, 512, 90.0))]    # GQA, 4 KV heads
    lib_models = [dict(kappa_bytes=k, arrival_rate=r, prompt_tokens=p, output_tokens=d, service_time_s=t)
                  for k, r, p, d, t in specs]
    orc_models = [dict(kappa=k, rate=r, prompt=p, output=d, residence=t) for k, r, p, d, t in specs]
    for q, seed in ((0.95, 1), (0.99, 2), (1.0, 3)):
        got = cpl.cp_plan_pool(lib_models, 3000.0, 3000, q, seed, 2 << 20)
        qb, mean, mx, pool, n_arr = plan_pool(orc_models, 3000.0, 3000, q, seed, 2 << 20)
        assert got["n_arrivals"] == n_arr
        assert math.isclose(got["quantile_bytes"], qb, rel_tol=1e-12)
        assert math.isclose(got["mean_bytes"], mean, rel_tol=1e-12)
        assert math.isclose(got["max_bytes"], mx, rel_tol=1e-12)
        assert got["pool_bytes"] == pool


def test_library_rejects_bad_inputs():
    cpl = _lib()
    ok = dict(kappa_bytes=1.0, arrival_rate=1.0, prompt_tokens=[10], output_tokens=[5], service_time_s=[2.0])
    with pytest.raises(cpl.CrossPoolError):
        cpl.cp_plan_pool([ok], 1.5, 10, 0.99, 1)            # horizon not past the residence time
    with pytest.raises(cpl.CrossPoolError):
        cpl.cp_plan_pool([ok], 10.0, 10, 0.0, 1)            # quantile outside (0, 1]
    with pytest.raises(cpl.CrossPoolError):
        cpl.cp_plan_pool([dict(ok, service_time_s=[0.0])], 10.0, 10, 0.99, 1)
    with pytest.raises(cpl.CrossPoolError):
        cpl.cp_plan_pool([dict(ok, arrival_rate=-1.0)], 10.0, 10, 0.99, 1)
    with pytest.raises(cpl.CrossPoolError):
        cpl.cp_plan_pool([], 10.0, 10, 0.99, 1)
