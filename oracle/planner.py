"""Oracle of the KV-cache planner (test infrastructure only; see __init__).

The planner sizes the shared KV-cache pool (Section 3.1, "KV-cache Planner
and Virtualizer"). For request i of model M, arriving at A_i with O_p,i
prompt tokens, O_d,i output tokens and decode residence time T_i, the active
KV tokens at age u grow linearly from the prompt to prompt + output over the
residence time and vanish when it ends (Eq. 1); the model's active KV bytes
at time t are kappa(M) times the sum over its requests; the pool demand is
the sum over models (Eq. 2). The budget is a high quantile (P95/P99) of the
pool demand at a random observation time, estimated by trace-driven Monte
Carlo: whole trace records are drawn, so the correlations between prompt
length, output length and residence time are kept. The quantile is then
rounded up to whole allocation units.

Readings where the paper leaves the procedure open:
  - arrivals of each model form a Poisson process of rate lambda_M over
    [0, H); each arrival draws one trace record uniformly;
  - observation times are uniform over [W, H), with W the longest residence
    time in any trace, so every request active at an observation time has
    its arrival inside the simulated window;
  - the q-quantile of n observations is the order statistic of rank
    ceil(q n) (the smallest value whose empirical CDF reaches q);
  - the budget rounds the quantile up to whole chunks of the pool allocator.

Random draws come from SplitMix64 (Steele, Lea and Flood, "Fast splittable
pseudorandom number generators", OOPSLA 2014), written here from its
published definition: the state advances by the golden-ratio increment and
each output is the state passed through the variant-13 mixing finalizer.
Uniforms take the top 53 bits. Draw order: for each model in order,
alternately an inter-arrival uniform and a record uniform until an arrival
falls at or past H (its record uniform is not drawn); then the observation
uniforms.
"""
from __future__ import annotations

import math
from typing import List, Sequence, Tuple

import numpy as np

_MASK = (1 << 64) - 1
_GAMMA = 0x9E3779B97F4A7C15


class SplitMix64:
    """SplitMix64 from its published definition (state += gamma; mix)."""

    def __init__(self, seed: int):
        self.state = seed & _MASK

    def next_u64(self) -> int:
        self.state = (self.state + _GAMMA) & _MASK
        z = self.state
        z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & _MASK
        z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & _MASK
        return z ^ (z >> 31)

    def uniform(self) -> float:
        """Uniform in [0, 1) with 53 random bits."""
        return (self.next_u64() >> 11) * (1.0 / 9007199254740992.0)


def active_tokens(age, prompt, output, residence):
    """Eq. 1: active KV tokens of a request at age u (0 outside [0, T))."""
    age = np.asarray(age, dtype=np.float64)
    inside = (age >= 0.0) & (age < residence)
    return np.where(inside, prompt + output * age / residence, 0.0)


def pool_demand(t: float, arrivals: Sequence[Tuple[float, float, float, float, float]]) -> float:
    """Eq. 1-2: pool KV bytes at time t for arrivals (A, kappa, O_p, O_d, T)."""
    total = 0.0
    for a, kappa, op, od, tr in arrivals:
        total += kappa * float(active_tokens(t - a, op, od, tr))
    return total


def simulate_arrivals(models, horizon: float, rng: SplitMix64) -> List[Tuple[float, float, float, float, float]]:
    """Poisson arrivals per model over [0, H), each drawing one whole trace record.

    models: sequence of dicts with kappa, rate, prompt, output, residence
    (the last three are equal-length arrays of trace records)."""
    out = []
    for m in models:
        n = len(m["prompt"])
        t = 0.0
        while True:
            u = rng.uniform()
            t += -math.log1p(-u) / m["rate"]
            if t >= horizon:
                break
            j = min(n - 1, int(rng.uniform() * n))
            out.append((t, float(m["kappa"]), float(m["prompt"][j]), float(m["output"][j]), float(m["residence"][j])))
    return out


def quantile_rank(values: Sequence[float], q: float) -> float:
    """Order statistic of rank ceil(q n) (1-based) of the values."""
    v = np.sort(np.asarray(values, dtype=np.float64))
    k = max(1, int(math.ceil(q * len(v))))
    return float(v[k - 1])


def plan_pool(models, horizon: float, n_obs: int, q: float, seed: int, chunk_bytes: int):
    """Monte Carlo pool budget: (quantile bytes, mean bytes, max bytes, pool bytes, n arrivals).

    Each observation sums Eq. 1 over the arrivals in (t - W, t], the only
    ones that can be active (no residence exceeds W), in arrival order."""
    rng = SplitMix64(seed)
    arrivals = simulate_arrivals(models, horizon, rng)
    warm = max(float(np.max(m["residence"])) for m in models)
    if not horizon > warm:
        raise ValueError("the horizon must exceed the longest residence time")
    obs = [warm + rng.uniform() * (horizon - warm) for _ in range(n_obs)]
    arr = sorted(arrivals, key=lambda x: x[0])  # stable: model order on equal times
    a = np.array([x[0] for x in arr])
    kap, op, od, tr = (np.array([x[i] for x in arr]) for i in (1, 2, 3, 4))
    demand = []
    for t in obs:
        lo, hi = np.searchsorted(a, t - warm, side="right"), np.searchsorted(a, t, side="right")
        demand.append(float(np.sum(kap[lo:hi] * active_tokens(t - a[lo:hi], op[lo:hi], od[lo:hi], tr[lo:hi]))))
    qb = quantile_rank(demand, q)
    pool = int(math.ceil(qb / chunk_bytes)) * chunk_bytes
    return qb, float(np.mean(demand)), float(np.max(demand)), pool, len(arrivals)
