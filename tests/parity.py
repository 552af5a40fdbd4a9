"""Comparison helpers for GPU-vs-oracle parity tests.

Bars (floating point): over a whole decode call, max |o_gpu - o_ref| <= 2e-2
and ||o_gpu - o_ref||_2 / ||o_ref||_2 <= 1e-2 with bf16 outputs upcast
exactly; max |lse_gpu - lse_ref| <= 1e-3 (natural log). Scatter and gather
are compared bit for bit.
"""
from __future__ import annotations

import numpy as np

import oracle

OUT_MAX_ABS = 2e-2
OUT_REL_L2 = 1e-2
LSE_MAX_ABS = 1e-3


def expected_for(wl, r, rows=None, q=None):
    rows = wl.rows_bits(r) if rows is None else rows
    q = wl.q_bits[r] if q is None else q
    return oracle.decode(rows, q, wl.model(r))


def compare(loaded, expected: dict, label: str = "") -> dict:
    """expected: request index -> (o [Hq, d_v], lse [Hq]) from the oracle."""
    num = den = 0.0
    max_abs = lse_abs = 0.0
    worst_head = 0.0
    for r, (o_ref, l_ref) in expected.items():
        o = oracle.bf16_bits_to_f64(loaded.out_bits(r))
        lse = loaded.lse_of(r)
        assert np.all(np.isfinite(o)) and np.all(np.isfinite(lse)), f"{label} request {r}: non-finite output"
        d = o - o_ref
        num += float((d * d).sum())
        den += float((o_ref * o_ref).sum())
        max_abs = max(max_abs, float(np.abs(d).max()))
        lse_abs = max(lse_abs, float(np.abs(lse - l_ref).max()))
        per_head = np.sqrt((d * d).sum(axis=1) / np.maximum((o_ref * o_ref).sum(axis=1), 1e-30))
        worst_head = max(worst_head, float(per_head.max()))
    rel = float(np.sqrt(num / max(den, 1e-30)))
    stats = dict(max_abs=max_abs, rel_l2=rel, lse_max_abs=lse_abs, worst_head_rel_l2=worst_head)
    print(f"[parity] {label} {stats}", flush=True)
    assert max_abs <= OUT_MAX_ABS, (label, stats)
    assert rel <= OUT_REL_L2, (label, stats)
    assert lse_abs <= LSE_MAX_ABS, (label, stats)
    return stats
