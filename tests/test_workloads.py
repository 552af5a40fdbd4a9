"""The seeded generators reproduce the documented workload shapes and sizes."""
import json
import os

import numpy as np
import torch

from workloads import MODELS, algorithmic_bytes, f32_to_bf16_bits, make_workload

GOLDEN = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "workload_totals.json")))


def test_totals_match_golden():
    for cfg in range(1, 6):
        wl = make_workload(cfg)
        g = GOLDEN[f"cfg{cfg}"]
        lens = [r.ctx_len for r in wl.requests]
        assert sum(lens) == g["tokens"]
        assert sum(-(-n // 64) for n in lens) == g["pages"]
        assert sum(n * wl.model(i).kappa for i, n in enumerate(lens)) == g["kv_bytes"]
        if "max" in g:
            assert max(lens) == g["max"]
        if "min" in g:
            assert min(lens) == g["min"]
        if "per_model_requests" in g:
            for name, cnt in g["per_model_requests"].items():
                assert sum(r.model == name for r in wl.requests) == cnt
    wl5 = make_workload(5)
    assert wl5.filler_pages + 8192 == GOLDEN["cfg5"]["filled_slots"]


def test_geometry():
    assert MODELS["mla16"].kappa == 1152 and MODELS["mla128"].kappa == 1152
    assert MODELS["mqa32"].kappa == 512 and MODELS["gqa32x4"].kappa == 2048
    assert MODELS["mla16"].d_k == 576 and MODELS["mla16"].d_v == 512


def test_algorithmic_bytes_tiny():
    wl = make_workload(1)
    m = MODELS["mla16"]
    lens = [128, 256, 384, 512]
    expect = 1474560 + 4 * 16 * (576 * 2 + 512 * 2 + 4) + 4 * 20
    assert algorithmic_bytes([m] * 4, lens) == expect
    assert [r.ctx_len for r in wl.requests] == lens


def test_bf16_rounding_matches_torch():
    rng = np.random.default_rng(0)
    x = (rng.standard_normal(100000) * np.exp(rng.uniform(-20, 20, 100000))).astype(np.float32)
    # include exact ties between two bf16 neighbours
    x[:4] = np.array([1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -(1.0 + 2 ** -8), 2.0 ** -130], dtype=np.float32)
    ours = f32_to_bf16_bits(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, ref)


def test_draws_are_reproducible_and_independent_per_request():
    a = make_workload(2)
    b = make_workload(2)
    assert all(np.array_equal(x, y) for x, y in zip(a.q_bits, b.q_bits))
    # drawing request 5 alone gives the same rows as drawing after request 4
    r4 = a.rows_bits(4)
    r5a = a.rows_bits(5)
    r5b = b.rows_bits(5)
    assert np.array_equal(r5a, r5b) and r4.shape[1] == 576
    assert a.q_bits[0].shape == (16, 576)
