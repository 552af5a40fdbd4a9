"""Pins that tie the fp64 oracle to facts outside itself.

Each pin is a closed form, an invariant of softmax attention, or a library
routine that computes the same special case, chosen so that a plausible slip
in the oracle (a dropped term, a wrong sign, a wrong head index, a transposed
operand, a wrong V slice, a wrong scale) fails at least one of them. The
last test plants such slips in copies of the oracle and checks exactly that.
"""
import math

import numpy as np
import pytest
import torch

import oracle
from oracle import attention as oa
from workloads import MODELS, ModelSpec


def tiny_mla(h=4, lat=16, rope=8, scale=None):
    return ModelSpec("t_mla", "mla", h, 1, latent_dim=lat, rope_dim=rope,
                     scale=scale if scale is not None else 1.0 / math.sqrt(12.0))


def tiny_gqa(hq=8, hkv=2, d=16):
    return ModelSpec("t_gqa", "gqa", hq, hkv, head_dim=d, scale=1.0 / math.sqrt(d))


GEOMS = [tiny_mla(), tiny_gqa(), tiny_gqa(8, 1, 16), tiny_gqa(4, 4, 8), MODELS["mla16"], MODELS["gqa32x4"]]


def rand_case(geom, n, seed):
    rng = np.random.default_rng(seed)
    rows = rng.standard_normal((n, geom.row_width))
    q = rng.standard_normal((geom.n_q_heads, geom.d_k))
    return rows, q


def v_of(rows, geom):
    """V rows per KV head, built from the layout description (not from kv_views)."""
    if geom.kind == "mla":
        return [rows[:, : geom.latent_dim]]
    d, hkv = geom.head_dim, geom.n_kv_heads
    return [rows[:, hkv * d + i * d : hkv * d + (i + 1) * d] for i in range(hkv)]


def kv_index(geom, h):
    return h // (geom.n_q_heads // geom.n_kv_heads)


# ---------------------------------------------------------------- pins ----

def pin_single_token(decode, geom):
    """n = 1: the softmax weight is exactly 1, so o = V_0 and lse = s_0.
    The score is built so its value is known in closed form: K_0 has one
    nonzero entry a at index i, q_h has b at index i, so s_0 = scale*a*b."""
    rng = np.random.default_rng(7)
    rows = rng.standard_normal((1, geom.row_width))
    q = np.zeros((geom.n_q_heads, geom.d_k))
    a, b = 1.5, -2.25
    if geom.kind == "mla":
        rows[0, : geom.d_k] = 0.0
        rows[0, 3] = a  # V = first latent entries, so V_0 = a * e_3
        q[:, 3] = b
    else:
        d = geom.head_dim
        for kv in range(geom.n_kv_heads):
            rows[0, kv * d : (kv + 1) * d] = 0.0
            rows[0, kv * d + 5] = a
        q[:, 5] = b
    o, lse = decode(rows, q, geom)
    vs = v_of(rows, geom)
    for h in range(geom.n_q_heads):
        assert np.array_equal(o[h], vs[kv_index(geom, h)][0]), "n=1 must return V_0 exactly"
    assert np.allclose(lse, geom.scale * a * b, rtol=0, atol=1e-14)


def pin_uniform(decode, geom):
    """q = 0: every score is 0, so o = mean_j V_j and lse = ln n."""
    n = 37
    rows, _ = rand_case(geom, n, 11)
    q = np.zeros((geom.n_q_heads, geom.d_k))
    o, lse = decode(rows, q, geom)
    vs = v_of(rows, geom)
    for h in range(geom.n_q_heads):
        assert np.allclose(o[h], vs[kv_index(geom, h)].mean(axis=0), rtol=0, atol=1e-13)
    assert np.allclose(lse, math.log(n), rtol=0, atol=1e-13)


def pin_two_tokens(decode, geom):
    """n = 2 with scores known in closed form: s_0 = scale*a*x, s_1 = scale*c*y.
    Then lse = logaddexp(s_0, s_1) and o = expit(s_0 - s_1) V_0 + expit(s_1 - s_0) V_1."""
    from scipy.special import expit

    rng = np.random.default_rng(5)
    rows = rng.standard_normal((2, geom.row_width))
    q = np.zeros((geom.n_q_heads, geom.d_k))
    a, c = 0.75, -1.25
    if geom.kind == "mla":
        rows[0, : geom.d_k] = 0.0
        rows[1, : geom.d_k] = 0.0
        rows[0, 1] = a
        rows[1, 2] = c
        i0, i1 = 1, 2
    else:
        d = geom.head_dim
        for kv in range(geom.n_kv_heads):
            rows[:, kv * d : (kv + 1) * d] = 0.0
            rows[0, kv * d + 1] = a
            rows[1, kv * d + 2] = c
        i0, i1 = 1, 2
    xs = np.linspace(-2.0, 3.0, geom.n_q_heads)
    ys = np.linspace(1.5, -2.5, geom.n_q_heads)
    q[:, i0] = xs
    q[:, i1] = ys
    o, lse = decode(rows, q, geom)
    vs = v_of(rows, geom)
    s0, s1 = geom.scale * a * xs, geom.scale * c * ys
    assert np.allclose(lse, np.logaddexp(s0, s1), rtol=0, atol=1e-13)
    for h in range(geom.n_q_heads):
        v = vs[kv_index(geom, h)]
        ref = expit(s0[h] - s1[h]) * v[0] + expit(s1[h] - s0[h]) * v[1]
        assert np.allclose(o[h], ref, rtol=0, atol=1e-13)


def pin_sdpa(decode, geom):
    """Library special case: torch's scaled_dot_product_attention in float64
    on the CPU (GQA grouping through enable_gqa; MLA as one KV head with
    K = whole row, V = its latent part)."""
    n = 53
    rows, q = rand_case(geom, n, 13)
    o, _ = decode(rows, q, geom)
    r = torch.from_numpy(rows)
    if geom.kind == "mla":
        k = r[:, : geom.d_k][None, None]  # [1, 1, n, d_k]
        v = r[:, : geom.latent_dim][None, None]
    else:
        d, hkv = geom.head_dim, geom.n_kv_heads
        k = r[:, : hkv * d].reshape(n, hkv, d).permute(1, 0, 2)[None].contiguous()
        v = r[:, hkv * d :].reshape(n, hkv, d).permute(1, 0, 2)[None].contiguous()
    qt = torch.from_numpy(q)[None, :, None, :]  # [1, Hq, 1, d_k]
    ref = torch.nn.functional.scaled_dot_product_attention(
        qt, k, v, scale=geom.scale, enable_gqa=geom.n_q_heads != k.shape[1])
    assert np.allclose(o, ref[0, :, 0].numpy(), rtol=0, atol=1e-12)


def pin_dominant(decode, geom):
    """One score far above the rest: o -> V_t and lse -> s_t."""
    n = 29
    rows, _ = rand_case(geom, n, 17)
    rows *= 0.01
    t = 19
    q = np.zeros((geom.n_q_heads, geom.d_k))
    if geom.kind == "mla":
        rows[t, 0] = 1.0
        q[:, 0] = 4000.0
    else:
        d = geom.head_dim
        for kv in range(geom.n_kv_heads):
            rows[t, kv * d] = 1.0
        q[:, 0] = 4000.0
    o, lse = decode(rows, q, geom)
    vs = v_of(rows, geom)
    for h in range(geom.n_q_heads):
        assert np.allclose(o[h], vs[kv_index(geom, h)][t], rtol=0, atol=1e-9)
    assert np.allclose(lse, geom.scale * 4000.0, rtol=1e-3)


def pin_row_permutation(decode, geom):
    """Attention over a set of rows does not depend on their order."""
    rows, q = rand_case(geom, 41, 19)
    perm = np.random.default_rng(3).permutation(41)
    o1, l1 = decode(rows, q, geom)
    o2, l2 = decode(rows[perm], q, geom)
    assert np.allclose(o1, o2, rtol=0, atol=1e-12) and np.allclose(l1, l2, rtol=0, atol=1e-12)


PINS = [pin_single_token, pin_uniform, pin_two_tokens, pin_sdpa, pin_dominant, pin_row_permutation]


@pytest.mark.parametrize("geom", GEOMS, ids=lambda g: f"{g.kind}{g.n_q_heads}x{g.n_kv_heads}")
@pytest.mark.parametrize("pin", PINS, ids=lambda p: p.__name__)
def test_oracle_pin(pin, geom):
    pin(oracle.decode, geom)


# ------------------------------------------------------ merge pins ----

@pytest.mark.parametrize("geom", GEOMS[:4], ids=lambda g: f"{g.kind}{g.n_q_heads}x{g.n_kv_heads}")
def test_split_merge_equals_unsplit(geom):
    n = 300
    rows, q = rand_case(geom, n, 23)
    o, lse = oracle.decode(rows, q, geom)
    rng = np.random.default_rng(29)
    for _ in range(6):
        k = int(rng.integers(1, 12))
        cuts = np.sort(rng.choice(np.arange(1, n), size=k, replace=False))
        bounds = [0, *cuts.tolist(), n]
        o2, l2 = oracle.decode_split(rows, q, geom, bounds)
        assert np.allclose(o, o2, rtol=0, atol=1e-12)
        assert np.allclose(lse, l2, rtol=0, atol=1e-12)


def test_merge_associative_and_single():
    geom = tiny_gqa()
    rows, q = rand_case(geom, 90, 31)
    a = oracle.decode(rows[:20], q, geom)
    b = oracle.decode(rows[20:55], q, geom)
    c = oracle.decode(rows[55:], q, geom)
    left = oracle.merge([oracle.merge([a, b]), c])
    right = oracle.merge([a, oracle.merge([b, c])])
    assert np.allclose(left[0], right[0], atol=1e-13) and np.allclose(left[1], right[1], atol=1e-13)
    one = oracle.merge([a])
    assert np.allclose(one[0], a[0], atol=1e-15) and np.allclose(one[1], a[1], atol=1e-15)


def test_merge_closed_form_two_equal_parts():
    """Two parts with equal lse and outputs o1, o2: lse grows by ln 2 and o is their mean."""
    o1 = np.array([[1.0, -2.0]])
    o2 = np.array([[3.0, 4.0]])
    lse = np.array([0.7])
    o, l = oracle.merge([(o1, lse), (o2, lse)])
    assert np.allclose(o, [[2.0, 1.0]], atol=1e-15)
    assert np.allclose(l, 0.7 + math.log(2.0), atol=1e-15)


# ---------------------------------------------------- MLA absorption ----

@pytest.mark.parametrize("dc,dr,dh,H,n", [(8, 4, 4, 1, 1), (16, 8, 8, 3, 5), (16, 4, 8, 2, 17), (8, 8, 4, 3, 17)])
def test_mla_absorbed_equals_explicit(dc, dr, dh, H, n):
    """Multiplying the no-rope query through W_UK and decoding over the latent
    cache, then projecting with W_UV, equals attention with K and V
    up-projected per head: <q_nope, W_UK c> = <W_UK^T q_nope, c> and
    sum_j w_j W_UV c_j = W_UV sum_j w_j c_j."""
    rng = np.random.default_rng(dc * 1000 + dr * 100 + n)
    c = rng.standard_normal((n, dc))
    kr = rng.standard_normal((n, dr))
    qn = rng.standard_normal((H, dh))
    qr = rng.standard_normal((H, dr))
    wuk = rng.standard_normal((H, dh, dc))
    wuv = rng.standard_normal((H, dh + 1, dc))
    scale = 1.0 / math.sqrt(dh + dr)
    explicit = oracle.mla_explicit(c, kr, qn, qr, wuk, wuv, scale)
    geom = ModelSpec("tiny", "mla", H, 1, latent_dim=dc, rope_dim=dr, scale=scale)
    qabs = oracle.mla_absorb_query(qn, qr, wuk)
    o_lat, _ = oracle.decode(np.concatenate([c, kr], axis=1), qabs, geom)
    absorbed = np.einsum("hvc,hc->hv", wuv, o_lat)
    assert np.allclose(explicit, absorbed, rtol=0, atol=1e-10)


def test_gqa_group_one_is_mha_and_mqa_is_one_kv_head():
    """Hq = Hkv is per-head attention; Hkv = 1 shares one K/V across heads."""
    mha = tiny_gqa(4, 4, 8)
    rows, q = rand_case(mha, 21, 37)
    o, _ = oracle.decode(rows, q, mha)
    d = 8
    for h in range(4):
        one = ModelSpec("one", "gqa", 1, 1, head_dim=d, scale=mha.scale)
        r1 = np.concatenate([rows[:, h * d : (h + 1) * d], rows[:, 4 * d + h * d : 4 * d + (h + 1) * d]], axis=1)
        o1, _ = oracle.decode(r1, q[h : h + 1], one)
        assert np.allclose(o[h], o1[0], atol=1e-14)
    mqa = tiny_gqa(4, 1, 8)
    rows, q = rand_case(mqa, 21, 41)
    o, _ = oracle.decode(rows, q, mqa)
    for h in range(4):
        one = ModelSpec("one", "gqa", 1, 1, head_dim=d, scale=mqa.scale)
        o1, _ = oracle.decode(rows, q[h : h + 1], one)
        assert np.allclose(o[h], o1[0], atol=1e-14)


def test_bf16_widening_is_exact():
    vals = torch.tensor([0.0, -0.0, 1.0, -2.5, 3.140625, 1e-30, -6.5e30], dtype=torch.bfloat16)
    bits = vals.view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(oracle.bf16_bits_to_f64(bits), vals.to(torch.float64).numpy())


# ------------------------------------------------- planted mistakes ----

def _mut_scale(rows, q, geom, scale=None):
    return oa.decode(rows, q, geom, scale=1.0 / math.sqrt(geom.d_k))


def _mut_head_map(rows, q, geom, scale=None):
    # interleaved instead of contiguous groups: q head h -> KV head h % Hkv
    hq, hkv = geom.n_q_heads, geom.n_kv_heads
    perm = np.array([(h % hkv) * (hq // hkv) + h // hkv for h in range(hq)])
    o, lse = oa.decode(rows, np.asarray(q)[np.argsort(perm)], geom, scale)
    return o[perm], lse[perm]


def _mut_vslice(rows, q, geom, scale=None):
    if geom.kind != "mla":
        # V taken from the K half
        k, _ = oa.kv_views(rows, geom)
        rr = np.asarray(rows, dtype=np.float64).copy()
        d, hkv = geom.head_dim, geom.n_kv_heads
        rr[:, hkv * d :] = rr[:, : hkv * d]
        return oa.decode(rr, q, geom, scale)
    rr = np.asarray(rows, dtype=np.float64).copy()
    rr[:, : geom.latent_dim] = np.roll(rr[:, : geom.d_k], -geom.rope_dim, axis=1)[:, : geom.latent_dim]
    o, lse = oa.decode(rows, q, geom, scale)
    o2, _ = oa.decode(rr, q, geom, scale)
    return o2, lse


def _mut_no_max_in_lse(rows, q, geom, scale=None):
    o, lse = oa.decode(rows, q, geom, scale)
    k, _ = oa.kv_views(rows, geom)
    g = geom.n_q_heads // geom.n_kv_heads
    qq = np.asarray(q, dtype=np.float64)
    sc = geom.scale if scale is None else scale
    for h in range(geom.n_q_heads):
        s = sc * (k[h // g] @ qq[h])
        lse[h] = np.log(np.exp(s - s.max()).sum())
    return o, lse


def _mut_log2(rows, q, geom, scale=None):
    o, lse = oa.decode(rows, q, geom, scale)
    return o, lse / math.log(2.0)


def _mut_unnormalised(rows, q, geom, scale=None):
    o, lse = oa.decode(rows, q, geom, scale)
    k, _ = oa.kv_views(rows, geom)
    n = k.shape[1]
    return o * n, lse


MUTANTS = [_mut_scale, _mut_head_map, _mut_vslice, _mut_no_max_in_lse, _mut_log2, _mut_unnormalised]


@pytest.mark.parametrize("mutant", MUTANTS, ids=lambda m: m.__name__)
def test_pins_catch_planted_mistakes(mutant):
    """Every planted slip must fail at least one pin on at least one geometry
    (head mapping only matters with more than one KV head)."""
    caught = False
    for geom in [tiny_mla(), tiny_gqa(8, 2, 16)]:
        for pin in PINS:
            try:
                pin(mutant, geom)
            except AssertionError:
                caught = True
    assert caught, f"no pin catches {mutant.__name__}"
