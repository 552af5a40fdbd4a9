"""Plain fp64 CPU oracle for decode attention over a shared, paged KV pool.

TEST INFRASTRUCTURE ONLY: tests/, __graft_entry__.smoke() and the CPU
baseline leg of bench.py may import this module. The HIP product path never
imports, links or calls it, and this module imports nothing from the product.

What it computes. The paper keeps attention next to the KV cache and lets
the existing paged attention kernels run over a *logical* KV address space,
while the virtualizer decides where physical pages live (Section 3.1, KV-cache
planner and virtualizer; Section 4, KV-cache virtualization). So the result
of a decode call must equal ordinary softmax attention of one query token over
the request's logically contiguous KV rows, whatever the page placement. The
attention families that share the pool are GQA, MQA and MLA (Section 1 and
Section 2.2). This module writes that definition out directly, in float64,
over contiguous rows; it never sees pages.

Readings taken where the paper is silent:
  * MLA caches one latent head per token, [latent | rope]; K is the whole
    row, V is its first ``latent_dim`` entries; the query arrives already
    absorbed (its no-rope part multiplied through W_UK) and post-rope.
  * GQA groups are contiguous: query head h reads KV head h // (Hq / Hkv).
  * lse is the natural log of the sum of exp(scaled score).

Inputs are bf16 bit patterns (uint16) or float arrays; bf16 is widened to
float64 exactly.
"""
from __future__ import annotations

from typing import List, Sequence, Tuple

import numpy as np


def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    """Exact widening of bfloat16 bit patterns (uint16) to float64."""
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16
    return b.view(np.float32).astype(np.float64)


def _as_f64(x: np.ndarray) -> np.ndarray:
    x = np.asarray(x)
    if x.dtype == np.uint16:
        return bf16_bits_to_f64(x)
    return x.astype(np.float64)


def kv_views(rows: np.ndarray, geom) -> Tuple[np.ndarray, np.ndarray]:
    """Split logical rows [n, row_width] into per-KV-head K [Hkv, n, d_k] and
    V [Hkv, n, d_v].

    MLA: one latent head; K_j = row_j (latent and rope), V_j = row_j[:latent].
    GQA/MQA: row_j = [K head 0 .. K head Hkv-1 | V head 0 .. V head Hkv-1].
    """
    rows = _as_f64(rows)
    n = rows.shape[0]
    if geom.kind == "mla":
        k = rows[None, :, : geom.latent_dim + geom.rope_dim]
        v = rows[None, :, : geom.latent_dim]
        return k, v
    hkv, d = geom.n_kv_heads, geom.head_dim
    k = rows[:, : hkv * d].reshape(n, hkv, d).transpose(1, 0, 2)
    v = rows[:, hkv * d : 2 * hkv * d].reshape(n, hkv, d).transpose(1, 0, 2)
    return k, v


def decode(rows: np.ndarray, q: np.ndarray, geom, scale: float = None) -> Tuple[np.ndarray, np.ndarray]:
    """One query token per head attending over all ``n`` rows.

    For query head h with KV head kv = h // g (g = Hq / Hkv):
        s_j = scale * <q_h, K_j>            j = 0 .. n-1
        m   = max_j s_j,  w_j = exp(s_j - m),  l = sum_j w_j
        o_h = (sum_j w_j V_j) / l,   lse_h = m + ln l
    Returns (o [Hq, d_v], lse [Hq]) in float64. ``n`` must be at least 1:
    softmax over an empty set is undefined.
    """
    q = _as_f64(q)
    k, v = kv_views(rows, geom)
    n = k.shape[1]
    if n < 1:
        raise ValueError("decode needs at least one KV row")
    if scale is None:
        scale = geom.scale
    hq, hkv = geom.n_q_heads, geom.n_kv_heads
    g = hq // hkv
    o = np.empty((hq, v.shape[2]), dtype=np.float64)
    lse = np.empty(hq, dtype=np.float64)
    for kv in range(hkv):
        qg = q[kv * g : (kv + 1) * g]  # [g, d_k]
        s = scale * (k[kv] @ qg.T)  # [n, g]
        m = s.max(axis=0)
        w = np.exp(s - m)
        l = w.sum(axis=0)
        o[kv * g : (kv + 1) * g] = (w.T @ v[kv]) / l[:, None]
        lse[kv * g : (kv + 1) * g] = m + np.log(l)
    return o, lse


def merge(parts: Sequence[Tuple[np.ndarray, np.ndarray]]) -> Tuple[np.ndarray, np.ndarray]:
    """Combine partial results of disjoint KV ranges, in the given order.

    Each part is (o_c [H, d_v], lse_c [H]) with o_c already normalised over
    its own range. With M = max_c lse_c:
        lse = M + ln sum_c exp(lse_c - M)
        o   = sum_c exp(lse_c - lse) * o_c
    """
    lse_c = np.stack([np.asarray(p[1], dtype=np.float64) for p in parts])  # [S, H]
    o_c = np.stack([np.asarray(p[0], dtype=np.float64) for p in parts])  # [S, H, d]
    big = lse_c.max(axis=0)
    lse = big + np.log(np.exp(lse_c - big).sum(axis=0))
    wts = np.exp(lse_c - lse)  # [S, H]
    o = (wts[:, :, None] * o_c).sum(axis=0)
    return o, lse


def decode_split(rows: np.ndarray, q: np.ndarray, geom, bounds: Sequence[int], scale: float = None):
    """Decode each contiguous range [bounds[i], bounds[i+1]) on its own, then
    merge. ``bounds`` starts at 0, ends at n and is strictly increasing."""
    parts = [decode(rows[a:b], q, geom, scale) for a, b in zip(bounds[:-1], bounds[1:])]
    return merge(parts)


def gather_rows(appends: Sequence[np.ndarray]) -> np.ndarray:
    """Logical contents of a request after appending row blocks in order:
    their concatenation. A device-side gather must return exactly this."""
    return np.concatenate([np.asarray(a) for a in appends], axis=0)


def mla_absorb_query(q_nope: np.ndarray, q_rope: np.ndarray, w_uk: np.ndarray) -> np.ndarray:
    """Absorbed MLA query per head: [W_UK[h]^T q_nope[h] ; q_rope[h]].

    q_nope [H, d_h], q_rope [H, d_r], w_uk [H, d_h, d_c] -> [H, d_c + d_r].
    """
    q_nope = _as_f64(q_nope)
    q_rope = _as_f64(q_rope)
    w_uk = _as_f64(w_uk)
    lat = np.einsum("hdc,hd->hc", w_uk, q_nope)
    return np.concatenate([lat, q_rope], axis=1)


def mla_explicit(c, k_rope, q_nope, q_rope, w_uk, w_uv, scale: float) -> np.ndarray:
    """Non-absorbed MLA attention, up-projecting the cache per head.

    c [n, d_c] latent cache, k_rope [n, d_r], q_nope [H, d_h], q_rope [H, d_r],
    w_uk [H, d_h, d_c], w_uv [H, d_v, d_c]. Per head h:
        k_j = [W_UK[h] c_j ; k_rope_j],  v_j = W_UV[h] c_j
        o_h = softmax_j(scale <[q_nope_h ; q_rope_h], k_j>) . v_j
    Returns o [H, d_v].
    """
    c, k_rope = _as_f64(c), _as_f64(k_rope)
    q_nope, q_rope = _as_f64(q_nope), _as_f64(q_rope)
    w_uk, w_uv = _as_f64(w_uk), _as_f64(w_uv)
    H = q_nope.shape[0]
    out: List[np.ndarray] = []
    for h in range(H):
        kh = np.concatenate([c @ w_uk[h].T, k_rope], axis=1)  # [n, d_h + d_r]
        vh = c @ w_uv[h].T  # [n, d_v]
        qh = np.concatenate([q_nope[h], q_rope[h]])
        s = scale * (kh @ qh)
        w = np.exp(s - s.max())
        out.append((w @ vh) / w.sum())
    return np.stack(out)
