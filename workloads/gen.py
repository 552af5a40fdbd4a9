"""Seeded synthetic decode batches shaped like the paper's cold, bursty,
long-context workloads (Section 5.1 uses LongAlign and ShareGPT traces; those
datasets are not used here and these draws stand in for them).

Draw recipe, for ``make_workload(cfg, seed)`` with ``rng = default_rng(seed)``:
  1. model choice per request (mixed batch only): Zipf(s=1.2) over the three
     models in rank order MLA, MQA, GQA;
  2. context lengths: fixed lists, or log-uniform integers
     floor(exp(U(ln lo, ln hi))) clipped to [lo, hi];
  3. queries, request by request in batch order, fp32 normals -> bf16 (RNE);
  4. KV rows of request r from their own stream ``default_rng([seed, 1, r])``
     (fp32 normals times sigma -> bf16 RNE), so one request can be drawn
     without drawing the others.
Rows appended by decode step ``t`` for request ``r`` come from
``default_rng([seed, 2, r, t])``.

Nothing here computes attention; only shapes, sizes and random numbers.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, List, Optional

import numpy as np

PAGE_TOKENS = 64
CHUNK_BYTES_DEFAULT = 2 << 20


@dataclasses.dataclass(frozen=True)
class ModelSpec:
    """KV geometry of one attention layer (bf16 storage)."""

    name: str
    kind: str  # "mla" or "gqa" (MQA is gqa with one KV head)
    n_q_heads: int
    n_kv_heads: int
    head_dim: int = 0  # gqa: K and V width per KV head
    latent_dim: int = 0  # mla: compressed latent width (V = first latent_dim of K)
    rope_dim: int = 0  # mla: decoupled rope width
    scale: float = 0.0

    @property
    def d_k(self) -> int:
        return self.latent_dim + self.rope_dim if self.kind == "mla" else self.head_dim

    @property
    def d_v(self) -> int:
        return self.latent_dim if self.kind == "mla" else self.head_dim

    @property
    def row_width(self) -> int:
        """Elements in one logical KV row (one token)."""
        if self.kind == "mla":
            return self.latent_dim + self.rope_dim
        return 2 * self.n_kv_heads * self.head_dim

    @property
    def kappa(self) -> int:
        """KV bytes per token."""
        return 2 * self.row_width


MODELS: Dict[str, ModelSpec] = {
    # DeepSeek-V2-Lite shaped MLA: 16 query heads on one latent head of 512 + 64.
    "mla16": ModelSpec("mla16", "mla", 16, 1, latent_dim=512, rope_dim=64, scale=1.0 / math.sqrt(192.0)),
    # DeepSeek-V3 shaped MLA: 128 query heads on one latent head.
    "mla128": ModelSpec("mla128", "mla", 128, 1, latent_dim=512, rope_dim=64, scale=1.0 / math.sqrt(192.0)),
    "mqa32": ModelSpec("mqa32", "gqa", 32, 1, head_dim=128, scale=1.0 / math.sqrt(128.0)),
    "gqa32x4": ModelSpec("gqa32x4", "gqa", 32, 4, head_dim=128, scale=1.0 / math.sqrt(128.0)),
    # Further geometries, used to exercise every kernel variant in tests.
    "mla32": ModelSpec("mla32", "mla", 32, 1, latent_dim=512, rope_dim=64, scale=1.0 / math.sqrt(192.0)),
    "mqa16": ModelSpec("mqa16", "gqa", 16, 1, head_dim=128, scale=1.0 / math.sqrt(128.0)),
    "gqa128x2": ModelSpec("gqa128x2", "gqa", 128, 2, head_dim=128, scale=1.0 / math.sqrt(128.0)),
    "mqa128": ModelSpec("mqa128", "gqa", 128, 1, head_dim=128, scale=1.0 / math.sqrt(128.0)),
    "gqa8x8d64": ModelSpec("gqa8x8d64", "gqa", 8, 8, head_dim=64, scale=1.0 / math.sqrt(64.0)),
    # Llama-style GQA with four query heads per KV head (the wavefront-reduction path).
    "gqa32x8": ModelSpec("gqa32x8", "gqa", 32, 8, head_dim=128, scale=1.0 / math.sqrt(128.0)),
    "gqa16x8": ModelSpec("gqa16x8", "gqa", 16, 8, head_dim=128, scale=1.0 / math.sqrt(128.0)),
    "gqa24x8": ModelSpec("gqa24x8", "gqa", 24, 8, head_dim=128, scale=1.0 / math.sqrt(128.0)),
    "gqa16x4d64": ModelSpec("gqa16x4d64", "gqa", 16, 4, head_dim=64, scale=1.0 / math.sqrt(64.0)),
}


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round finite float32 values to bfloat16 (round to nearest, ties to even); uint16 bits."""
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    bias = ((b >> 16) & 1) + np.uint32(0x7FFF)
    return ((b + bias) >> 16).astype(np.uint16)


def normal_bf16(rng: np.random.Generator, shape, sigma: float) -> np.ndarray:
    x = rng.standard_normal(shape, dtype=np.float32)
    if sigma != 1.0:
        x *= np.float32(sigma)
    return f32_to_bf16_bits(x)


def _log_uniform(rng: np.random.Generator, lo: int, hi: int, n: int) -> np.ndarray:
    x = np.floor(np.exp(rng.uniform(math.log(lo), math.log(hi), size=n))).astype(np.int64)
    return np.clip(x, lo, hi)


@dataclasses.dataclass
class RequestSpec:
    model: str
    ctx_len: int


@dataclasses.dataclass
class Workload:
    name: str
    seed: int
    requests: List[RequestSpec]
    q_bits: List[np.ndarray]  # per request uint16 [Hq, d_k]
    sigma_kv: float
    pool_bytes: int
    chunk_bytes: int
    placement_seed: int
    # extra pages occupied by filler requests of the given model (burst workload)
    filler_model: Optional[str] = None
    filler_pages: int = 0

    def model(self, r: int) -> ModelSpec:
        return MODELS[self.requests[r].model]

    def models_used(self) -> List[str]:
        seen: List[str] = []
        for rq in self.requests:
            if rq.model not in seen:
                seen.append(rq.model)
        return seen

    def rows_bits(self, r: int) -> np.ndarray:
        """Logical KV rows of request r, uint16 [ctx_len, row_width]."""
        m = self.model(r)
        rng = np.random.default_rng([self.seed, 1, r])
        return normal_bf16(rng, (self.requests[r].ctx_len, m.row_width), self.sigma_kv)

    def step_rows_bits(self, r: int, step: int, n_new: int = 1) -> np.ndarray:
        """Rows appended to request r at decode step `step`."""
        m = self.model(r)
        rng = np.random.default_rng([self.seed, 2, r, step])
        return normal_bf16(rng, (n_new, m.row_width), self.sigma_kv)

    @property
    def total_tokens(self) -> int:
        return int(sum(rq.ctx_len for rq in self.requests))


def algorithmic_bytes(specs, ctx_lens) -> int:
    """Bytes a decode call must move at least once: each request's KV, its
    query, output and log-sum-exp, and one 4-byte page-table entry per page."""
    total = 0
    for m, n in zip(specs, ctx_lens):
        total += n * m.kappa + m.n_q_heads * (2 * m.d_k + 2 * m.d_v + 4) + 4 * (-(-n // PAGE_TOKENS))
    return int(total)


def _draw_queries(rng, models: List[str], sigma_q: float) -> List[np.ndarray]:
    out = []
    for name in models:
        m = MODELS[name]
        out.append(normal_bf16(rng, (m.n_q_heads, m.d_k), sigma_q))
    return out


def make_workload(cfg: int, seed: Optional[int] = None, *, scale_ctx: float = 1.0) -> Workload:
    """Build one of the five decode workloads.

    cfg 1: tiny MLA-16, 4 requests {128, 256, 384, 512}, 64-page pool, one page per chunk.
    cfg 2: MLA-16, 32 requests log-uniform in [1K, 32K], 2 GiB pool.
    cfg 3: MLA-128, 8 requests of 128K, 2 GiB pool.
    cfg 4: mixed MLA-16 / MQA-32 / GQA-32x4, 48 requests, Zipf(1.2), log-uniform [512, 64K], 8 GiB pool.
    cfg 5: MLA-128, 1 request of 512K in a 2 GiB pool filled to 90% by fillers.

    ``scale_ctx`` < 1 shrinks every context length (for tests that need the
    same shape mix at oracle-friendly sizes); it never changes the draw order.
    """
    if seed is None:
        seed = cfg
    rng = np.random.default_rng(seed)
    sigma_q, sigma_kv = 1.0, math.sqrt(0.5)

    def scaled(lens):
        return [max(1, int(round(n * scale_ctx))) for n in lens]

    if cfg == 1:
        sigma_kv = 1.0
        models = ["mla16"] * 4
        lens = scaled([128, 256, 384, 512])
        pool_bytes, chunk = 64 * 73_728, 73_728
    elif cfg == 2:
        models = ["mla16"] * 32
        lens = scaled(_log_uniform(rng, 1024, 32768, 32).tolist())
        pool_bytes, chunk = 2 << 30, CHUNK_BYTES_DEFAULT
    elif cfg == 3:
        models = ["mla128"] * 8
        lens = scaled([131072] * 8)
        pool_bytes, chunk = 2 << 30, CHUNK_BYTES_DEFAULT
    elif cfg == 4:
        names = ["mla16", "mqa32", "gqa32x4"]
        p = np.arange(1, 4, dtype=np.float64) ** -1.2
        p /= p.sum()
        choice = rng.choice(3, size=48, p=p)
        models = [names[c] for c in choice]
        lens = scaled(_log_uniform(rng, 512, 65536, 48).tolist())
        pool_bytes, chunk = 8 << 30, CHUNK_BYTES_DEFAULT
    elif cfg == 5:
        models = ["mla128"]
        lens = scaled([524288])
        pool_bytes, chunk = 2 << 30, CHUNK_BYTES_DEFAULT
    else:
        raise ValueError(f"unknown workload {cfg}")

    qs = _draw_queries(rng, models, sigma_q)
    wl = Workload(
        name=f"cfg{cfg}",
        seed=seed,
        requests=[RequestSpec(m, int(n)) for m, n in zip(models, lens)],
        q_bits=qs,
        sigma_kv=sigma_kv,
        pool_bytes=pool_bytes,
        chunk_bytes=chunk,
        placement_seed=seed,
    )
    if cfg == 5:
        m = MODELS["mla128"]
        page_bytes = PAGE_TOKENS * m.kappa
        slots = (pool_bytes // chunk) * (chunk // page_bytes)
        burst_pages = -(-lens[0] // PAGE_TOKENS)
        wl.filler_model = "mla128"
        wl.filler_pages = max(0, int(slots * 0.9) - burst_pages)
    return wl
