"""Loads a seeded workload into a device pool through the C ABI.

Plumbing shared by the GPU tests, smoke() and the bench: create the pool,
register the workload's models, open one request per batch entry, and append
every request's rows with cp_kv_append (optionally interleaved so pages of
different requests alternate physically). No attention arithmetic here.
"""
from __future__ import annotations

import dataclasses
from typing import Dict, List, Optional

import numpy as np

from .gen import MODELS, PAGE_TOKENS, Workload


@dataclasses.dataclass
class Loaded:
    pool: object  # crosspool.Pool
    workload: Workload
    model_ids: Dict[str, int]
    req_ids: List[int]
    q: object  # torch uint16-as-int16 device tensor, packed in batch order
    out: object
    lse: object
    fillers: List[int] = dataclasses.field(default_factory=list)

    def decode(self, **opts):
        self.pool.decode(self.req_ids, self.q, self.out, self.lse, **opts)

    def out_bits(self, r: int) -> np.ndarray:
        """bf16 bits of request r's output, [Hq, d_v]."""
        m = self.workload.model(r)
        off = sum(self.workload.model(i).n_q_heads * self.workload.model(i).d_v for i in range(r))
        n = m.n_q_heads * m.d_v
        return self.out[off:off + n].cpu().numpy().view(np.uint16).reshape(m.n_q_heads, m.d_v)

    def lse_of(self, r: int) -> np.ndarray:
        off = sum(self.workload.model(i).n_q_heads for i in range(r))
        return self.lse[off:off + self.workload.model(r).n_q_heads].cpu().numpy().astype(np.float64)

    def close(self):
        import torch

        torch.cuda.synchronize()  # no queued kernel may still read the pages
        for r in self.req_ids + self.fillers:
            self.pool.close(r)
        self.pool.destroy()


def to_device_u16(arr: np.ndarray, device):
    import torch

    return torch.from_numpy(np.ascontiguousarray(arr).view(np.int16)).to(device)


def load(wl: Workload, device: int = 0, *, placement_seed: Optional[int] = None, reserve_extra: int = 0,
         interleave: int = 0, rows_override: Optional[Dict[int, np.ndarray]] = None,
         q_override: Optional[List[np.ndarray]] = None, chunk_rows: int = 1 << 17, backing: int = 0,
         n_layers: int = 1, device_pages: int = 0, page_tokens: int = PAGE_TOKENS) -> Loaded:
    """Build a pool holding the workload.

    interleave > 0 appends rows in rounds of `interleave` tokens per request,
    so physical pages of different requests alternate. rows_override maps a
    request index to its rows (uint16 bits) instead of the seeded draw.
    backing selects the pool's memory (0 one buffer, 1 virtual ranges).
    n_layers > 1 registers the models with that many KV planes, each holding
    the same rows. device_pages = 1 gives the models device free-page stacks
    (decode steps take new pages on the device). page_tokens sets the pool's
    page size (tokens per page).
    """
    import torch

    from paper_2606_24506_amd import crosspool as cpl

    dev = torch.device("cuda", device)
    seed = wl.placement_seed if placement_seed is None else placement_seed
    pool = cpl.Pool(page_tokens=page_tokens, pool_bytes=wl.pool_bytes, chunk_bytes=wl.chunk_bytes,
                    placement_seed=seed, device=device, backing=backing, device_pages=device_pages)
    mids = {name: pool.register_spec(MODELS[name], n_layers=n_layers) for name in wl.models_used()}
    if wl.filler_model and wl.filler_model not in mids:
        mids[wl.filler_model] = pool.register_spec(MODELS[wl.filler_model], n_layers=n_layers)
    rids = [pool.open(mids[rq.model], rq.ctx_len + reserve_extra) for rq in wl.requests]

    # Filler requests occupy pool pages around the batch (their content is
    # never read); each holds at most 256 pages.
    fillers: List[int] = []
    fcap: List[int] = []
    left = wl.filler_pages
    while left > 0:
        take = min(256, left)
        fillers.append(pool.open(mids[wl.filler_model], take * page_tokens))
        fcap.append(take)
        left -= take
    filler_page = None
    if fillers:
        filler_page = torch.zeros((n_layers, page_tokens, MODELS[wl.filler_model].row_width), dtype=torch.int16,
                                  device=dev)

    def rows_of(r):
        if rows_override and r in rows_override:
            return rows_override[r]
        return wl.rows_bits(r)

    if interleave <= 0:
        for r, rid in enumerate(rids):
            rows = rows_of(r)
            for s in range(0, rows.shape[0], chunk_rows):
                part = rows[s:s + chunk_rows]
                blk = to_device_u16(np.tile(part.reshape(-1), n_layers), dev)  # [layers][tokens][row]
                pool.append([rid], [part.shape[0]], blk)
            torch.cuda.synchronize(dev)
        for f, cap in zip(fillers, fcap):
            for _ in range(cap):
                pool.append([f], [page_tokens], filler_page)
    else:
        all_rows = [rows_of(r) for r in range(len(rids))]
        pos = [0] * len(rids)
        fpos = [0] * len(fillers)
        while any(pos[r] < all_rows[r].shape[0] for r in range(len(rids))) or any(
                fpos[i] < fcap[i] for i in range(len(fillers))):
            ids, nn, blocks = [], [], []
            for r, rid in enumerate(rids):
                k = min(interleave, all_rows[r].shape[0] - pos[r])
                if k > 0:
                    ids.append(rid)
                    nn.append(k)
                    blocks.append(np.tile(all_rows[r][pos[r]:pos[r] + k].reshape(-1), n_layers))
                    pos[r] += k
            if ids:
                pool.append(ids, nn, to_device_u16(np.concatenate(blocks), dev))
            for i, f in enumerate(fillers):
                if fpos[i] < fcap[i]:
                    pool.append([f], [page_tokens], filler_page)
                    fpos[i] += 1
    torch.cuda.synchronize(dev)

    qs = q_override if q_override is not None else wl.q_bits
    q = to_device_u16(np.concatenate([x.reshape(-1) for x in qs]), dev)
    n_out = sum(MODELS[rq.model].n_q_heads * MODELS[rq.model].d_v for rq in wl.requests)
    n_lse = sum(MODELS[rq.model].n_q_heads for rq in wl.requests)
    out = torch.zeros(n_out, dtype=torch.int16, device=dev)
    lse = torch.zeros(n_lse, dtype=torch.float32, device=dev)
    return Loaded(pool, wl, mids, rids, q, out, lse, fillers)
