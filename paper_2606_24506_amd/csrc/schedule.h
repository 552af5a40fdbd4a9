// Work distribution shared by the decode kernels. A decode launch covers
// several requests (possibly of different models); `seg(rq, sg)` runs one
// piece of work: pages [sg.pg_begin, sg.pg_end) of request rq for KV head
// (or head block) sg.hblk, writing partial slot sg.slot when the request is
// split.
#pragma once

#include <hip/hip_runtime.h>

#include "device_common.h"
#include "kargs.h"

namespace cp {

// Finds the next piece of work of this workgroup for the balanced
// schedule: head block *hb or a later one of request *r, or the first head
// block of a later request, whose pages meet the workgroup's share
// [L0, L1) of the cost line (page j of a request sits at its cost position
// plus j times its model's page cost). Lane i evaluates request i: one
// round of loads from the argument segment (the models' page sizes and
// costs are uniform loads) and one ballot, so that the first piece of a
// launch starts after a single round trip. All arithmetic fits 32 bits:
// the host keeps the cost line below 2^32 and the grid below 2^16.
// Returns false when the workgroup's share is exhausted.
__device__ __forceinline__ bool next_balanced(const DecodeArgs &a, int *r, uint32_t *hb, Seg *sg) {
  const uint32_t W = gridDim.x, w = blockIdx.x, T = a.total_cost;
  const uint32_t q = T / W, rm = T % W;  // floor(w T / W) = w q + floor(w rm / W), and w rm < 2^32
  const uint32_t L0 = w * q + w * rm / W, L1 = (w + 1) * q + (w + 1) * rm / W;
  const int i = threadIdx.x & 63;
  const DecReq &ri = a.req[i < a.n_req ? i : 0];
  const uint32_t C = ri.unit_begin, model = ri.model, nh = ri.n_hblk;
  uint32_t P = (uint32_t)a.geom[0].page_tokens, c = (uint32_t)a.geom[0].page_cost;
#pragma unroll
  for (int m = 1; m < kMaxLaunchModels; ++m)
    if (model == (uint32_t)m) {
      P = (uint32_t)a.geom[m].page_tokens;
      c = (uint32_t)a.geom[m].page_cost;
    }
  const uint32_t pages = (ri.ctx_len + P - 1) / P;
  const uint32_t jb = L0 > C ? (L0 - C + c - 1) / c : 0u;
  const uint32_t je = C < L1 ? min(pages, (L1 - C + c - 1) / c) : 0u;
  const bool ok = i < a.n_req && i >= *r && jb < je && (i > *r || *hb < nh);
  const uint64_t b = __builtin_amdgcn_ballot_w64(ok);
  if (b == 0) return false;
  const int k = __builtin_ctzll(b);
  if (k != *r) {
    *r = k;
    *hb = 0;
  }
  sg->pg_begin = __builtin_amdgcn_readlane(jb, k);
  sg->pg_end = __builtin_amdgcn_readlane(je, k);
  sg->slot = w - __builtin_amdgcn_readlane((uint32_t)ri.chunk_pages, k);
  sg->hblk = *hb;
  sg->model = __builtin_amdgcn_readlane(model, k);
  return true;
}

// Decodes unit u of the queue and grid schedules into (request, piece).
__device__ __forceinline__ int unit_segment(const DecodeArgs &a, uint32_t u, Seg *sg) {
  const int r = sorted_search(a.n_req, u, [&](int i) { return a.req[i].unit_begin; });
  const DecReq &rq = a.req[r];
  const uint32_t local = u - rq.unit_begin;
  const uint32_t chunk = local / rq.n_hblk;
  const uint32_t pages = (rq.ctx_len + a.geom[rq.model].page_tokens - 1) / a.geom[rq.model].page_tokens;
  sg->pg_begin = chunk * rq.chunk_pages;
  sg->pg_end = min(pages, sg->pg_begin + rq.chunk_pages);
  sg->slot = chunk;
  sg->hblk = local % rq.n_hblk;
  sg->model = rq.model;
  return r;
}

// Device page stack (kAppPop; run by one thread): the first piece of this
// launch to reach request rq's new page (in any of its planes, when several
// layers of the request share the launch) claims the request's pop, takes
// one page per KV plane from the top of the model's stack and writes their
// page-table entries (plane l gets the entry l below the top); any other
// piece waits until the claimant has published them. The claimant waits on
// nothing, so every wait ends. Returns the entry of the new page of the
// plane rq attends over.
__device__ __forceinline__ uint32_t pop_new_pages(const DecodeArgs &a, const DecReq &rq, uint32_t pg) {
  const GeomK &g = a.geom[rq.model];
  const uint32_t rid = rq.app_pte;
  uint32_t *st = a.pop_state + rid;
  const uint32_t claim = a.epoch << 1, done = claim | 1u;
  uint32_t s = __hip_atomic_load(st, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_AGENT);
  if (s != done) {
    if (s != claim && atomicCAS(st, s, claim) == s) {
      const int32_t L = g.layers;
      const uint32_t base = a.req_geo[2 * rid], plane = a.req_geo[2 * rid + 1];
      const int32_t top = atomicSub(&a.stack_top[g.pool_model], L);
      const uint32_t *stk = a.stack + (uint64_t)g.pool_model * kStackCap;
      for (int32_t l = 0; l < L; ++l) a.pte[base + (uint32_t)l * plane + pg] = stk[top - 1 - l];
      __hip_atomic_store(st, done, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
    } else {
      while (__hip_atomic_load(st, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_AGENT) != done) __builtin_amdgcn_s_sleep(1);
    }
  }
  return __hip_atomic_load(a.pte + rq.pte_base + pg, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Fused append (cp_attn_decode_step): every piece whose page range holds a
// request's last context token, when that token is new in this call, first
// writes the page-table entry of a newly allocated page (taken from the
// launch arguments, or popped from the model's device stack) and copies
// the new logical row into its page; then the piece reads the page as
// usual. When several pieces (head blocks) cover that page they all write
// the same bytes, which is harmless; each one's own stores precede its
// loads through the workgroup barrier.
__device__ __forceinline__ void fused_append(const DecodeArgs &a, const DecReq &rq, const Seg &sg) {
  const GeomK &g = a.geom[sg.model];
  const uint32_t P = (uint32_t)g.page_tokens;
  const uint32_t pos = rq.ctx_len - 1, pg = pos / P;
  if (pg < sg.pg_begin || pg >= sg.pg_end) return;
  uint32_t pte;
  if (rq.app_flags & kAppPop) {
    __shared__ uint32_t popped;
    if (threadIdx.x == 0) popped = pop_new_pages(a, rq, pg);
    __syncthreads();
    pte = popped;
  } else if (rq.app_flags & kAppPage) {
    pte = rq.app_pte;
    if (threadIdx.x == 0) a.pte[rq.pte_base + pg] = pte;
  } else {
    pte = a.pte[rq.pte_base + pg];
  }
  uint8_t *page = a.pool + ((uint64_t)pte << 8);
  const uint4 *src = reinterpret_cast<const uint4 *>(a.rows + rq.app_off);
  const uint32_t nseg = (uint32_t)g.row_elems / 8;
  for (uint32_t sgi = threadIdx.x; sgi < nseg; sgi += blockDim.x)
    *reinterpret_cast<uint4 *>(page + row_seg_offset(g, pos % P, sgi)) = src[sgi];
  __syncthreads();
}

// Layer cursor of an all-layer launch (Section 3.2's per-batch layer
// cursor and completion state, driven by the launch itself; run by one
// thread after the piece's outputs or partials are written): the last of
// the pieces of launch entry r (one KV layer of one request) moves the
// request's cursor on by one layer; the one that completes the last layer
// sets it back to 0 and counts the token as carried through every layer.
__device__ __forceinline__ void piece_done(const DecodeArgs &a, int r) {
  const DecReq &rq = a.req[r];
  const uint32_t tag = a.ent_tag[r];
  __threadfence();
  const uint32_t pieces = (uint32_t)rq.n_chunks * rq.n_hblk;
  if (atomicAdd(&a.entry_done[r], 1u) + 1 != pieces) return;
  atomicExch(&a.entry_done[r], 0u);
  const uint32_t rid = tag & ((1u << kTagLayerShift) - 1), layers = tag >> kTagLayerShift;
  if (atomicAdd(&a.layer_cursor[2 * rid], 1u) + 1 == layers) {
    atomicExch(&a.layer_cursor[2 * rid], 0u);
    if (rq.app_flags & kAppRow) atomicAdd(&a.layer_tokens[2 * rid], 1u);
  }
}

// Work loop of every decode kernel; `seg` is inlined once. Queue schedule:
// workgroups pull unit indices from a device counter until the queue is
// empty; the last workgroup to leave resets the counters for the next
// launch.
template <class F>
__device__ __forceinline__ void decode_loop(const DecodeArgs &a, uint32_t *next, F &&seg) {
  int br = 0;        // balanced: request of the last piece
  uint32_t bhb = 0;  // balanced: next head block of that request
  bool first = true;
  for (;;) {
    Seg sg;
    int r;
    if (a.schedule == kSchedBalanced) {
      if (!next_balanced(a, &br, &bhb, &sg)) break;
      r = br;
      ++bhb;
    } else if (a.schedule == kSchedGrid) {
      if (!first) break;
      r = unit_segment(a, blockIdx.x, &sg);
    } else {
      if (threadIdx.x == 0) *next = atomicAdd(&a.queue[0], 1u);
      __syncthreads();
      const uint32_t u = *next;
      __syncthreads();
      if (u >= (uint32_t)a.n_units) break;
      r = unit_segment(a, u, &sg);
    }
    first = false;
    if (a.req[r].app_flags & kAppRow) fused_append(a, a.req[r], sg);
    seg(a.req[r], sg);
    __syncthreads();  // LDS reuse by the next piece; the piece's stores are issued
    if (a.ent_tag[r] != 0 && threadIdx.x == 0) piece_done(a, r);
  }
  if (a.schedule == kSchedQueue && threadIdx.x == 0) {
    __threadfence();
    if (atomicAdd(&a.queue[1], 1u) == gridDim.x - 1) {
      atomicExch(&a.queue[0], 0u);
      atomicExch(&a.queue[1], 0u);
    }
  }
}

}  // namespace cp
