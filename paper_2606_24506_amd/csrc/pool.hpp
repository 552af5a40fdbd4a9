// Host-side bookkeeping of the shared KV pool: model geometry, the chunk
// and page allocator, admission against the page budget, per-request page
// tables, and the split-KV work planner. Plain C++17, no HIP: the device
// side lives in api.cpp and kernels.hip.
//
// Terms. The pool budget is n_chunks chunks of chunk_bytes. A chunk is
// carved into pages of one model at a time (a per-model slab), so models
// with different per-token bytes kappa(M) share one budget without mixing
// page sizes inside a chunk (Section 3.1: one pool page budget across
// heterogeneous models; Section 2.3 C1). A page holds page_tokens tokens.
// A page-table entry (PTE) is the page's byte offset in the pool >> 8.
//
// Two backings share this bookkeeping. Buffer: the chunks are the n_chunks
// consecutive slices of one device buffer. Virtual (Section 3.1, "KV-cache
// Planner and Virtualizer"; Section 4, KV-cache virtualization): each model
// owns a contiguous range of n_chunks chunk slots in one reserved address
// span, and a slot is backed by physical memory only while it holds pages;
// the budget caps the number of backed slots, not the span. The mapping
// itself is done through the map_chunk / unmap_chunk hooks.
#pragma once

#include <cstdint>
#include <functional>
#include <map>
#include <queue>
#include <string>
#include <vector>

namespace cp {

enum Kind : int32_t { kMLA = 0, kGQA = 1 };

// Mirror value of a page-table entry written by the device and not yet read
// back (device page stacks).
constexpr uint32_t kPendingPte = 0xFFFFFFFFu;

struct Geom {
  int32_t kind = 0;
  int32_t hq = 0, hkv = 0, g = 0;  // g = query heads per KV head
  int32_t head_dim = 0, latent = 0, rope = 0;
  int32_t d_k = 0, d_v = 0;
  int32_t row_elems = 0;  // bf16 elements of one logical row
  int32_t kappa = 0;      // bytes per token
  int64_t page_bytes = 0;
  int32_t ppc = 0;        // pages per chunk
  float scale = 0.f;
  int32_t layers = 1;     // attention layers: one KV plane (page set) each
};

// A request of a model with L layers owns L KV planes (Section 3.2: the
// layer-wise pipeline decodes one layer per stage). Plane l's page-table
// entries are [pte_base + l * plane, pte_base + l * plane + pages_used);
// every plane holds the same token positions. A decode step visits one layer:
// `cursor` is the next layer of the request's token in flight (`inflight`
// = 1 while the new token has been placed but not yet seen by all layers).
struct Request {
  bool open = false;
  int32_t model = -1;
  int64_t ctx_len = 0;        // committed tokens (present in every plane)
  int64_t reserve_pages = 0;  // all planes
  int64_t plane = 0;          // page-table entries per plane
  int64_t pages_used = 0;     // per plane
  uint32_t pte_base = 0;
  int32_t layers = 1;
  int32_t cursor = 0;
  int32_t inflight = 0;
  int64_t attend_len() const { return ctx_len + inflight; }
  uint32_t plane_base(int32_t layer) const { return pte_base + (uint32_t)(layer * plane); }
};

// Deterministic 64-bit generator (splitmix64), used for seeded placement.
struct SplitMix64 {
  uint64_t s;
  explicit SplitMix64(uint64_t seed = 0) : s(seed) {}
  uint64_t next() {
    uint64_t z = (s += 0x9E3779B97F4A7C15ull);
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
  }
};

// First-fit allocator of contiguous ranges in [0, capacity), with coalescing.
class RangeAlloc {
 public:
  void init(uint64_t capacity);
  bool alloc(uint64_t len, uint64_t *start);
  void release(uint64_t start, uint64_t len);
  uint64_t capacity() const { return cap_; }

 private:
  uint64_t cap_ = 0;
  std::map<uint64_t, uint64_t> free_;  // start -> len
};

class PoolState {
 public:
  // Returns "" on success, or an error message.
  std::string init(int32_t page_tokens, uint64_t pool_bytes, uint64_t chunk_bytes, uint64_t seed,
                   int32_t max_requests, bool virt = false);

  int32_t page_tokens() const { return P_; }
  uint64_t chunk_bytes() const { return chunk_bytes_; }
  uint64_t n_chunks() const { return n_chunks_; }
  uint64_t pte_capacity() const { return pte_.size(); }
  uint64_t pool_bytes_used() const { return n_chunks_ * chunk_bytes_; }
  bool virt() const { return virt_; }
  // Bytes of address space the page-table entries can point into: the
  // buffer, or for a virtual pool one budget-sized range per model slot.
  uint64_t span_bytes() const { return (virt_ ? max_models_ * n_chunks_ : n_chunks_) * chunk_bytes_; }
  int32_t max_models() const { return (int32_t)max_models_; }

  // Virtual pools: back / release chunk slot c (byte offset c * chunk_bytes
  // in the span). map_chunk returns false if no physical memory could be
  // mapped. Unset hooks do nothing (host-only pools).
  std::function<bool(int32_t)> map_chunk;
  std::function<void(int32_t)> unmap_chunk;

  // Models.
  std::string add_model(const Geom &g_in, int32_t *id);
  int32_t n_models() const { return (int32_t)models_.size(); }
  const Geom &model(int32_t i) const { return models_[i]; }

  // Requests.
  int32_t max_requests() const { return (int32_t)reqs_.size(); }
  bool valid_open(int32_t id) const { return id >= 0 && id < (int32_t)reqs_.size() && reqs_[id].open; }
  const Request &req(int32_t id) const { return reqs_[id]; }
  // Admission (returns 0, or -3 for budget exhausted, -1 for bad args, -2
  // when a virtual pool could not map the reservation's chunks). A virtual
  // pool backs the whole reservation at admission and keeps a model's
  // chunks while its open reservations may need their slots, so the growth
  // of admitted requests never maps or unmaps memory.
  int open(int32_t model, int64_t reserve_tokens, int32_t *id, std::string *err);
  void close(int32_t id);
  int32_t n_open() const { return n_open_; }

  // Would growing these requests to the given lengths stay within their
  // reservations? (checked before any state change)
  bool fits_reservation(int32_t id, int64_t new_len) const;
  // Allocate the pages needed to grow request id to new_len tokens in every
  // plane, record them in the PTE mirror, and commit new_len. Returns the
  // index range covering the PTEs written as [*first, *first + *count).
  // Never fails for admitted requests within their reservation (after
  // ensure_slots).
  void grow(int32_t id, int64_t new_len, uint64_t *first, uint64_t *count);
  // Places a new token at position ctx_len (pages in every plane as
  // needed) without committing it: the request's layers then see it one
  // decode step at a time. Requires cursor 0 and no token in flight.
  void begin_token(int32_t id, uint64_t *first, uint64_t *count);
  // After a decode step at the request's cursor: moves to the next layer;
  // past the last one, commits the token in flight.
  void advance(int32_t id);
  // After a launch that took the token in flight through every layer at
  // once (the cursor stays at 0): commits it.
  void commit_token(int32_t id);
  // Pages request id still needs (all planes) to reach new_len tokens.
  int64_t pages_to_grow(int32_t id, int64_t new_len) const;
  // Carves fresh chunks for a model until it has at least `pages` free page
  // slots, appending each to *carved. Returns false if a chunk could not be
  // taken or mapped; the caller then gives the carved chunks back with
  // release_empty. Run before grow, so that grow itself cannot fail.
  bool ensure_slots(int32_t model, int64_t pages, std::vector<int32_t> *carved);
  // Returns chunks of *carved that hold no pages to the free list.
  void release_empty(const std::vector<int32_t> &carved);

  // Device page stacks (pools whose decode steps take new pages on the
  // device). Pages handed to a model's stack are allocated (they count
  // against the model's reservations) but belong to no request until a
  // step pops them.
  // Pages the model may still hand out: its reservations minus its
  // allocated pages.
  int64_t stack_room(int32_t model) const { return acct_[model].reserved - acct_[model].used; }
  int64_t in_stack(int32_t model) const { return acct_[model].in_stack; }
  // Allocates k pages for the model's stack (after ensure_slots).
  void take_pages(int32_t model, int64_t k, std::vector<uint32_t> *out);
  // Frees pages taken back from a stack.
  void return_pages(const std::vector<uint32_t> &ptes);
  // Places a new token that opens a page in every plane, the pages being
  // popped from the model's device stack by the step: their entries stay
  // kPendingPte in the mirror until read back. Appends the entries' slots.
  void begin_token_popped(int32_t id, std::vector<uint64_t> *slots);

  const uint32_t *pte_mirror() const { return pte_.data(); }
  uint32_t *pte_mirror_mut() { return pte_.data(); }

  // Accounting.
  uint64_t chunks_used() const { return n_chunks_ - free_count(); }
  uint64_t pages_used() const;
  uint64_t pages_reserved() const;
  // Chunks the budget must hold if every open reservation were filled.
  uint64_t committed_chunks(int32_t extra_model, int64_t extra_pages) const;

 private:
  struct Chunk {
    int32_t model = -1;
    int32_t used = 0;
    std::vector<uint64_t> bits;  // free-slot bitmap while carved
  };
  struct ModelAcct {
    int64_t reserved = 0;   // pages promised to open requests
    int64_t used = 0;       // pages holding KV
    int64_t held = 0;       // chunks carved for this model
    int64_t in_stack = 0;   // allocated pages held by the model's device stack
    std::map<int32_t, int32_t> partial;  // chunk -> free slots (chunks with room)
  };

  uint64_t free_count() const {
    return virt_ ? n_chunks_ - mapped_ : (seed_ ? free_rand_.size() : free_heap_.size());
  }
  int32_t take_chunk(int32_t model);
  void give_chunk(int32_t c);
  void carve(int32_t c, int32_t model);
  void uncarve(int32_t c);
  // virtual pools: release a model's empty chunks that no open reservation
  // still needs, highest slots first
  void trim(int32_t model);
  uint32_t alloc_page(int32_t model);
  void free_page(uint32_t pte);

  int32_t P_ = 64;
  uint64_t chunk_bytes_ = 0, n_chunks_ = 0, seed_ = 0;
  SplitMix64 rng_;
  std::vector<Chunk> chunks_;
  std::priority_queue<int32_t, std::vector<int32_t>, std::greater<int32_t>> free_heap_;
  std::vector<int32_t> free_rand_;
  // virtual pools: per model, slots given back (lowest first) and the next
  // never-used slot of its range
  bool virt_ = false;
  uint64_t max_models_ = 16, mapped_ = 0;
  std::vector<std::priority_queue<int32_t, std::vector<int32_t>, std::greater<int32_t>>> vfree_;
  std::vector<uint64_t> vnext_;
  std::vector<Geom> models_;
  std::vector<ModelAcct> acct_;
  std::vector<Request> reqs_;
  std::vector<int32_t> free_ids_;
  int32_t n_open_ = 0;
  std::vector<uint32_t> pte_;
  RangeAlloc pte_ranges_;
};

// ---------------------------------------------------------------- planner

// One request of a decode call as the planner sees it.
struct PlanIn {
  int32_t model;
  int64_t ctx_len;
};

struct PlanReq {
  int32_t n_chunks = 1;     // KV ranges (splits)
  int32_t chunk_pages = 1;  // pages per range (last may be shorter)
  int32_t n_hblk = 1;       // head blocks per range
};

// Split rule. Every request's pages are cut into page-aligned ranges so the
// whole batch yields about target_units work units of similar byte cost,
// and never fewer pages per range than min_pages. force_splits > 0 gives
// each request min(force_splits, pages) ranges. The result depends only on
// the batch's models and lengths, never on page placement.
void plan_splits(const std::vector<PlanIn> &in, const std::vector<Geom> &models, int32_t page_tokens,
                 int64_t target_units, int32_t min_pages, int32_t force_splits, const std::vector<int32_t> &hblk,
                 std::vector<PlanReq> *out);

}  // namespace cp
