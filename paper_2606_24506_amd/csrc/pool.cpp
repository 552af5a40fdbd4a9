// Host-side bookkeeping of the shared KV pool (see pool.hpp).
#include "pool.hpp"

#include <algorithm>
#include <cmath>

namespace cp {

static inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

// ------------------------------------------------------------ RangeAlloc

void RangeAlloc::init(uint64_t capacity) {
  cap_ = capacity;
  free_.clear();
  if (capacity) free_[0] = capacity;
}

bool RangeAlloc::alloc(uint64_t len, uint64_t *start) {
  if (len == 0) {
    *start = 0;
    return true;
  }
  for (auto it = free_.begin(); it != free_.end(); ++it) {
    if (it->second >= len) {
      *start = it->first;
      uint64_t rest = it->second - len, s = it->first + len;
      free_.erase(it);
      if (rest) free_[s] = rest;
      return true;
    }
  }
  return false;
}

void RangeAlloc::release(uint64_t start, uint64_t len) {
  if (len == 0) return;
  auto it = free_.emplace(start, len).first;
  // coalesce with the following range
  auto nx = std::next(it);
  if (nx != free_.end() && it->first + it->second == nx->first) {
    it->second += nx->second;
    free_.erase(nx);
  }
  // and with the preceding one
  if (it != free_.begin()) {
    auto pv = std::prev(it);
    if (pv->first + pv->second == it->first) {
      pv->second += it->second;
      free_.erase(it);
    }
  }
}

// ------------------------------------------------------------- PoolState

std::string PoolState::init(int32_t page_tokens, uint64_t pool_bytes, uint64_t chunk_bytes, uint64_t seed,
                            int32_t max_requests, bool virt) {
  if (page_tokens < 1 || page_tokens > 4096) return "page_tokens must be in [1, 4096]";
  if (chunk_bytes == 0) chunk_bytes = 2ull << 20;
  if (chunk_bytes % 256) return "chunk_bytes must be a multiple of 256";
  uint64_t n = pool_bytes / chunk_bytes;
  if (n < 1) return "pool_bytes holds less than one chunk";
  if (n > (1ull << 30)) return "too many chunks";
  if (n * chunk_bytes > (1ull << 40)) return "pool larger than 1 TiB cannot be addressed by 32-bit page entries";
  if (max_requests <= 0) max_requests = 4096;
  if (max_requests > (1 << 20)) return "max_requests too large";
  P_ = page_tokens;
  chunk_bytes_ = chunk_bytes;
  n_chunks_ = n;
  seed_ = seed;
  rng_ = SplitMix64(seed);
  virt_ = virt;
  mapped_ = 0;
  vfree_.clear();
  vnext_.clear();
  free_heap_ = decltype(free_heap_)();
  free_rand_.clear();
  if (virt) {
    // one budget-sized range of chunk slots per model, all of them
    // addressable by 32-bit page entries; a model's slots are created when
    // it registers (placement_seed plays no part: the driver places memory)
    max_models_ = std::min<uint64_t>(16, (1ull << 40) / (n * chunk_bytes));
    chunks_.clear();
  } else {
    max_models_ = 16;
    chunks_.assign(n, Chunk{});
    if (seed) {
      free_rand_.resize(n);
      for (uint64_t i = 0; i < n; ++i) free_rand_[i] = (int32_t)i;
    } else {
      for (uint64_t i = 0; i < n; ++i) free_heap_.push((int32_t)i);
    }
  }
  // The smallest page allowed is page_tokens * 128 bytes; page-table space
  // for twice the pages that could ever be carved leaves room for
  // fragmentation of the per-request ranges.
  uint64_t min_page = (uint64_t)page_tokens * 128;
  uint64_t ppc_max = std::max<uint64_t>(1, chunk_bytes / min_page);
  uint64_t cap = 2 * n * ppc_max + 64;
  if (cap > (1ull << 31)) return "page table too large";
  pte_.assign(cap, 0u);
  pte_ranges_.init(cap);
  reqs_.assign(max_requests, Request{});
  free_ids_.clear();
  for (int32_t i = max_requests - 1; i >= 0; --i) free_ids_.push_back(i);
  models_.clear();
  acct_.clear();
  n_open_ = 0;
  return "";
}

std::string PoolState::add_model(const Geom &gi, int32_t *id) {
  if (models_.size() >= 16) return "at most 16 models per pool";
  if (virt_ && models_.size() >= max_models_)
    return "a virtual pool of this budget has address space for " + std::to_string(max_models_) + " models";
  Geom g = gi;
  if (g.hq < 1 || g.hq > 256) return "n_q_heads must be in [1, 256]";
  if (g.kind == kMLA) {
    if (g.hkv != 1) return "MLA models have exactly one (latent) KV head";
    if (g.latent <= 0 || g.latent % 8 || g.rope < 0 || g.rope % 8) return "latent_dim and rope_dim must be multiples of 8";
    if (!(g.scale > 0.f)) return "MLA models need an explicit softmax_scale > 0";
    g.d_k = g.latent + g.rope;
    g.d_v = g.latent;
    g.row_elems = g.d_k;
    g.head_dim = 0;
  } else if (g.kind == kGQA) {
    if (g.hkv < 1 || g.hq % g.hkv) return "n_kv_heads must divide n_q_heads";
    if (g.head_dim <= 0 || g.head_dim % 8) return "head_dim must be a positive multiple of 8";
    g.d_k = g.head_dim;
    g.d_v = g.head_dim;
    g.row_elems = 2 * g.hkv * g.head_dim;
    g.latent = g.rope = 0;
    if (g.scale == 0.f) g.scale = 1.0f / std::sqrt((float)g.head_dim);
    if (!(g.scale > 0.f)) return "softmax_scale must be > 0";
  } else {
    return "unknown model kind";
  }
  if (g.d_k > 1024) return "K width above 1024";
  if (!(g.d_v == 64 || g.d_v == 128 || g.d_v == 256 || g.d_v == 512)) return "V width must be 64, 128, 256 or 512";
  if (g.layers < 1 || g.layers > 1024) return "n_layers must be in [1, 1024]";
  g.g = g.hq / g.hkv;
  g.kappa = 2 * g.row_elems;
  if (g.kappa < 128) return "per-token KV bytes below 128";
  g.page_bytes = (int64_t)P_ * g.kappa;
  if (g.page_bytes % 256) return "page bytes must be a multiple of 256";
  if ((uint64_t)g.page_bytes > chunk_bytes_) return "a page of this model does not fit in one chunk";
  g.ppc = (int32_t)(chunk_bytes_ / (uint64_t)g.page_bytes);
  models_.push_back(g);
  acct_.push_back(ModelAcct{});
  if (virt_) {
    chunks_.resize(models_.size() * n_chunks_);
    vfree_.emplace_back();
    vnext_.push_back(0);
  }
  *id = (int32_t)models_.size() - 1;
  return "";
}

uint64_t PoolState::committed_chunks(int32_t extra_model, int64_t extra_pages) const {
  uint64_t total = 0;
  for (size_t m = 0; m < models_.size(); ++m) {
    const ModelAcct &a = acct_[m];
    int64_t reserved = a.reserved + ((int32_t)m == extra_model ? extra_pages : 0);
    int64_t free_slots = a.held * models_[m].ppc - a.used;
    int64_t owed = reserved - a.used - free_slots;  // pages that still need fresh chunks
    total += (uint64_t)a.held + (owed > 0 ? (uint64_t)ceil_div(owed, models_[m].ppc) : 0);
  }
  return total;
}

int PoolState::open(int32_t model, int64_t reserve_tokens, int32_t *id, std::string *err) {
  if (model < 0 || model >= (int32_t)models_.size()) {
    *err = "unknown model id";
    return -1;
  }
  if (reserve_tokens < 1) {
    *err = "reserve_tokens must be >= 1";
    return -1;
  }
  const int64_t plane = ceil_div(reserve_tokens, P_);
  const int32_t layers = models_[model].layers;
  if (plane > (int64_t)pte_.size() / layers) {
    *err = "reservation larger than the pool";
    return -3;
  }
  int64_t pages = plane * layers;
  if (pages > (int64_t)pte_.size()) {
    *err = "reservation larger than the pool";
    return -3;
  }
  if (free_ids_.empty()) {
    *err = "request table full";
    return -3;
  }
  if (committed_chunks(model, pages) > n_chunks_) {
    *err = "pool page budget exhausted";
    return -3;
  }
  uint64_t base = 0;
  if (!pte_ranges_.alloc((uint64_t)pages, &base)) {
    *err = "page-table space exhausted";
    return -3;
  }
  int32_t rid = free_ids_.back();
  free_ids_.pop_back();
  Request &r = reqs_[rid];
  r.open = true;
  r.model = model;
  r.ctx_len = 0;
  r.reserve_pages = pages;
  r.plane = plane;
  r.pages_used = 0;
  r.pte_base = (uint32_t)base;
  r.layers = layers;
  r.cursor = 0;
  r.inflight = 0;
  acct_[model].reserved += pages;
  ++n_open_;
  *id = rid;
  if (virt_) {
    // back the whole reservation now: admission is the slow path, and the
    // growth of an admitted request then never maps memory
    std::vector<int32_t> carved;
    if (!ensure_slots(model, acct_[model].reserved - acct_[model].used, &carved)) {
      close(rid);  // trims the chunks carved above
      *err = "could not map physical memory for the reservation";
      return -2;
    }
  }
  return 0;
}

void PoolState::close(int32_t id) {
  Request &r = reqs_[id];
  const int32_t model = r.model;
  for (int32_t l = 0; l < r.layers; ++l)
    for (int64_t p = 0; p < r.pages_used; ++p) free_page(pte_[r.plane_base(l) + p]);
  acct_[model].reserved -= r.reserve_pages;
  pte_ranges_.release(r.pte_base, (uint64_t)r.reserve_pages);
  r = Request{};
  free_ids_.push_back(id);
  --n_open_;
  if (virt_) trim(model);
}

bool PoolState::fits_reservation(int32_t id, int64_t new_len) const {
  const Request &r = reqs_[id];
  return ceil_div(new_len, P_) <= r.plane;
}

// Allocates pages of every plane up to new_len tokens; the entries written
// lie in [*first, *first + *count) (plane-major, so the range may include
// unchanged entries between planes).
static void grow_planes(Request &r, int64_t new_len, uint64_t *first, uint64_t *count,
                        std::vector<uint32_t> &pte, const std::function<uint32_t()> &alloc, int32_t P) {
  const int64_t need = (new_len + P - 1) / P;
  *first = 0;
  *count = 0;
  if (need <= r.pages_used) return;
  for (int32_t l = 0; l < r.layers; ++l)
    for (int64_t p = r.pages_used; p < need; ++p) pte[r.plane_base(l) + p] = alloc();
  *first = r.plane_base(0) + (uint64_t)r.pages_used;
  *count = (uint64_t)(r.plane_base(r.layers - 1) + need) - *first;
  r.pages_used = need;
}

void PoolState::grow(int32_t id, int64_t new_len, uint64_t *first, uint64_t *count) {
  Request &r = reqs_[id];
  grow_planes(r, new_len, first, count, pte_, [&] { return alloc_page(r.model); }, P_);
  r.ctx_len = new_len;
}

void PoolState::begin_token(int32_t id, uint64_t *first, uint64_t *count) {
  Request &r = reqs_[id];
  grow_planes(r, r.ctx_len + 1, first, count, pte_, [&] { return alloc_page(r.model); }, P_);
  r.inflight = 1;
}

void PoolState::take_pages(int32_t model, int64_t k, std::vector<uint32_t> *out) {
  for (int64_t i = 0; i < k; ++i) out->push_back(alloc_page(model));
  acct_[model].in_stack += k;
}

void PoolState::return_pages(const std::vector<uint32_t> &ptes) {
  for (uint32_t pte : ptes) {
    const int32_t model = chunks_[(size_t)(((uint64_t)pte << 8) / chunk_bytes_)].model;
    acct_[model].in_stack -= 1;
    free_page(pte);
  }
}

void PoolState::begin_token_popped(int32_t id, std::vector<uint64_t> *slots) {
  Request &r = reqs_[id];
  for (int32_t l = 0; l < r.layers; ++l) {
    const uint64_t slot = r.plane_base(l) + (uint64_t)r.pages_used;
    pte_[slot] = kPendingPte;
    slots->push_back(slot);
  }
  r.pages_used += 1;
  r.inflight = 1;
  acct_[r.model].in_stack -= r.layers;
}

void PoolState::advance(int32_t id) {
  Request &r = reqs_[id];
  if (++r.cursor == r.layers) {
    r.cursor = 0;
    r.ctx_len += r.inflight;
    r.inflight = 0;
  }
}

void PoolState::commit_token(int32_t id) {
  Request &r = reqs_[id];
  r.ctx_len += r.inflight;
  r.inflight = 0;
}

int64_t PoolState::pages_to_grow(int32_t id, int64_t new_len) const {
  const Request &r = reqs_[id];
  int64_t need = ceil_div(new_len, P_);
  return need > r.pages_used ? (need - r.pages_used) * r.layers : 0;
}

bool PoolState::ensure_slots(int32_t model, int64_t pages, std::vector<int32_t> *carved) {
  const Geom &g = models_[model];
  ModelAcct &a = acct_[model];
  while (a.held * g.ppc - a.used < pages) {
    int32_t c = take_chunk(model);
    if (c < 0) return false;
    carve(c, model);
    carved->push_back(c);
  }
  return true;
}

void PoolState::release_empty(const std::vector<int32_t> &carved) {
  for (int32_t c : carved)
    if (chunks_[c].model >= 0 && chunks_[c].used == 0) uncarve(c);
}

void PoolState::carve(int32_t c, int32_t model) {
  const Geom &g = models_[model];
  Chunk &ch = chunks_[c];
  ch.model = model;
  ch.used = 0;
  ch.bits.assign((size_t)(g.ppc + 63) / 64, 0ull);
  for (int32_t s = 0; s < g.ppc; ++s) ch.bits[s >> 6] |= 1ull << (s & 63);
  acct_[model].held += 1;
  acct_[model].partial[c] = g.ppc;
}

void PoolState::uncarve(int32_t c) {
  Chunk &ch = chunks_[c];
  ModelAcct &a = acct_[ch.model];
  a.partial.erase(c);
  a.held -= 1;
  ch.model = -1;
  ch.bits.clear();
  give_chunk(c);
}

int32_t PoolState::take_chunk(int32_t model) {
  if (virt_) {
    if (mapped_ >= n_chunks_) return -1;
    auto &fr = vfree_[model];
    int32_t c;
    bool reused = !fr.empty();
    if (reused) {
      c = fr.top();
    } else {
      if (vnext_[model] >= n_chunks_) return -1;  // unreachable: the range holds the whole budget
      c = (int32_t)((uint64_t)model * n_chunks_ + vnext_[model]);
    }
    if (map_chunk && !map_chunk(c)) return -1;
    if (reused)
      fr.pop();
    else
      vnext_[model] += 1;
    mapped_ += 1;
    return c;
  }
  if (seed_) {
    if (free_rand_.empty()) return -1;
    size_t i = (size_t)(rng_.next() % free_rand_.size());
    int32_t c = free_rand_[i];
    free_rand_[i] = free_rand_.back();
    free_rand_.pop_back();
    return c;
  }
  if (free_heap_.empty()) return -1;
  int32_t c = free_heap_.top();
  free_heap_.pop();
  return c;
}

void PoolState::give_chunk(int32_t c) {
  if (virt_) {
    if (unmap_chunk) unmap_chunk(c);
    mapped_ -= 1;
    vfree_[(uint64_t)c / n_chunks_].push(c);
    return;
  }
  if (seed_)
    free_rand_.push_back(c);
  else
    free_heap_.push(c);
}

uint32_t PoolState::alloc_page(int32_t model) {
  const Geom &g = models_[model];
  ModelAcct &a = acct_[model];
  int32_t c;
  if (!a.partial.empty()) {
    c = a.partial.begin()->first;
  } else {
    // unreachable: ensure_slots carved every chunk this growth needs
    c = take_chunk(model);
    if (c < 0) return 0xFFFFFFFFu;
    carve(c, model);
  }
  Chunk &ch = chunks_[c];
  int32_t slot = -1;
  for (size_t w = 0; w < ch.bits.size(); ++w) {
    if (ch.bits[w]) {
      slot = (int32_t)(w * 64 + (size_t)__builtin_ctzll(ch.bits[w]));
      ch.bits[w] &= ch.bits[w] - 1;
      break;
    }
  }
  ch.used += 1;
  a.used += 1;
  if (--a.partial[c] == 0) a.partial.erase(c);
  uint64_t off = (uint64_t)c * chunk_bytes_ + (uint64_t)slot * (uint64_t)g.page_bytes;
  return (uint32_t)(off >> 8);
}

void PoolState::free_page(uint32_t pte) {
  uint64_t off = (uint64_t)pte << 8;
  int32_t c = (int32_t)(off / chunk_bytes_);
  Chunk &ch = chunks_[c];
  const Geom &g = models_[ch.model];
  ModelAcct &a = acct_[ch.model];
  int32_t slot = (int32_t)((off % chunk_bytes_) / (uint64_t)g.page_bytes);
  ch.bits[slot >> 6] |= 1ull << (slot & 63);
  ch.used -= 1;
  a.used -= 1;
  if (ch.used == 0 && !virt_) {
    uncarve(c);
  } else {
    a.partial[c] += 1;  // a virtual pool's empty chunks wait for trim
  }
}

void PoolState::trim(int32_t model) {
  const Geom &g = models_[model];
  ModelAcct &a = acct_[model];
  std::vector<int32_t> empty;
  for (auto it = a.partial.rbegin(); it != a.partial.rend(); ++it)
    if (chunks_[it->first].used == 0) empty.push_back(it->first);
  for (int32_t c : empty) {  // highest slots first
    if ((a.held - 1) * g.ppc < a.reserved) break;  // the remaining slots are still owed
    uncarve(c);
  }
}

uint64_t PoolState::pages_used() const {
  uint64_t t = 0;
  for (auto &a : acct_) t += (uint64_t)(a.used - a.in_stack);
  return t;
}

uint64_t PoolState::pages_reserved() const {
  uint64_t t = 0;
  for (auto &a : acct_) t += (uint64_t)a.reserved;
  return t;
}

// --------------------------------------------------------------- planner

void plan_splits(const std::vector<PlanIn> &in, const std::vector<Geom> &models, int32_t P, int64_t target_units,
                 int32_t min_pages, int32_t force_splits, const std::vector<int32_t> &hblk,
                 std::vector<PlanReq> *out) {
  out->assign(in.size(), PlanReq{});
  if (min_pages < 1) min_pages = 1;
  double weighted = 0.0;
  for (size_t i = 0; i < in.size(); ++i) {
    int64_t pages = ceil_div(in[i].ctx_len, P);
    weighted += (double)pages * (double)models[in[i].model].page_bytes * (double)hblk[i];
  }
  double unit_cost = target_units > 0 ? weighted / (double)target_units : weighted;
  for (size_t i = 0; i < in.size(); ++i) {
    PlanReq &p = (*out)[i];
    int64_t pages = ceil_div(in[i].ctx_len, P);
    int64_t nch;
    if (force_splits > 0) {
      nch = std::min<int64_t>(force_splits, pages);
    } else {
      double cost = (double)pages * (double)models[in[i].model].page_bytes;
      nch = unit_cost > 0 ? (int64_t)std::ceil(cost / unit_cost - 1e-9) : 1;
      nch = std::max<int64_t>(1, std::min<int64_t>(nch, pages / min_pages));
    }
    if (nch < 1) nch = 1;
    int64_t cp = ceil_div(pages, nch);
    nch = ceil_div(pages, cp);
    p.n_chunks = (int32_t)nch;
    p.chunk_pages = (int32_t)cp;
    p.n_hblk = hblk[i];
  }
}

}  // namespace cp
