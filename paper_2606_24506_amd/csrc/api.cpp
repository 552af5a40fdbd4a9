// C ABI of the shared KV pool (declared in include/crosspool.h): argument
// checks, page allocation, split planning, and kernel launches.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <string>
#include <type_traits>
#include <unordered_map>
#include <vector>

#include "crosspool.h"
#include "kargs.h"
static_assert(cp::kNoAllocScratchBytes == CP_NOALLOC_WORKSPACE_BYTES, "the header states the fixed workspace size");
#include "status.hpp"
#include "pool.hpp"

namespace cp {
hipError_t launch_append(const AppendArgs &a, hipStream_t stream);
hipError_t launch_gather(const GatherArgs &a, hipStream_t stream);
hipError_t launch_decode(const DecodeArgs &a, int grid, uint32_t mask, hipStream_t stream, hipEvent_t ev0,
                         hipEvent_t ev1);
hipError_t launch_decode_wide(const DecodeArgs &a, int grid, int variant, hipStream_t stream, hipEvent_t ev0,
                              hipEvent_t ev1);
int decode_wgs_per_cu(uint32_t mask);
int narrow_streams(int variant);
hipError_t launch_merge(const MergeArgs &a, hipStream_t stream);
hipError_t launch_stack_push(const StackPushArgs &a, hipStream_t stream);
hipError_t scratch_device_address(int device, void **out);
}  // namespace cp

using namespace cp;

namespace {
thread_local std::string g_err;
}  // namespace

namespace cp {
cp_status fail(cp_status code, const char *fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}
}  // namespace cp

namespace {

cp_status hip_fail(hipError_t e, const char *what) {
  return fail(CP_EHIP, "%s: %s", what, hipGetErrorString(e));
}

// Makes the pool's device current for the duration of a call.
struct DeviceGuard {
  int prev = -1;
  bool active = false;
  explicit DeviceGuard(int dev) {
    if (dev < 0) return;
    if (hipGetDevice(&prev) == hipSuccess && prev != dev) {
      active = hipSetDevice(dev) == hipSuccess;
    }
  }
  ~DeviceGuard() {
    if (active) (void)hipSetDevice(prev);
  }
};


// One fused append of cp_attn_decode_step, per request in call order.
struct AppendPlan {
  uint8_t flags = 0;  // kAppRow, kAppPage, kAppPop
  uint32_t off = 0;   // element offset of the row in the caller's rows
  uint32_t pte = 0;   // entry of the new page (kAppPop: the request id)
};
cp_status decode_impl(cp_pool *p, int32_t n, const int32_t *req_ids, const void *q, void *out, float *lse,
                      void *hip_stream, const cp_decode_opts *opts);
}  // namespace

struct cp_pool {
  PoolState st;
  int device = -1;
  bool host_only = true;
  uint8_t *dev_pool = nullptr;  // the buffer, or the base of the reserved span
  bool owns_pool = false;
  // virtual backing: one physical allocation per mapped chunk slot
  bool vmm = false;
  bool vmm_synced = false;  // device synchronized since the current close began
  hipError_t vmm_err = hipSuccess;  // first failed unmap or release of the current close
  hipMemAllocationProp vmm_prop{};
  std::unordered_map<int32_t, hipMemGenericAllocationHandle_t> vmm_handles;
  uint32_t *dev_pte = nullptr;
  uint32_t *pin_pte = nullptr;  // pinned staging copy of the page table
  uint32_t *queue = nullptr;    // work-queue counters
  uint16_t *ws_o = nullptr;  // split partial outputs (bf16)
  float *ws_l = nullptr;
  uint64_t ws_o_cap = 0, ws_l_cap = 0;  // elements
  uint64_t ws_limit = 0;                // bytes of workspace the pool may hold (0: no cap)
  std::vector<void *> ws_retired;         // outgrown workspaces, freed with the pool
  int num_cus = 256;
  // Device page stacks (desc.device_pages): per model kStackCap entries,
  // their counts, per-request pop state and plane strides. The host keeps
  // each stack's entries [0, depth) (bottom first: the device pops from the
  // top, so these are the ones still there) and the page-table slots that
  // steps filled on the device and that it has not read back yet.
  bool dev_pages = false;
  bool broken = false;  // a step's launch failed after its pops were booked
  uint32_t *dev_stack = nullptr;
  int32_t *dev_top = nullptr;
  uint32_t *dev_pop = nullptr;
  uint32_t *dev_geo = nullptr;  // per request id: {first page-table entry, entries per plane}
  uint32_t epoch = 0;
  std::vector<std::vector<uint32_t>> stk;
  std::vector<uint64_t> pending;
  // All-layer launches: per request id its layer cursor and the tokens
  // carried through every layer ([2 id], [2 id + 1]); per launch entry the
  // pieces finished.
  uint32_t *dev_layer = nullptr;
  uint32_t *dev_entry = nullptr;
};

namespace {

// Backs chunk slot c of a virtual pool with a fresh physical allocation
// (Section 4, KV-cache virtualization: pages are mapped on demand, off the
// per-token path). Returns false, with nothing left mapped, on failure.
bool vmm_map(cp_pool *p, int32_t c) {
  DeviceGuard g(p->device);
  const size_t cb = p->st.chunk_bytes();
  void *va = p->dev_pool + (uint64_t)c * cb;
  if (p->vmm_handles.count(c)) return false;  // an earlier unmap of the slot failed
  hipMemGenericAllocationHandle_t h{};
  if (hipMemCreate(&h, cb, &p->vmm_prop, 0) != hipSuccess) return false;
  if (hipMemMap(va, cb, 0, h, 0) != hipSuccess) {
    (void)hipMemRelease(h);
    return false;
  }
  hipMemAccessDesc ad{};
  ad.location = p->vmm_prop.location;
  ad.flags = hipMemAccessFlagsProtReadWrite;
  if (hipMemSetAccess(va, cb, &ad, 1) != hipSuccess) {
    (void)hipMemUnmap(va, cb);
    (void)hipMemRelease(h);
    return false;
  }
  p->vmm_handles[c] = h;
  return true;
}

// Releases the physical memory behind chunk slot c. Work still queued on
// the device may read the slot (a close only requires the caller to have
// synchronized the closed request's own streams), so the device is drained
// once per close before the first unmap.
void vmm_unmap(cp_pool *p, int32_t c) {
  DeviceGuard g(p->device);
  if (!p->vmm_synced) {
    (void)hipDeviceSynchronize();
    p->vmm_synced = true;
  }
  auto it = p->vmm_handles.find(c);
  if (it == p->vmm_handles.end()) return;
  const size_t cb = p->st.chunk_bytes();
  hipError_t e = hipMemUnmap(p->dev_pool + (uint64_t)c * cb, cb);
  if (e != hipSuccess) {
    // still mapped: the slot cannot be mapped again (vmm_map refuses it);
    // destroy retries the unmap
    if (p->vmm_err == hipSuccess) p->vmm_err = e;
    return;
  }
  e = hipMemRelease(it->second);
  if (e != hipSuccess && p->vmm_err == hipSuccess) p->vmm_err = e;
  p->vmm_handles.erase(it);
}

// Reserves the address span of a virtual pool and installs the mapping
// hooks of its allocator.
cp_status vmm_setup(cp_pool *p, int dev) {
  int supported = 0;
  if (hipDeviceGetAttribute(&supported, hipDeviceAttributeVirtualMemoryManagementSupported, dev) != hipSuccess ||
      !supported)
    return fail(CP_EINVAL, "device %d does not support virtual memory management", dev);
  p->vmm_prop.type = hipMemAllocationTypePinned;
  p->vmm_prop.location.type = hipMemLocationTypeDevice;
  p->vmm_prop.location.id = dev;
  size_t gran = 0;
  hipError_t e = hipMemGetAllocationGranularity(&gran, &p->vmm_prop, hipMemAllocationGranularityMinimum);
  if (e != hipSuccess) return hip_fail(e, "mapping granularity query");
  const uint64_t cb = p->st.chunk_bytes();
  if (gran == 0 || cb % gran)
    return fail(CP_EINVAL, "chunk_bytes (%llu) must be a multiple of the device's mapping granularity (%zu)",
                (unsigned long long)cb, gran);
  const size_t align = cb % (2u << 20) == 0 ? (2u << 20) : 0;
  void *base = nullptr;
  e = hipMemAddressReserve(&base, p->st.span_bytes(), align, nullptr, 0);
  if (e != hipSuccess) return fail(CP_ENOMEM, "reserving %llu bytes of address space failed: %s",
                                   (unsigned long long)p->st.span_bytes(), hipGetErrorString(e));
  p->dev_pool = (uint8_t *)base;
  p->vmm = true;
  p->st.map_chunk = [p](int32_t c) { return vmm_map(p, c); };
  p->st.unmap_chunk = [p](int32_t c) { vmm_unmap(p, c); };
  return CP_OK;
}

// ---------------------------------------------------- device page stacks
// (Section 3.3, control lowering: the pool's per-token page allocation runs
// on the device; Section 3.1 keeps the host's mapping work off the
// per-token path.)

// Reads the page-table entries that decode steps wrote on the device back
// into the host mirror. Waits for the device; a slow-path call.
cp_status reconcile_pages(cp_pool *p) {
  if (p->pending.empty()) return CP_OK;
  DeviceGuard g(p->device);
  hipError_t e = hipDeviceSynchronize();
  if (e != hipSuccess) return hip_fail(e, "waiting for the device before reading back popped page entries");
  const uint64_t lo = *std::min_element(p->pending.begin(), p->pending.end());
  const uint64_t hi = *std::max_element(p->pending.begin(), p->pending.end()) + 1;
  std::vector<uint32_t> dev(hi - lo);
  e = hipMemcpy(dev.data(), p->dev_pte + lo, (hi - lo) * 4, hipMemcpyDeviceToHost);
  if (e != hipSuccess) return hip_fail(e, "reading back popped page entries");
  uint32_t *mirror = p->st.pte_mirror_mut();
  for (uint64_t slot : p->pending) mirror[slot] = dev[slot - lo];
  p->pending.clear();
  return CP_OK;
}

// Enqueues the refill of model m's device stack with `fresh` on top of its
// `depth` remaining entries.
cp_status push_stack(cp_pool *p, int32_t m, int64_t depth, const std::vector<uint32_t> &fresh, hipStream_t s) {
  StackPushArgs a{};
  a.top = p->dev_top + m;
  int64_t done = 0;
  do {
    const int32_t k = (int32_t)std::min<int64_t>(kStackPushMax, (int64_t)fresh.size() - done);
    a.dst = p->dev_stack + (uint64_t)m * kStackCap + (uint64_t)(depth + done);
    a.n = k;
    std::copy(fresh.begin() + done, fresh.begin() + done + k, a.ent);
    done += k;
    a.new_top = (int32_t)(depth + done);
    hipError_t e = launch_stack_push(a, s);
    if (e != hipSuccess) return hip_fail(e, "device page stack refill");
  } while (done < (int64_t)fresh.size());
  return CP_OK;
}

// Before a step that pops need[m] pages of model m: refills every stack
// that holds fewer, with at least a chunk's worth of pages (capped by the
// stack and by what the model's reservations may still take). Pages taken
// for a stack count against the reservations like request pages, so they
// cannot push the pool past its budget. On failure nothing is enqueued.
cp_status refill_stacks(cp_pool *p, const std::vector<int64_t> &need, hipStream_t s) {
  for (int32_t m = 0; m < p->st.n_models(); ++m) {
    std::vector<uint32_t> &st = p->stk[(size_t)m];
    const int64_t depth = (int64_t)st.size();
    if (need[(size_t)m] <= depth) continue;
    const Geom &g = p->st.model(m);
    int64_t k = std::max<int64_t>(need[(size_t)m] - depth, std::min<int64_t>(g.ppc, kStackRefill));
    k = std::min<int64_t>({k, p->st.stack_room(m), kStackCap - depth});
    if (depth + k < need[(size_t)m])  // unreachable: every pop is within a reservation
      return fail(CP_ESTATE, "device page stack of model %d cannot hold the pages this step needs", m);
    std::vector<int32_t> carved;
    if (!p->st.ensure_slots(m, k, &carved)) {
      p->st.release_empty(carved);
      return fail(CP_ENOMEM, "could not map physical memory for %lld pages of model %d", (long long)k, m);
    }
    std::vector<uint32_t> fresh;
    p->st.take_pages(m, k, &fresh);
    cp_status rc = push_stack(p, m, depth, fresh, s);
    if (rc) {
      p->st.return_pages(fresh);
      return rc;
    }
    st.insert(st.end(), fresh.begin(), fresh.end());
  }
  return CP_OK;
}

// After request id of model m closes (or is about to): gives back the
// stack's top entries beyond what the model's open reservations may still
// take, so that pages in a stack never hold chunks the budget owes to
// other models. Waits for the device.
cp_status drain_stack(cp_pool *p, int32_t m, int64_t room) {
  std::vector<uint32_t> &st = p->stk[(size_t)m];
  if ((int64_t)st.size() <= room) return CP_OK;
  DeviceGuard g(p->device);
  hipError_t e = hipDeviceSynchronize();
  if (e != hipSuccess) return hip_fail(e, "waiting for the device before draining a page stack");
  const int32_t top = (int32_t)std::max<int64_t>(0, room);
  e = hipMemcpy(p->dev_top + m, &top, 4, hipMemcpyHostToDevice);
  if (e != hipSuccess) return hip_fail(e, "lowering a device page stack");
  std::vector<uint32_t> back(st.begin() + top, st.end());
  st.resize((size_t)top);
  p->st.return_pages(back);
  return CP_OK;
}

// Carves, before any page is allocated, the chunks that growing the
// requests by n_new tokens needs, so that the allocation itself cannot
// fail. (A virtual pool mapped these at admission; this then carves
// nothing.) On failure nothing has changed.
cp_status prepare_growth(cp_pool *p, int32_t n, const int32_t *ids, const int32_t *n_new) {
  std::vector<int64_t> need((size_t)p->st.n_models(), 0);
  for (int32_t i = 0; i < n; ++i) {
    const Request &r = p->st.req(ids[i]);
    need[(size_t)r.model] += p->st.pages_to_grow(ids[i], r.ctx_len + n_new[i]);
  }
  std::vector<int32_t> carved;
  for (int32_t m = 0; m < p->st.n_models(); ++m) {
    if (need[(size_t)m] > 0 && !p->st.ensure_slots(m, need[(size_t)m], &carved)) {
      p->st.release_empty(carved);
      return fail(CP_ENOMEM, "could not map physical memory for %lld new pages of model %d",
                  (long long)need[(size_t)m], m);
    }
  }
  return CP_OK;
}

}  // namespace

extern "C" {

const char *cp_last_error(void) { return g_err.c_str(); }

int32_t cp_version(void) { return (0 << 16) | 1; }

cp_status cp_pool_create(const cp_pool_desc *d, cp_pool **out) {
  if (!d || !out) return fail(CP_EINVAL, "null argument");
  *out = nullptr;
  auto *p = new (std::nothrow) cp_pool();
  if (!p) return fail(CP_ENOMEM, "host allocation failed");
  if (d->backing != CP_BACKING_BUFFER && d->backing != CP_BACKING_VIRTUAL) {
    delete p;
    return fail(CP_EINVAL, "unknown backing %d", d->backing);
  }
  const bool virt = d->backing == CP_BACKING_VIRTUAL;
  if (virt && d->device_mem) {
    delete p;
    return fail(CP_EINVAL, "a virtual pool maps its own memory: device_mem must be NULL");
  }
  std::string e =
      p->st.init(d->page_tokens, d->pool_bytes, d->chunk_bytes, d->placement_seed, d->max_requests, virt);
  if (!e.empty()) {
    delete p;
    return fail(CP_EINVAL, "%s", e.c_str());
  }
  p->device = d->device;
  p->host_only = d->device < 0;
  p->ws_limit = d->max_workspace_bytes;
  if (d->device_pages != 0 && d->device_pages != 1) {
    delete p;
    return fail(CP_EINVAL, "device_pages must be 0 or 1");
  }
  p->dev_pages = d->device_pages == 1;
  p->stk.assign(16, {});
  if (!p->host_only) {
    int ndev = 0;
    if (hipGetDeviceCount(&ndev) != hipSuccess || d->device >= ndev) {
      delete p;
      return fail(CP_EINVAL, "device %d not present", d->device);
    }
    DeviceGuard g(d->device);
    hipError_t he;
    uint64_t bytes = p->st.n_chunks() * p->st.chunk_bytes();
    if (virt) {
      cp_status rc = vmm_setup(p, d->device);
      if (rc) {
        delete p;
        return rc;
      }
    } else if (d->device_mem) {
      if ((uintptr_t)d->device_mem % 256) {
        delete p;
        return fail(CP_EINVAL, "device_mem must be 256-byte aligned");
      }
      p->dev_pool = (uint8_t *)d->device_mem;
    } else {
      he = hipMalloc((void **)&p->dev_pool, bytes);
      if (he != hipSuccess) {
        delete p;
        return fail(CP_ENOMEM, "hipMalloc of %llu pool bytes failed", (unsigned long long)bytes);
      }
      p->owns_pool = true;
    }
    uint64_t nptes = p->st.pte_capacity();
    bool ok = hipMalloc((void **)&p->dev_pte, nptes * 4) == hipSuccess &&
              hipHostMalloc((void **)&p->pin_pte, nptes * 4, hipHostMallocDefault) == hipSuccess &&
              hipMalloc((void **)&p->queue, 64 * sizeof(uint32_t)) == hipSuccess;
    if (ok) ok = hipMemset(p->dev_pte, 0, nptes * 4) == hipSuccess && hipMemset(p->queue, 0, 64 * 4) == hipSuccess;
    if (ok && d->device_pages) {
      const uint64_t nm = 16, nr = (uint64_t)p->st.max_requests();
      ok = hipMalloc((void **)&p->dev_stack, nm * kStackCap * 4) == hipSuccess &&
           hipMalloc((void **)&p->dev_top, nm * 4) == hipSuccess &&
           hipMalloc((void **)&p->dev_pop, nr * 4) == hipSuccess &&
           hipMalloc((void **)&p->dev_geo, nr * 8) == hipSuccess;
      if (ok)
        ok = hipMemset(p->dev_top, 0, nm * 4) == hipSuccess && hipMemset(p->dev_pop, 0, nr * 4) == hipSuccess &&
             hipMemset(p->dev_geo, 0, nr * 8) == hipSuccess;
    }
    if (ok) {
      const uint64_t nr = (uint64_t)p->st.max_requests();
      ok = hipMalloc((void **)&p->dev_layer, nr * 8) == hipSuccess &&
           hipMalloc((void **)&p->dev_entry, kMaxReqPerLaunch * 4) == hipSuccess;
      if (ok) ok = hipMemset(p->dev_layer, 0, nr * 8) == hipSuccess && hipMemset(p->dev_entry, 0, kMaxReqPerLaunch * 4) == hipSuccess;
    }
    if (ok) std::memset(p->pin_pte, 0, nptes * 4);
    int cus = 0;
    if (ok && hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, d->device) == hipSuccess && cus > 0)
      p->num_cus = cus;
    if (ok) ok = hipDeviceSynchronize() == hipSuccess;
    if (!ok) {
      cp_pool_destroy(p);
      return fail(CP_ENOMEM, "device allocation of pool metadata failed");
    }
  }
  *out = p;
  return CP_OK;
}

cp_status cp_pool_destroy(cp_pool *p) {
  if (!p) return fail(CP_EINVAL, "null pool");
  if (p->st.n_open() > 0) return fail(CP_ESTATE, "%d requests still open", p->st.n_open());
  if (!p->host_only) {
    DeviceGuard g(p->device);
    if (p->vmm) {
      (void)hipDeviceSynchronize();
      for (auto &kv : p->vmm_handles) {
        (void)hipMemUnmap(p->dev_pool + (uint64_t)kv.first * p->st.chunk_bytes(), p->st.chunk_bytes());
        (void)hipMemRelease(kv.second);
      }
      (void)hipMemAddressFree(p->dev_pool, p->st.span_bytes());
    }
    if (p->owns_pool && p->dev_pool) (void)hipFree(p->dev_pool);
    if (p->dev_pte) (void)hipFree(p->dev_pte);
    if (p->pin_pte) (void)hipHostFree(p->pin_pte);
    if (p->queue) (void)hipFree(p->queue);
    for (void *b : {(void *)p->dev_stack, (void *)p->dev_top, (void *)p->dev_pop, (void *)p->dev_geo,
                    (void *)p->dev_layer, (void *)p->dev_entry})
      if (b) (void)hipFree(b);
    if (p->ws_o) (void)hipFree(p->ws_o);
    if (p->ws_l) (void)hipFree(p->ws_l);
    for (void *w : p->ws_retired) (void)hipFree(w);
  }
  delete p;
  return CP_OK;
}

cp_status cp_pool_stats(cp_pool *p, cp_pool_stats_t *o) {
  if (!p || !o) return fail(CP_EINVAL, "null argument");
  o->chunks_total = p->st.n_chunks();
  o->chunks_used = p->st.chunks_used();
  o->pages_used = p->st.pages_used();
  o->pages_reserved = p->st.pages_reserved();
  o->requests_open = p->st.n_open();
  o->models = p->st.n_models();
  o->span_bytes = p->st.span_bytes();
  o->backing = p->st.virt() ? CP_BACKING_VIRTUAL : CP_BACKING_BUFFER;
  o->max_models = p->st.max_models();
  return CP_OK;
}

cp_status cp_model_register(cp_pool *p, const cp_model_desc *m, int32_t *model_id) {
  if (!p || !m || !model_id) return fail(CP_EINVAL, "null argument");
  if (m->dtype != CP_BF16) return fail(CP_EINVAL, "only bf16 KV is supported");
  Geom g;
  g.kind = m->kind;
  g.hq = m->n_q_heads;
  g.hkv = m->n_kv_heads;
  g.head_dim = m->head_dim;
  g.latent = m->latent_dim;
  g.rope = m->rope_dim;
  g.scale = m->softmax_scale;
  g.layers = m->n_layers == 0 ? 1 : m->n_layers;
  std::string e = p->st.add_model(g, model_id);
  if (!e.empty()) return fail(CP_EINVAL, "%s", e.c_str());
  return CP_OK;
}

cp_status cp_model_info(cp_pool *p, int32_t id, cp_model_info_t *o) {
  if (!p || !o) return fail(CP_EINVAL, "null argument");
  if (id < 0 || id >= p->st.n_models()) return fail(CP_EINVAL, "unknown model id %d", id);
  const Geom &g = p->st.model(id);
  o->d_k = g.d_k;
  o->d_v = g.d_v;
  o->kappa = g.kappa;
  o->page_bytes = (int32_t)g.page_bytes;
  o->pages_per_chunk = g.ppc;
  o->row_elems = g.row_elems;
  o->n_layers = g.layers;
  return CP_OK;
}

cp_status cp_request_open(cp_pool *p, int32_t model_id, int64_t reserve_tokens, int32_t *req_id) {
  if (!p || !req_id) return fail(CP_EINVAL, "null argument");
  std::string err;
  int rc = p->st.open(model_id, reserve_tokens, req_id, &err);
  if (rc == -3) return fail(CP_ENOSPC, "%s", err.c_str());
  if (rc == -2) return fail(CP_ENOMEM, "%s", err.c_str());
  if (rc != 0) return fail(CP_EINVAL, "%s", err.c_str());
  if (!p->host_only) {
    // the page-table geometry the device pops use, and a fresh layer cursor
    DeviceGuard g(p->device);
    const Request &r = p->st.req(*req_id);
    const uint32_t geo[2] = {r.pte_base, (uint32_t)r.plane}, zero[2] = {0u, 0u};
    hipError_t e = hipMemcpy(p->dev_layer + 2 * (uint64_t)*req_id, zero, 8, hipMemcpyHostToDevice);
    if (e == hipSuccess && p->dev_pages) e = hipMemcpy(p->dev_geo + 2 * (uint64_t)*req_id, geo, 8, hipMemcpyHostToDevice);
    if (e != hipSuccess) {
      p->st.close(*req_id);
      return hip_fail(e, "initialising the request's device state");
    }
  }
  return CP_OK;
}

cp_status cp_request_close(cp_pool *p, int32_t req_id) {
  if (!p) return fail(CP_EINVAL, "null pool");
  if (!p->st.valid_open(req_id)) return fail(CP_EINVAL, "request %d is not open", req_id);
  cp_status rc = reconcile_pages(p);
  if (rc) return rc;
  if (p->dev_pages) {
    // what the model's other open reservations may still take
    const Request &r = p->st.req(req_id);
    const int32_t m = r.model;
    const int64_t room = p->st.stack_room(m) + p->st.in_stack(m) - (r.reserve_pages - r.pages_used * r.layers);
    rc = drain_stack(p, m, room);
    if (rc) return rc;
  }
  p->vmm_synced = false;
  p->vmm_err = hipSuccess;
  p->st.close(req_id);
  if (p->vmm_err != hipSuccess) return hip_fail(p->vmm_err, "request closed, but unmapping its chunks failed");
  return CP_OK;
}

cp_status cp_request_len(cp_pool *p, int32_t req_id, int64_t *ctx_len) {
  if (!p || !ctx_len) return fail(CP_EINVAL, "null argument");
  if (!p->st.valid_open(req_id)) return fail(CP_EINVAL, "request %d is not open", req_id);
  *ctx_len = p->st.req(req_id).ctx_len;
  return CP_OK;
}

cp_status cp_request_cursor(cp_pool *p, int32_t req_id, int32_t *layer, int32_t *in_flight) {
  if (!p || !layer || !in_flight) return fail(CP_EINVAL, "null argument");
  if (!p->st.valid_open(req_id)) return fail(CP_EINVAL, "request %d is not open", req_id);
  *layer = p->st.req(req_id).cursor;
  *in_flight = p->st.req(req_id).inflight;
  return CP_OK;
}

cp_status cp_request_pages(cp_pool *p, int32_t req_id, int64_t first, int64_t count, uint32_t *ptes) {
  if (!p || (!ptes && count > 0)) return fail(CP_EINVAL, "null argument");
  if (!p->st.valid_open(req_id)) return fail(CP_EINVAL, "request %d is not open", req_id);
  cp_status rc = reconcile_pages(p);
  if (rc) return rc;
  const Request &r = p->st.req(req_id);
  if (first < 0 || count < 0 || first + count > r.pages_used)
    return fail(CP_EINVAL, "page range [%lld, %lld) outside the %lld used pages", (long long)first,
                (long long)(first + count), (long long)r.pages_used);
  for (int32_t l = 0; l < r.layers; ++l)  // [layers][count]
    std::memcpy(ptes + (size_t)l * (size_t)count, p->st.pte_mirror() + r.plane_base(l) + first, (size_t)count * 4);
  return CP_OK;
}

}  // extern "C"

namespace {

// Fills the kernel view of a model's geometry. `variant` selects the code
// path (set by the caller for decode).
GeomK geom_k(const Geom &g, int32_t P) {
  GeomK k{};
  k.kind = g.kind;
  k.hq = g.hq;
  k.hkv = g.hkv;
  k.g = g.g;
  k.d_k = g.d_k;
  k.d_v = g.d_v;
  k.row_elems = g.row_elems;
  k.page_tokens = P;
  k.page_bytes = (int32_t)g.page_bytes;
  k.scale_log2 = g.scale * 1.4426950408889634f;
  k.variant = 0;
  k.nb = 1;
  k.layers = g.layers;
  return k;
}

cp_status check_ids(cp_pool *p, int32_t n, const int32_t *ids) {
  if (n < 0) return fail(CP_EINVAL, "negative request count");
  if (n > 0 && !ids) return fail(CP_EINVAL, "null req_ids");
  std::vector<int32_t> s(ids, ids + n);
  for (int32_t i = 0; i < n; ++i)
    if (!p->st.valid_open(s[i])) return fail(CP_EINVAL, "request %d is not open", s[i]);
  std::sort(s.begin(), s.end());
  for (int32_t i = 1; i < n; ++i)
    if (s[i] == s[i - 1]) return fail(CP_EINVAL, "request %d appears twice in one call", s[i]);
  return CP_OK;
}

// Copies page-table entries [lo, hi) to the device through the pinned copy.
cp_status push_ptes(cp_pool *p, uint64_t lo, uint64_t hi, hipStream_t s) {
  if (hi <= lo) return CP_OK;
  std::memcpy(p->pin_pte + lo, p->st.pte_mirror() + lo, (size_t)(hi - lo) * 4);
  hipError_t e = hipMemcpyAsync(p->dev_pte + lo, p->pin_pte + lo, (size_t)(hi - lo) * 4, hipMemcpyHostToDevice, s);
  if (e != hipSuccess) return hip_fail(e, "page-table copy");
  return CP_OK;
}


// One request's rows of one KV plane for launch_appends.
struct AppItem {
  int32_t model;
  uint32_t n_new, old_len;  // rows, and the tokens already in the plane
  uint32_t pte_base;        // the plane's first page-table entry
  uint64_t src_off;         // element offset of the first row in `rows`
};

// Append launches for rows already accounted for in the host tables, in
// groups of at most kMaxReqPerLaunch items and kMaxLaunchModels models.
cp_status launch_appends(cp_pool *p, const std::vector<AppItem> &items, const void *rows, hipStream_t s) {
  const int32_t P = p->st.page_tokens();
  size_t i = 0;
  while (i < items.size()) {
    AppendArgs a{};
    a.pool = p->dev_pool;
    a.pte = p->dev_pte;
    a.rows = (const uint16_t *)rows;
    int32_t nm = 0, model_map[16];
    for (int k = 0; k < 16; ++k) model_map[k] = -1;
    uint32_t grid_rows = 0;
    while (i < items.size() && a.n_req < kMaxReqPerLaunch) {
      const AppItem &it = items[i];
      int32_t mi = model_map[it.model];
      if (mi < 0) {
        if (nm == kMaxLaunchModels) break;
        mi = model_map[it.model] = nm;
        a.geom[nm++] = geom_k(p->st.model(it.model), P);
      }
      if (it.n_new > 0) {
        AppReq &q = a.req[a.n_req++];
        q.src_off = it.src_off;
        q.row_begin = grid_rows;
        q.n_new = it.n_new;
        q.old_len = it.old_len;
        q.pte_base = it.pte_base;
        q.model = (uint32_t)mi;
        grid_rows += it.n_new;
      }
      ++i;
    }
    a.total_rows = (int32_t)grid_rows;
    if (a.n_req > 0) {
      hipError_t e = launch_append(a, s);
      if (e != hipSuccess) return hip_fail(e, "append launch");
    }
  }
  return CP_OK;
}

}  // namespace

extern "C" {

cp_status cp_kv_append(cp_pool *p, int32_t n, const int32_t *req_ids, const int32_t *n_new, const void *rows,
                       void *hip_stream) {
  if (!p) return fail(CP_EINVAL, "null pool");
  cp_status rc = check_ids(p, n, req_ids);
  if (rc) return rc;
  if (n > 0 && !n_new) return fail(CP_EINVAL, "null n_new");
  if (p->broken) return fail(CP_ESTATE, "a failed decode step left the device page stacks out of step; destroy the pool");
  // the page-table copies below must not overwrite entries a step popped
  rc = reconcile_pages(p);
  if (rc) return rc;
  int64_t total = 0;
  for (int32_t i = 0; i < n; ++i) {
    if (n_new[i] < 0) return fail(CP_EINVAL, "negative n_new for request %d", req_ids[i]);
    const Request &r = p->st.req(req_ids[i]);
    if (n_new[i] > 0 && (r.cursor != 0 || r.inflight))
      return fail(CP_EINVAL, "request %d has a token in flight at layer %d; finish its decode steps first",
                  req_ids[i], r.cursor);
    int64_t nl = r.ctx_len + n_new[i];
    if (nl > 0xFFFFFFF0ll) return fail(CP_EINVAL, "context length overflow");
    if (!p->st.fits_reservation(req_ids[i], nl))
      return fail(CP_EINVAL, "request %d would grow to %lld tokens, past its reservation of %lld pages", req_ids[i],
                  (long long)nl, (long long)r.reserve_pages);
    total += (int64_t)n_new[i] * r.layers;
  }
  if (p->host_only) {
    if (rows) return fail(CP_EINVAL, "host-only pool: rows must be NULL");
  } else if (total > 0 && !rows) {
    return fail(CP_EINVAL, "null rows");
  }
  if (total == 0) return CP_OK;
  if (total > 0x7FFFFFFF) return fail(CP_EINVAL, "too many rows in one call");

  // All checks passed: carve (and map) chunks, then allocate pages and
  // update host page tables.
  rc = prepare_growth(p, n, req_ids, n_new);
  if (rc) return rc;
  // Rows of request i are [layers][n_new][row_elems], requests in call order.
  std::vector<AppItem> items;
  uint64_t lo = UINT64_MAX, hi = 0, src = 0;
  for (int32_t i = 0; i < n; ++i) {
    const Request &r = p->st.req(req_ids[i]);
    const uint32_t old_len = (uint32_t)r.ctx_len;
    const uint64_t row_elems = (uint64_t)p->st.model(r.model).row_elems;
    uint64_t first, count;
    p->st.grow(req_ids[i], r.ctx_len + n_new[i], &first, &count);
    if (count) {
      lo = std::min(lo, first);
      hi = std::max(hi, first + count);
    }
    for (int32_t l = 0; l < r.layers && n_new[i] > 0; ++l) {
      items.push_back(AppItem{r.model, (uint32_t)n_new[i], old_len, r.plane_base(l), src});
      src += (uint64_t)n_new[i] * row_elems;
    }
  }
  if (p->host_only) return CP_OK;

  DeviceGuard g(p->device);
  hipStream_t s = (hipStream_t)hip_stream;
  rc = push_ptes(p, lo, hi, s);
  if (rc) return rc;

  return launch_appends(p, items, rows, s);
}

cp_status cp_kv_gather(cp_pool *p, int32_t req_id, int64_t start, int64_t n_tok, void *dst, void *hip_stream) {
  if (!p) return fail(CP_EINVAL, "null pool");
  if (p->host_only) return fail(CP_ESTATE, "host-only pool has no device data");
  if (!p->st.valid_open(req_id)) return fail(CP_EINVAL, "request %d is not open", req_id);
  const Request &r = p->st.req(req_id);
  if (start < 0 || n_tok < 0 || start + n_tok > r.ctx_len)
    return fail(CP_EINVAL, "range [%lld, %lld) outside the context of %lld tokens", (long long)start,
                (long long)(start + n_tok), (long long)r.ctx_len);
  if (n_tok == 0) return CP_OK;
  if (!dst) return fail(CP_EINVAL, "null dst");
  DeviceGuard g(p->device);
  const uint64_t row_elems = (uint64_t)p->st.model(r.model).row_elems;
  for (int32_t l = 0; l < r.layers; ++l) {  // dst is [layers][n_tok][row_elems]
    GatherArgs a{};
    a.pool = p->dev_pool;
    a.pte = p->dev_pte;
    a.dst = (uint16_t *)dst + (uint64_t)l * (uint64_t)n_tok * row_elems;
    a.pte_base = r.plane_base(l);
    a.start = (uint32_t)start;
    a.n_tok = (uint32_t)n_tok;
    a.geom = geom_k(p->st.model(r.model), p->st.page_tokens());
    hipError_t e = launch_gather(a, (hipStream_t)hip_stream);
    if (e != hipSuccess) return hip_fail(e, "gather launch");
  }
  return CP_OK;
}

}  // extern "C"

namespace {

// Vector-path variant for a model: heads per block and V values per lane.
void choose_valu(const Geom &g, GeomK *k, int32_t P) {
  // GQA/MHA groups of 1 to 4 heads with head_dim 64 or 128 take the
  // small-group kernel (one KV head per unit)
  if (g.kind == kGQA && g.g <= 4 && (g.head_dim == 64 || g.head_dim == 128) && P % 16 == 0) {
    const int gi = g.g == 1 ? 0 : g.g == 2 ? 1 : 2;  // 3 heads run as 4, one padded
    k->variant = (g.head_dim == 64 ? kS_G1_D64 : kS_G1_D128) + gi;
    k->nb = 1;
    return;
  }
  const int hb = g.g > 8 ? 16 : 8;
  const int dpl = g.d_v / 64;
  int v = 0;
  switch (dpl) {
    case 8: v = 0; break;
    case 4: v = 1; break;
    case 2: v = 2; break;
    default: v = 3; break;
  }
  k->variant = v + (hb == 8 ? 4 : 0);
  k->nb = (g.g + hb - 1) / hb;
}

constexpr int32_t kMatrixFirst = 16;

// Matrix-core variant for a model, or -1 when none fits its geometry. The
// matrix path serves models whose query heads share a KV head in groups of
// 8 or more (the MLA latent head, MQA, GQA), where the per-KV-head work is a
// contraction over the group: the narrow variants (8-32 heads) stream
// wave-private slices of 16 (MLA) or 32 (head_dim 128) tokens, the wide ones
// (64-128 heads) 32-token tiles shared by the workgroup. Pages must hold a
// whole number of slices or tiles.
int32_t matrix_variant(const Geom &g, int32_t P) {
  if (g.kind == kMLA && g.latent == 512 && g.rope == 64) {
    if (g.g == 16 && P % 16 == 0) return kM_MLA_G16;
    if (g.g == 32 && P % 16 == 0) return kM_MLA_G32;
    if (g.g == 128 && P % 32 == 0) return kM_MLA_G128;
    return -1;
  }
  if (g.kind == kGQA && g.head_dim == 128 && P % 32 == 0) {
    if (g.g == 8) return kM_D128_G8;
    if (g.g == 16) return kM_D128_G16;
    if (g.g == 32) return kM_D128_G32;
    if (g.g == 64) return kM_D128_G64;
    if (g.g == 128) return kM_D128_G128;
  }
  return -1;
}

// Work units per KV range of a request: the narrow matrix kernel takes one
// KV head per token stream at once when the model's KV heads are a multiple
// of its stream count; otherwise every KV head (times its head blocks) is a
// unit of its own.
int32_t units_per_range(const Geom &g, const GeomK &k) {
  const int ns = narrow_streams(k.variant);
  if (ns > 0 && g.hkv % ns == 0) return g.hkv / ns;
  return g.hkv * k.nb;
}

// Split workspace: o_elems bf16 partial outputs and l_floats fp32 partial
// lse values.
cp_status ensure_ws(cp_pool *p, uint64_t o_elems, uint64_t l_floats) {
  if (o_elems <= p->ws_o_cap && l_floats <= p->ws_l_cap) return CP_OK;
  const uint64_t need_bytes = o_elems * sizeof(uint16_t) + l_floats * sizeof(float);
  if (p->ws_limit && need_bytes > p->ws_limit)
    return fail(CP_ENOMEM, "the split plan needs %llu bytes of workspace, past the pool's cap of %llu",
                (unsigned long long)need_bytes, (unsigned long long)p->ws_limit);
  // Growth allocates twice what is asked, so that the slow drift of split
  // plans as contexts grow rarely repeats it, and keeps the old buffers
  // until the pool is destroyed: kernels already queued may still use them,
  // and freeing them here would stall the host until the device drains.
  // With a cap, growth takes what is asked and no more, and outgrown
  // buffers are not kept: the cap bounds the bytes held.
  auto grow = [&](auto **buf, uint64_t *cap, uint64_t need) -> cp_status {
    if (need <= *cap) return CP_OK;
    const uint64_t c = p->ws_limit ? need : std::max<uint64_t>(2 * need, 2 * *cap);
    void *nb = nullptr;
    if (p->ws_limit && *buf) {
      // queued kernels may still read the old buffer: drain the device first
      (void)hipDeviceSynchronize();
      (void)hipFree(*buf);
      *buf = nullptr;
      *cap = 0;
    }
    if (hipMalloc(&nb, c * sizeof(**buf)) != hipSuccess) return fail(CP_ENOMEM, "workspace allocation failed");
    if (*buf) p->ws_retired.push_back(*buf);
    *buf = static_cast<std::remove_reference_t<decltype(*buf)>>(nb);
    *cap = c;
    return CP_OK;
  };
  cp_status rc = grow(&p->ws_o, &p->ws_o_cap, o_elems);
  if (rc) return rc;
  return grow(&p->ws_l, &p->ws_l_cap, l_floats);
}

}  // namespace

extern "C" {

cp_status cp_attn_decode_ex(cp_pool *p, int32_t n, const int32_t *req_ids, const void *q, void *out, float *lse,
                            void *hip_stream, const cp_decode_opts *opts) {
  return decode_impl(p, n, req_ids, q, out, lse, hip_stream, opts);
}

}  // extern "C"

namespace {

// Checks what every decode call needs; fills the options and the per-model
// kernel geometry (variant, head blocking, page cost).
cp_status decode_prepare(cp_pool *p, int32_t n, const int32_t *req_ids, const void *q, void *out, float *lse,
                         const cp_decode_opts *opts, cp_decode_opts *o_out, std::vector<GeomK> *gk_out) {
  if (!p) return fail(CP_EINVAL, "null pool");
  if (p->host_only) return fail(CP_ESTATE, "host-only pool cannot decode");
  if (p->broken) return fail(CP_ESTATE, "a failed decode step left the device page stacks out of step; destroy the pool");
  if (n < 1) return fail(CP_EINVAL, "decode needs at least one request");
  cp_status rc = check_ids(p, n, req_ids);
  if (rc) return rc;
  if (!q || !out || !lse) return fail(CP_EINVAL, "null q, out or lse");
  cp_decode_opts o{};
  if (opts) o = *opts;
  if (o.num_splits < 0) return fail(CP_EINVAL, "num_splits must be >= 0");
  if (o.path < CP_PATH_AUTO || o.path > CP_PATH_MFMA) return fail(CP_EINVAL, "unknown path %d", o.path);
  if (o.schedule < CP_SCHED_BALANCED || o.schedule > CP_SCHED_GRID)
    return fail(CP_EINVAL, "unknown schedule %d", o.schedule);
  if (o.schedule == CP_SCHED_BALANCED && o.num_splits != 0)
    return fail(CP_EINVAL, "num_splits applies to the queue and grid schedules only");
  const int32_t P = p->st.page_tokens();

  // Per-model kernel variant, head blocking and page cost.
  std::vector<GeomK> gk(p->st.n_models());
  for (int32_t m = 0; m < p->st.n_models(); ++m) {
    const Geom &g = p->st.model(m);
    gk[m] = geom_k(g, P);
    gk[m].pool_model = m;
    const int32_t mv = o.path == CP_PATH_VALU ? -1 : matrix_variant(g, P);
    if (mv >= 0) {
      gk[m].variant = mv;
      gk[m].nb = mv == kM_MLA_G32 ? 2 : 1;  // units of 16 heads per KV range
    } else {
      choose_valu(g, &gk[m], P);
    }
    // relative work of one page: its bytes, times the head blocks that each
    // reread it on the MLA vector path
    const int64_t unit = std::max<int64_t>(1, (g.page_bytes + 8191) / 8192);
    gk[m].page_cost = (int32_t)(unit * (g.kind == kMLA ? gk[m].nb : 1));
  }
  for (int32_t i = 0; i < n; ++i) {
    const int32_t m = p->st.req(req_ids[i]).model;
    if (o.path == CP_PATH_MFMA && gk[m].variant < kMatrixFirst)
      return fail(CP_EINVAL, "model %d has no matrix-core variant (needs a group of 8, 16, 32, 64 or 128 query heads per KV head)", m);
  }
  *o_out = o;
  *gk_out = std::move(gk);
  return CP_OK;
}

// Everything one decode call launches: per-request offsets, launch groups,
// split plan and workspace layout. Built and checked in full before any
// pool state changes or anything is enqueued.
struct DecodePlan {
  struct Group {
    std::vector<int32_t> idx;
    std::vector<int32_t> models;  // pool model ids, launch-local order
    uint32_t mask = 0;
    int grid = 0;
    uint32_t total_cost = 0;
    uint32_t n_units = 0;
  };
  cp_decode_opts o{};
  std::vector<GeomK> gk;
  std::vector<int64_t> attend;  // tokens each request attends over (call order)
  std::vector<uint64_t> q_off, o_off, l_off;
  std::vector<Group> groups;
  std::vector<int32_t> n_slots, chunk_pages, first_worker, hblk;
  std::vector<uint32_t> cost_prefix, ws_base, ws_orow;
  uint64_t ws_rows = 0, ws_elems = 0;  // partial lse rows and partial output elements
  uint16_t *ws_o = nullptr;            // bound by the caller before launch
  float *ws_l = nullptr;
};

// Plans a decode over requests whose attended lengths are their current
// ones plus extra[i] (tokens a fused step places before the launch; NULL:
// none). pl->o and pl->gk come from decode_prepare. Runs every capacity
// check of the call; changes nothing.
cp_status plan_decode(cp_pool *p, int32_t n, const int32_t *req_ids, const int32_t *extra, DecodePlan *pl) {
  const cp_decode_opts &o = pl->o;
  const std::vector<GeomK> &gk = pl->gk;
  const int32_t P = p->st.page_tokens();
  auto model_of = [&](int32_t i) { return p->st.req(req_ids[i]).model; };
  pl->attend.assign(n, 0);
  for (int32_t i = 0; i < n; ++i) {
    pl->attend[i] = p->st.req(req_ids[i]).attend_len() + (extra ? extra[i] : 0);
    if (pl->attend[i] < 1) return fail(CP_EINVAL, "request %d has an empty context", req_ids[i]);
  }

  // Packed offsets in call order.
  pl->q_off.assign(n, 0);
  pl->o_off.assign(n, 0);
  pl->l_off.assign(n, 0);
  std::vector<int64_t> pages(n);
  uint64_t qo = 0, oo = 0, lo = 0;
  for (int32_t i = 0; i < n; ++i) {
    const Geom &g = p->st.model(model_of(i));
    pl->q_off[i] = qo;
    pl->o_off[i] = oo;
    pl->l_off[i] = lo;
    qo += (uint64_t)g.hq * g.d_k;
    oo += (uint64_t)g.hq * g.d_v;
    lo += (uint64_t)g.hq;
    pages[i] = (pl->attend[i] + P - 1) / P;
  }
  if (qo > 0xFFFFFFFFull || oo > 0xFFFFFFFFull) return fail(CP_EINVAL, "batch too large");
  // kernel family: vector variants share a launch, narrow matrix variants
  // share another, and each wide variant has a kernel of its own
  auto wclass = [&](int32_t i) {
    const int v = gk[model_of(i)].variant;
    // (launch classes: vector, narrow matrix, small-group vector, each wide variant)
    return is_wide_variant(v) ? v : v >= kMatrixFirst ? 1 : (v >= kS_G1_D64 && v <= kS_G4_D128) ? 2 : 0;
  };

  // Launch groups: requests whose kernels share a workgroup size, at most
  // kMaxReqPerLaunch requests and kMaxLaunchModels models each. Within the
  // queue and grid schedules the costliest units go first.
  std::vector<int32_t> order(n);
  for (int32_t i = 0; i < n; ++i) order[i] = i;
  std::stable_sort(order.begin(), order.end(), [&](int32_t x, int32_t y) { return wclass(x) < wclass(y); });
  using Group = DecodePlan::Group;
  std::vector<Group> &groups = pl->groups;
  groups.clear();
  for (int32_t k = 0; k < n;) {
    Group g;
    const int cls = wclass(order[k]);
    while (k < n && (int)g.idx.size() < kMaxReqPerLaunch && wclass(order[k]) == cls) {
      const int32_t m = model_of(order[k]);
      if (std::find(g.models.begin(), g.models.end(), m) == g.models.end()) {
        if ((int)g.models.size() == kMaxLaunchModels) break;
        g.models.push_back(m);
      }
      g.idx.push_back(order[k++]);
    }
    for (int32_t m : g.models) g.mask |= 1u << gk[m].variant;
    groups.push_back(std::move(g));
  }

  // Per-request plan: partial slots and the fields the kernels read.
  std::vector<int32_t> &n_slots = pl->n_slots, &chunk_pages = pl->chunk_pages, &first_worker = pl->first_worker,
                       &hblk = pl->hblk;
  std::vector<uint32_t> &cost_prefix = pl->cost_prefix;
  n_slots.assign(n, 1);
  chunk_pages.assign(n, 0);
  first_worker.assign(n, 0);
  hblk.assign(n, 1);
  cost_prefix.assign(n, 0);
  for (int32_t i = 0; i < n; ++i) hblk[i] = units_per_range(p->st.model(model_of(i)), gk[model_of(i)]);
  for (Group &g : groups) {
    const bool wide = g.mask && is_wide_variant(__builtin_ctz(g.mask));
    const int wgs = wide ? 1 : decode_wgs_per_cu(g.mask);
    const int64_t slots = (int64_t)p->num_cus * wgs;
    if (o.schedule == CP_SCHED_BALANCED) {
      // Every workgroup pays the fixed cost of its first piece, so the cost
      // line charges kPieceFixedCost only where a request boundary falls
      // inside a workgroup's share (that workgroup runs a second piece):
      // not before the launch's first request, and not at a boundary that
      // coincides with a share boundary of the line without fixed costs
      // (equal requests over a multiple of their count of workgroups).
      uint64_t T0 = 0, maxc = 1;
      for (int32_t i : g.idx) {
        const uint64_t c = (uint64_t)gk[model_of(i)].page_cost;
        T0 += (uint64_t)pages[i] * c;
        maxc = std::max(maxc, c);
      }
      const uint64_t W0 = std::max<uint64_t>(1, std::min<uint64_t>((uint64_t)slots, T0 / maxc));
      uint64_t T = 0, pre0 = 0;
      for (size_t k = 0; k < g.idx.size(); ++k) {
        const int32_t i = g.idx[k];
        const uint64_t c = (uint64_t)gk[model_of(i)].page_cost;
        const bool straddled = k > 0 && (pre0 * W0) % T0 != 0;
        T += straddled ? kPieceFixedCost : 0;
        cost_prefix[i] = (uint32_t)std::min<uint64_t>(T, 0xFFFFFFFFull);  // the request's first page
        T += (uint64_t)pages[i] * c;
        pre0 += (uint64_t)pages[i] * c;
      }
      if (T > 0xFFFFFFFFull) return fail(CP_EINVAL, "batch too large for one launch");
      // every range spans at least one page of any model, so no request has
      // an empty slot between its first and last worker
      const uint64_t W = std::max<uint64_t>(1, std::min<uint64_t>((uint64_t)slots, T / maxc));
      auto owner = [&](uint64_t x) { return (uint32_t)(((x + 1) * W - 1) / T); };
      for (int32_t i : g.idx) {
        // page j of the request sits at C + j c
        const uint64_t c = (uint64_t)gk[model_of(i)].page_cost, C = cost_prefix[i];
        const uint32_t w0 = owner(C), w1 = owner(C + (uint64_t)(pages[i] - 1) * c);
        first_worker[i] = (int32_t)w0;
        n_slots[i] = (int32_t)(w1 - w0 + 1);
      }
      g.grid = (int)W;
      g.total_cost = (uint32_t)T;
      if (g.grid > 0xFFFF) return fail(CP_EINVAL, "too many workers");
    } else {
      // queue / grid: page-aligned KV ranges of similar cost, about two per
      // workgroup slot (one when every request is a 128-head matrix model,
      // whose partials are large); at least four pages per range on the
      // matrix path so all waves of a workgroup get pages
      bool all_wide = true, any_matrix = false;
      std::vector<PlanIn> pin;
      std::vector<int32_t> hb;
      for (int32_t i : g.idx) {
        const int32_t v = gk[model_of(i)].variant;
        all_wide = all_wide && is_wide_variant(v);
        any_matrix = any_matrix || v >= kMatrixFirst;
        pin.push_back(PlanIn{model_of(i), pl->attend[i]});
        hb.push_back(hblk[i]);
      }
      std::vector<Geom> geoms;
      for (int32_t m = 0; m < p->st.n_models(); ++m) geoms.push_back(p->st.model(m));
      std::vector<PlanReq> plan;
      plan_splits(pin, geoms, P, slots * (all_wide ? 1 : 2), any_matrix ? 4 : 1, o.num_splits, hb, &plan);
      // costliest units first
      std::vector<int32_t> pos(g.idx.size());
      for (size_t k = 0; k < pos.size(); ++k) pos[k] = (int32_t)k;
      std::stable_sort(pos.begin(), pos.end(), [&](int32_t x, int32_t y) {
        const Geom &gx = p->st.model(model_of(g.idx[x])), &gy = p->st.model(model_of(g.idx[y]));
        return (double)plan[x].chunk_pages * gx.page_bytes > (double)plan[y].chunk_pages * gy.page_bytes;
      });
      std::vector<int32_t> idx2;
      uint32_t units = 0;
      for (int32_t k : pos) {
        const int32_t i = g.idx[k];
        if (plan[k].chunk_pages > 0xFFFF || plan[k].n_chunks > 0xFFFF) return fail(CP_EINVAL, "context too long to split");
        chunk_pages[i] = plan[k].chunk_pages;
        n_slots[i] = plan[k].n_chunks;
        cost_prefix[i] = units;  // first unit
        units += (uint32_t)plan[k].n_chunks * (uint32_t)hblk[i];
        idx2.push_back(i);
      }
      g.idx = idx2;
      g.n_units = units;
      g.grid = o.schedule == CP_SCHED_QUEUE ? (int)std::min<int64_t>(units, slots) : (int)units;
    }
  }

  // Workspace for requests split over several slots.
  uint64_t ws_rows = 0, ws_elems = 0;
  pl->ws_base.assign(n, kNoWs);
  pl->ws_orow.assign(n, 0);
  for (int32_t i = 0; i < n; ++i) {
    if (n_slots[i] <= 1) continue;
    const Geom &g = p->st.model(model_of(i));
    pl->ws_base[i] = (uint32_t)ws_rows;
    ws_rows += (uint64_t)n_slots[i] * g.hq;
    ws_elems = (ws_elems + 511) / 512 * 512;
    pl->ws_orow[i] = (uint32_t)(ws_elems / (uint64_t)g.d_v);
    ws_elems += (uint64_t)n_slots[i] * g.hq * g.d_v;
  }
  if (ws_rows >= kNoWs || ws_elems / 64 >= kNoWs) return fail(CP_EINVAL, "split workspace too large");
  pl->ws_rows = ws_rows;
  pl->ws_elems = ws_elems;
  return CP_OK;
}

// Binds the pool's own split workspace to a plan, growing it if needed.
cp_status bind_pool_workspace(cp_pool *p, DecodePlan *pl) {
  if (pl->ws_rows) {
    DeviceGuard dg(p->device);
    cp_status rc = ensure_ws(p, pl->ws_elems, pl->ws_rows);
    if (rc) return rc;
  }
  pl->ws_o = p->ws_o;
  pl->ws_l = p->ws_l;
  return CP_OK;
}

// Enqueues a planned decode: the attention launches (with `app`, one entry
// per request in call order, they also perform the fused appends of
// cp_attn_decode_step) and the merges of split requests. Only HIP failures
// remain possible here.
cp_status launch_plan(cp_pool *p, const DecodePlan &pl, int32_t n, const int32_t *req_ids, const void *q,
                      void *out, float *lse, void *hip_stream, const void *rows, const std::vector<AppendPlan> *app,
                      const int32_t *layer = nullptr, const uint32_t *tag = nullptr) {
  const cp_decode_opts &o = pl.o;
  DeviceGuard dg(p->device);
  hipStream_t s = (hipStream_t)hip_stream;
  // The caller's events take the start of the first decode launch and the
  // end of the last one (timestamps of the launches themselves, no marker
  // packets between them).
  for (size_t gi = 0; gi < pl.groups.size(); ++gi) {
    const DecodePlan::Group &g = pl.groups[gi];
    DecodeArgs a{};
    a.pool = p->dev_pool;
    a.pte = p->dev_pte;
    a.q = (const uint16_t *)q;
    a.out = (uint16_t *)out;
    a.lse = lse;
    a.rows = (const uint16_t *)rows;
    a.ws_o = pl.ws_o;
    a.ws_l = pl.ws_l;
    a.queue = p->queue;
    a.stack = p->dev_stack;
    a.stack_top = p->dev_top;
    a.pop_state = p->dev_pop;
    a.req_geo = p->dev_geo;
    a.epoch = p->epoch;
    a.layer_cursor = p->dev_layer;
    a.layer_tokens = p->dev_layer + 1;  // indexed by 2 * request id below
    a.entry_done = p->dev_entry;
    a.schedule = o.schedule;
    a.total_cost = g.total_cost;
    a.n_units = (int32_t)g.n_units;
    for (size_t k = 0; k < g.models.size(); ++k) a.geom[k] = pl.gk[g.models[k]];
    for (int32_t i : g.idx) {
      const Request &r = p->st.req(req_ids[i]);
      DecReq &d = a.req[a.n_req++];
      // the KV plane of the entry's layer, or of the request's current layer
      d.pte_base = r.plane_base(layer ? layer[i] : r.cursor);
      a.ent_tag[a.n_req - 1] = tag ? tag[i] : 0u;
      d.ctx_len = (uint32_t)pl.attend[i];
      d.q_off = (uint32_t)pl.q_off[i];
      d.o_off = (uint32_t)pl.o_off[i];
      d.lse_off = (uint32_t)pl.l_off[i];
      d.ws_base = pl.ws_base[i];
      d.ws_orow = pl.ws_orow[i];
      d.unit_begin = pl.cost_prefix[i];
      d.chunk_pages = (uint16_t)(o.schedule == CP_SCHED_BALANCED ? pl.first_worker[i] : pl.chunk_pages[i]);
      d.n_chunks = (uint16_t)pl.n_slots[i];
      d.model = (uint8_t)(std::find(g.models.begin(), g.models.end(), r.model) - g.models.begin());
      d.n_hblk = (uint16_t)pl.hblk[i];
      if (app) {
        d.app_flags = (*app)[i].flags;
        d.app_off = (*app)[i].off;
        d.app_pte = (*app)[i].pte;
      }
    }
    const int v0 = __builtin_ctz(g.mask);
    const hipEvent_t ev0 = gi == 0 ? (hipEvent_t)o.ev_begin : nullptr;
    const hipEvent_t ev1 = gi + 1 == pl.groups.size() ? (hipEvent_t)o.ev_end : nullptr;
    hipError_t e = is_wide_variant(v0) ? launch_decode_wide(a, g.grid, v0, s, ev0, ev1)
                                       : launch_decode(a, g.grid, g.mask, s, ev0, ev1);
    if (e != hipSuccess) return hip_fail(e, "decode launch");
  }

  // Merge launches for split requests.
  MergeArgs ma{};
  ma.ws_o = pl.ws_o;
  ma.ws_l = pl.ws_l;
  ma.out = (uint16_t *)out;
  ma.lse = lse;
  auto flush = [&]() -> cp_status {
    if (ma.n_req == 0) return CP_OK;
    hipError_t e = launch_merge(ma, s);
    if (e != hipSuccess) return hip_fail(e, "merge launch");
    ma.n_req = 0;
    ma.n_blocks = 0;
    return CP_OK;
  };
  for (int32_t i = 0; i < n; ++i) {
    if (pl.ws_base[i] == kNoWs) continue;
    if (ma.n_req == kMaxReqPerLaunch) {
      cp_status rc = flush();
      if (rc) return rc;
    }
    const Geom &g = p->st.model(p->st.req(req_ids[i]).model);
    MergeReq &m = ma.req[ma.n_req++];
    m.block_begin = (uint32_t)ma.n_blocks;  // first merge workgroup of this request
    m.hq = (uint32_t)g.hq;
    m.d_v = (uint32_t)g.d_v;
    m.n_chunks = (uint32_t)pl.n_slots[i];
    m.ws_base = pl.ws_base[i];
    m.ws_orow = pl.ws_orow[i];
    m.o_off = (uint32_t)pl.o_off[i];
    m.lse_off = (uint32_t)pl.l_off[i];
    // one workgroup per (head, block of V columns)
    ma.n_blocks += g.hq * (int32_t)((uint32_t)g.d_v / merge_block_cols((uint32_t)g.d_v));
  }
  return flush();
}

// cp_attn_decode_step on a pool with device page stacks: a new token that
// opens a page takes that page, in every plane, from its model's stack
// inside the decode launch (fused_append / pop_new_pages). The host only
// counts: it refills stacks that would run short (a chunk's worth at a
// time, rarely) and marks the popped entries for reading back at the next
// slow-path call. A later layer's step finds its plane's entry already in
// the device page table.
cp_status step_device_pages(cp_pool *p, const DecodePlan &pl, int32_t n, const int32_t *req_ids,
                            const int32_t *n_new, const std::vector<int32_t> &placing, const void *rows,
                            const void *q, void *out, float *lse, void *hip_stream) {
  const int32_t P = p->st.page_tokens();
  std::vector<int64_t> need((size_t)p->st.n_models(), 0);
  std::vector<uint8_t> pops(n, 0);
  for (int32_t i = 0; i < n; ++i) {
    const Request &r = p->st.req(req_ids[i]);
    if (placing[i] && r.ctx_len % P == 0) {
      pops[i] = 1;
      need[(size_t)r.model] += r.layers;
    }
  }
  for (int32_t m = 0; m < p->st.n_models(); ++m)
    if (need[(size_t)m] > kStackCap - kStackRefill)
      return fail(CP_EINVAL, "a step opens %lld pages of model %d; a device page stack serves at most %d per step",
                  (long long)need[(size_t)m], m, kStackCap - kStackRefill);
  DeviceGuard g(p->device);
  hipStream_t s = (hipStream_t)hip_stream;
  cp_status rc = refill_stacks(p, need, s);
  if (rc) return rc;
  if (++p->epoch >= (1u << 31)) p->epoch = 1;  // pop states hold epoch << 1
  std::vector<AppendPlan> plan(n);
  uint64_t off = 0;
  for (int32_t i = 0; i < n; ++i) {
    if (!n_new[i]) continue;
    const Request &r = p->st.req(req_ids[i]);
    plan[i].flags = kAppRow;
    plan[i].off = (uint32_t)off;
    if (pops[i]) {
      p->st.begin_token_popped(req_ids[i], &p->pending);
      p->stk[(size_t)r.model].resize(p->stk[(size_t)r.model].size() - (size_t)r.layers);
      plan[i].flags |= kAppPop;
      plan[i].pte = (uint32_t)req_ids[i];
    } else if (placing[i]) {
      uint64_t first, count;
      p->st.begin_token(req_ids[i], &first, &count);  // the page exists: nothing to allocate
    }
    off += (uint64_t)p->st.model(r.model).row_elems;
  }
  rc = launch_plan(p, pl, n, req_ids, q, out, lse, hip_stream, rows, &plan);
  for (int32_t i = 0; i < n; ++i) p->st.advance(req_ids[i]);
  if (rc) {
    // the launch did not run: its pops never happened, so the host's view
    // of the stacks and page tables is no longer the device's
    p->broken = true;
    return rc;
  }
  return CP_OK;
}

// cp_attn_decode_layers: every KV layer of every request in one planned
// call. Launch entries are (request, layer) pairs, request-major, so the
// packed query, output and lse offsets the planner computes are [request]
// [layer][head] ones; entry (i, l) attends over plane l, and its last piece
// moves request i's device layer cursor on (piece_done).
cp_status decode_layers_impl(cp_pool *p, int32_t n, const int32_t *req_ids, const int32_t *n_new, const void *rows,
                             const void *q, void *out, float *lse, void *hip_stream, const cp_decode_opts *opts) {
  DecodePlan pl;
  cp_status rc = decode_prepare(p, n, req_ids, q, out, lse, opts, &pl.o, &pl.gk);
  if (rc) return rc;
  if (!n_new) return fail(CP_EINVAL, "null n_new");
  int64_t entries = 0;
  bool any = false;
  for (int32_t i = 0; i < n; ++i) {
    const Request &r = p->st.req(req_ids[i]);
    if (r.cursor != 0 || r.inflight)
      return fail(CP_ESTATE, "request %d has a token in flight at layer %d; finish it with cp_attn_decode_step first",
                  req_ids[i], r.cursor);
    if (n_new[i] != 0 && n_new[i] != 1)
      return fail(CP_EINVAL, "cp_attn_decode_layers appends 0 or 1 tokens per request (request %d: %d)", req_ids[i],
                  n_new[i]);
    if (r.ctx_len + n_new[i] < 1) return fail(CP_EINVAL, "request %d has an empty context", req_ids[i]);
    if (r.ctx_len + n_new[i] > 0xFFFFFFF0ll) return fail(CP_EINVAL, "context length overflow");
    if (!p->st.fits_reservation(req_ids[i], r.ctx_len + n_new[i]))
      return fail(CP_EINVAL, "request %d would grow past its reservation of %lld pages", req_ids[i],
                  (long long)r.reserve_pages);
    if ((uint32_t)req_ids[i] >= (1u << kTagLayerShift) || r.layers >= (1 << (32 - kTagLayerShift)))
      return fail(CP_EINVAL, "request id or layer count too large for an all-layer launch");
    entries += r.layers;
    any = any || n_new[i] != 0;
  }
  if (any && !rows) return fail(CP_EINVAL, "null rows");
  if (entries > (1 << 20)) return fail(CP_EINVAL, "too many (request, layer) entries in one call");
  const int32_t E = (int32_t)entries;
  std::vector<int32_t> eid(E), elayer(E), extra(E);
  std::vector<uint32_t> etag(E);
  uint64_t total_elems = 0;
  for (int32_t i = 0, k = 0; i < n; ++i) {
    const Request &r = p->st.req(req_ids[i]);
    for (int32_t l = 0; l < r.layers; ++l, ++k) {
      eid[k] = req_ids[i];
      elayer[k] = l;
      extra[k] = n_new[i];
      etag[k] = (uint32_t)req_ids[i] | ((uint32_t)r.layers << kTagLayerShift);
    }
    if (n_new[i]) total_elems += (uint64_t)r.layers * (uint64_t)p->st.model(r.model).row_elems;
  }
  if (total_elems > 0xFFFFFFFFull) return fail(CP_EINVAL, "too many rows in one call");
  rc = plan_decode(p, E, eid.data(), extra.data(), &pl);
  if (rc) return rc;
  rc = bind_pool_workspace(p, &pl);
  if (rc) return rc;
  DeviceGuard g(p->device);
  hipStream_t s = (hipStream_t)hip_stream;
  if (!any) return launch_plan(p, pl, E, eid.data(), q, out, lse, hip_stream, nullptr, nullptr, elayer.data(), etag.data());

  // New tokens: pages of every plane, from the host allocator (their
  // entries travel with the launch, one per entry) or from the device
  // stacks (one claim per request pops them all).
  const int32_t P = p->st.page_tokens();
  std::vector<uint8_t> opens(n, 0);
  std::vector<int64_t> need((size_t)p->st.n_models(), 0);
  for (int32_t i = 0; i < n; ++i) {
    const Request &r = p->st.req(req_ids[i]);
    if (n_new[i] && r.ctx_len % P == 0) {
      opens[i] = 1;
      need[(size_t)r.model] += r.layers;
    }
  }
  if (p->dev_pages) {
    for (int32_t m = 0; m < p->st.n_models(); ++m)
      if (need[(size_t)m] > kStackCap - kStackRefill)
        return fail(CP_EINVAL, "a call opens %lld pages of model %d; a device page stack serves at most %d per call",
                    (long long)need[(size_t)m], m, kStackCap - kStackRefill);
    rc = refill_stacks(p, need, s);
    if (rc) return rc;
    if (++p->epoch >= (1u << 31)) p->epoch = 1;
  } else {
    rc = prepare_growth(p, n, req_ids, n_new);
    if (rc) return rc;
  }
  std::vector<AppendPlan> plan(E);
  uint64_t off = 0;
  for (int32_t i = 0, k = 0; i < n; ++i) {
    const Request &r = p->st.req(req_ids[i]);
    const int32_t L = r.layers;
    const uint32_t row = (uint32_t)p->st.model(r.model).row_elems;
    const uint64_t pg = (uint64_t)(r.ctx_len / P);  // the new token's page
    if (!n_new[i]) {
      k += L;
      continue;
    }
    if (opens[i] && p->dev_pages) {
      p->st.begin_token_popped(req_ids[i], &p->pending);
      p->stk[(size_t)r.model].resize(p->stk[(size_t)r.model].size() - (size_t)L);
    } else {
      uint64_t first, count;
      p->st.begin_token(req_ids[i], &first, &count);
    }
    for (int32_t l = 0; l < L; ++l, ++k) {
      plan[k].flags = kAppRow;
      plan[k].off = (uint32_t)(off + (uint64_t)l * row);
      if (opens[i] && p->dev_pages) {
        plan[k].flags |= kAppPop;
        plan[k].pte = (uint32_t)req_ids[i];
      } else if (opens[i]) {
        plan[k].flags |= kAppPage;
        plan[k].pte = p->st.pte_mirror()[r.plane_base(l) + pg];
      }
    }
    off += (uint64_t)L * row;
  }
  rc = launch_plan(p, pl, E, eid.data(), q, out, lse, hip_stream, rows, &plan, elayer.data(), etag.data());
  for (int32_t i = 0; i < n; ++i) p->st.commit_token(req_ids[i]);
  if (rc) {
    // the launch did not run: its rows, and any popped page entries, are
    // missing on the device
    p->broken = true;
    return rc;
  }
  return CP_OK;
}

// The decode of cp_attn_decode_ex.
cp_status decode_impl(cp_pool *p, int32_t n, const int32_t *req_ids, const void *q, void *out, float *lse,
                      void *hip_stream, const cp_decode_opts *opts) {
  DecodePlan pl;
  cp_status rc = decode_prepare(p, n, req_ids, q, out, lse, opts, &pl.o, &pl.gk);
  if (rc) return rc;
  rc = plan_decode(p, n, req_ids, nullptr, &pl);
  if (rc) return rc;
  rc = bind_pool_workspace(p, &pl);
  if (rc) return rc;
  return launch_plan(p, pl, n, req_ids, q, out, lse, hip_stream, nullptr, nullptr);
}

}  // namespace

extern "C" {

cp_status cp_attn_decode(cp_pool *p, int32_t n, const int32_t *req_ids, const void *q, void *out, float *lse,
                         void *hip_stream) {
  return cp_attn_decode_ex(p, n, req_ids, q, out, lse, hip_stream, nullptr);
}

cp_status cp_attn_decode_noalloc(cp_pool *p, int32_t n, const int32_t *req_ids, const void *q, void *out, float *lse,
                                 void *hip_stream, const cp_decode_opts *opts) {
  DecodePlan pl;
  cp_status rc = decode_prepare(p, n, req_ids, q, out, lse, opts, &pl.o, &pl.gk);
  if (rc) return rc;
  rc = plan_decode(p, n, req_ids, nullptr, &pl);
  if (rc) return rc;
  // partial outputs first, then the partial lse values (256-byte aligned)
  const uint64_t o_bytes = (pl.ws_elems * sizeof(uint16_t) + 255) / 256 * 256;
  const uint64_t need = o_bytes + pl.ws_rows * sizeof(float);
  if (need > kNoAllocScratchBytes)
    return fail(CP_EINVAL,
                "the split plan needs %llu bytes of workspace; cp_attn_decode_noalloc has %llu (use fewer KV ranges: "
                "the queue or grid schedule with a smaller num_splits)",
                (unsigned long long)need, (unsigned long long)kNoAllocScratchBytes);
  if (pl.ws_rows) {
    DeviceGuard dg(p->device);
    void *base = nullptr;
    hipError_t e = scratch_device_address(p->device, &base);
    if (e != hipSuccess) return hip_fail(e, "address of the fixed split workspace");
    pl.ws_o = static_cast<uint16_t *>(base);
    pl.ws_l = reinterpret_cast<float *>(static_cast<uint8_t *>(base) + o_bytes);
  }
  return launch_plan(p, pl, n, req_ids, q, out, lse, hip_stream, nullptr, nullptr);
}

cp_status cp_attn_decode_layers(cp_pool *p, int32_t n, const int32_t *req_ids, const int32_t *n_new, const void *rows,
                                const void *q, void *out, float *lse, void *hip_stream, const cp_decode_opts *opts) {
  return decode_layers_impl(p, n, req_ids, n_new, rows, q, out, lse, hip_stream, opts);
}

cp_status cp_request_layer_state(cp_pool *p, int32_t req_id, int32_t *layer, int64_t *tokens) {
  if (!p || !layer || !tokens) return fail(CP_EINVAL, "null argument");
  if (!p->st.valid_open(req_id)) return fail(CP_EINVAL, "request %d is not open", req_id);
  if (p->host_only) return fail(CP_ESTATE, "host-only pool has no device state");
  DeviceGuard g(p->device);
  hipError_t e = hipDeviceSynchronize();
  uint32_t v[2] = {0u, 0u};
  if (e == hipSuccess) e = hipMemcpy(v, p->dev_layer + 2 * (uint64_t)req_id, 8, hipMemcpyDeviceToHost);
  if (e != hipSuccess) return hip_fail(e, "reading the request's layer cursor");
  *layer = (int32_t)v[0];
  *tokens = (int64_t)v[1];
  return CP_OK;
}

cp_status cp_attn_decode_step(cp_pool *p, int32_t n, const int32_t *req_ids, const int32_t *n_new, const void *rows,
                              const void *q, void *out, float *lse, void *hip_stream, const cp_decode_opts *opts) {
  DecodePlan pl;
  cp_status rc = decode_prepare(p, n, req_ids, q, out, lse, opts, &pl.o, &pl.gk);
  if (rc) return rc;
  if (!n_new) return fail(CP_EINVAL, "null n_new");
  bool any = false;
  for (int32_t i = 0; i < n; ++i) {
    if (n_new[i] != 0 && n_new[i] != 1)
      return fail(CP_EINVAL, "cp_attn_decode_step appends 0 or 1 rows per request (request %d: %d)", req_ids[i],
                  n_new[i]);
    const Request &r = p->st.req(req_ids[i]);
    if (r.cursor == 0) {
      // the first layer's step may place a new token
      if (r.ctx_len + n_new[i] < 1) return fail(CP_EINVAL, "request %d has an empty context", req_ids[i]);
      if (r.ctx_len + n_new[i] > 0xFFFFFFF0ll) return fail(CP_EINVAL, "context length overflow");
      if (!p->st.fits_reservation(req_ids[i], r.ctx_len + n_new[i]))
        return fail(CP_EINVAL, "request %d would grow past its reservation of %lld pages", req_ids[i],
                    (long long)r.reserve_pages);
    } else if (n_new[i] != r.inflight) {
      // later layers write the row of the token in flight, if there is one
      return fail(CP_EINVAL, "request %d is at layer %d of %d %s a token in flight: n_new must be %d", req_ids[i],
                  r.cursor, r.layers, r.inflight ? "with" : "without", r.inflight);
    }
    any = any || n_new[i] != 0;
  }
  if (any && !rows) return fail(CP_EINVAL, "null rows");
  uint64_t total_elems = 0;
  std::vector<int32_t> placing(n, 0);  // new tokens, placed at the first layer
  for (int32_t i = 0; i < n; ++i) {
    if (!n_new[i]) continue;
    const Request &r = p->st.req(req_ids[i]);
    total_elems += (uint64_t)p->st.model(r.model).row_elems;
    placing[i] = r.cursor == 0 ? 1 : 0;
  }
  if (total_elems > 0xFFFFFFFFull) return fail(CP_EINVAL, "too many rows in one call");
  // The whole launch is planned, checked and its workspace bound at the
  // lengths the step will attend over, before any page is allocated: a
  // refused call changes nothing.
  rc = plan_decode(p, n, req_ids, placing.data(), &pl);
  if (rc) return rc;
  rc = bind_pool_workspace(p, &pl);
  if (rc) return rc;
  auto advance_all = [&] {
    for (int32_t i = 0; i < n; ++i) p->st.advance(req_ids[i]);
  };
  if (!any) {
    rc = launch_plan(p, pl, n, req_ids, q, out, lse, hip_stream, nullptr, nullptr);
    if (rc == CP_OK) advance_all();
    return rc;
  }
  if (p->dev_pages) return step_device_pages(p, pl, n, req_ids, n_new, placing, rows, q, out, lse, hip_stream);
  rc = prepare_growth(p, n, req_ids, placing.data());
  if (rc) return rc;

  // Place new tokens (pages of every plane allocated on the host). The
  // entry of a new page of the current layer's plane travels with the
  // launch; a multi-layer model's other planes get theirs by one copy.
  DeviceGuard g(p->device);
  hipStream_t s = (hipStream_t)hip_stream;
  const int32_t P = p->st.page_tokens();
  std::vector<AppendPlan> plan(n);
  uint64_t off = 0, lo = UINT64_MAX, hi = 0, lo_rest = UINT64_MAX, hi_rest = 0;
  for (int32_t i = 0; i < n; ++i) {
    if (!n_new[i]) continue;
    const Request &r = p->st.req(req_ids[i]);
    if (placing[i]) {
      const int64_t used = r.pages_used;
      uint64_t first, count;
      p->st.begin_token(req_ids[i], &first, &count);
      if (count) {
        lo = std::min(lo, first);
        hi = std::max(hi, first + count);
        if (r.layers > 1) {
          lo_rest = std::min<uint64_t>(lo_rest, r.plane_base(1) + (uint64_t)used);
          hi_rest = std::max<uint64_t>(hi_rest, r.plane_base(r.layers - 1) + (uint64_t)r.pages_used);
        }
      }
    }
    plan[i].flags = kAppRow;
    plan[i].off = (uint32_t)off;
    if (r.ctx_len % P == 0) {  // the token in flight opens a page
      plan[i].flags |= kAppPage;
      plan[i].pte = p->st.pte_mirror()[r.plane_base(r.cursor) + (uint64_t)(r.ctx_len / P)];
    }
    off += (uint64_t)p->st.model(r.model).row_elems;
  }
  rc = push_ptes(p, lo_rest, hi_rest, s);
  if (rc == CP_OK) rc = launch_plan(p, pl, n, req_ids, q, out, lse, hip_stream, rows, &plan);
  if (rc) {
    // a HIP failure after the tokens were placed: keep the device pool in
    // step with the host tables by writing the new page entries and rows
    // the unfused way (rewriting a fused row is harmless)
    const std::string msg = cp_last_error();
    std::vector<AppItem> items;
    for (int32_t i = 0; i < n; ++i) {
      if (!n_new[i]) continue;
      const Request &r = p->st.req(req_ids[i]);
      items.push_back(AppItem{r.model, 1u, (uint32_t)r.ctx_len, r.plane_base(r.cursor), plan[i].off});
    }
    push_ptes(p, std::min(lo, lo_rest), std::max(hi, hi_rest), s);
    launch_appends(p, items, rows, s);
    advance_all();
    return fail(rc, "%s", msg.c_str());
  }
  advance_all();
  return CP_OK;
}

}  // extern "C"
