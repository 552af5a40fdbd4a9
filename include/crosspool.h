/*
 * crosspool.h -- C ABI of a shared, virtualised KV-cache pool with batched
 * decode attention, for AMD Instinct MI355X (gfx950).
 *
 * The operations follow the KV-cache pool of CrossPool (arXiv 2606.24506):
 *   - one pool whose size is a page budget shared by several cold models
 *     (Section 3.1, planner output "pool page budget"; Section 4);
 *   - per-model KV geometry, i.e. per-token KV bytes kappa(M) that differ
 *     between MLA, MQA and GQA models (Section 2.3 C1; Section 3.1);
 *   - a paged logical KV interface in front of physical pages that the
 *     virtualizer places, with page mapping kept off the per-token path
 *     (Section 3.1, last paragraph; Section 4, KV-cache virtualization);
 *   - admission that queues or rejects new requests when the budget is
 *     exhausted and never interrupts admitted ones, whose pages live until
 *     they finish (Section 3.1; Section 4);
 *   - attention run next to the KV, reading it at every decode step
 *     (Section 2.3 C2).
 *
 * Conventions for every call:
 *   - Return value: CP_OK (0) or a negative cp_status. No call aborts or
 *     throws. cp_last_error() gives a thread-local message for the last
 *     failure on the calling thread.
 *   - All argument and capacity checks run on the host before anything is
 *     enqueued; on any error they report, no pool state changes
 *     (all-or-nothing across a whole batch). A HIP failure after the checks
 *     (CP_EHIP from a copy or launch of an append or decode step) leaves
 *     the host tables updated as if the call had succeeded; the device
 *     state is then undefined and the pool should be closed.
 *   - Device-memory arguments are device pointers on the pool's device;
 *     host arguments are ordinary host pointers and are not retained after
 *     the call returns. Streams are hipStream_t passed as void* (NULL = the
 *     default stream).
 *   - Calls that enqueue GPU work (append, decode, gather) return once the
 *     work is enqueued; host-side metadata (context lengths, page tables) is
 *     already updated at return, so append-then-decode on one stream is
 *     ordered. Launch failures return CP_EHIP; device faults surface at the
 *     caller's next synchronisation.
 *   - A pool is not thread-safe: the caller serialises calls on one pool.
 *     Decode calls on one pool must not overlap on the GPU (one stream, or
 *     the caller orders streams), because they share the pool's workspace.
 *     Different pools share no device state: their calls may run at the
 *     same time on different streams (two batches in flight, Section 3.2).
 *     cp_attn_decode_noalloc is the exception: its workspace is per GPU.
 *   - bf16 is IEEE-754 binary32 truncated to its upper 16 bits; values are
 *     produced with round-to-nearest-even.
 */
#ifndef CROSSPOOL_H
#define CROSSPOOL_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t cp_status;
enum {
  CP_OK = 0,
  CP_EINVAL = -1, /* bad argument, unknown id, out-of-range value */
  CP_ENOMEM = -2, /* device or host allocation failed */
  CP_ENOSPC = -3, /* pool page budget exhausted (admission reject) */
  CP_EHIP = -4,   /* a HIP runtime call failed */
  CP_ESTATE = -5  /* call not valid in the current state */
};

/* Message for the last failing call on this thread ("" if none). The
 * returned string stays valid until the next failing call on this thread. */
const char *cp_last_error(void);

/* Library version, (major << 16) | minor. */
int32_t cp_version(void);

/* ------------------------------------------------------------------ pool */

typedef struct cp_pool cp_pool; /* opaque */

/* Where the pool's pages live (Section 3.1, "KV-cache Planner and
 * Virtualizer"; Section 4, KV-cache virtualization). */
typedef enum {
  /* One device buffer of pool_bytes (allocated, or device_mem), carved
   * into chunks; all of it is held for the pool's lifetime. */
  CP_BACKING_BUFFER = 0,
  /* Virtualized: the pool reserves address space only, one range of
   * pool_bytes per model (at most 16 models, and at most 1 TiB in all,
   * which caps the models of budgets above 64 GiB), and maps physical
   * allocations of chunk_bytes into a model's range on demand: when a
   * request is admitted, enough chunks to back its whole reservation; at
   * close, chunks that no open reservation of the model needs any more are
   * unmapped and their memory returned to the device. Mapping stays on the
   * admission and release slow paths: appends and decode steps never map.
   * The budget limits the chunks mapped at once. Kernels see the same
   * page-table interface as with a buffer. chunk_bytes must be a multiple
   * of the device's mapping granularity; placement_seed is ignored (the
   * driver places physical memory); device_mem must be NULL. The mapping
   * calls wait for the device to finish queued work. */
  CP_BACKING_VIRTUAL = 1
} cp_backing;

typedef struct {
  /* Tokens per page, pool-wide (64 in the shipped workloads). A page of a
   * model with kappa bytes per token holds page_tokens * kappa bytes. */
  int32_t page_tokens;
  /* HIP device ordinal, or -1 for a host-only pool: all bookkeeping
   * (admission, page allocation, page tables) works, no device memory is
   * touched, and append must pass rows == NULL; decode and gather return
   * CP_ESTATE. Used to test the allocator without a GPU. */
  int32_t device;
  /* KV budget in bytes; rounded down to whole chunks. This is the shared
   * page budget the planner emits (Section 3.1). */
  uint64_t pool_bytes;
  /* Allocation unit carved into pages of one model at a time; 0 means
   * 2 MiB. Must be a multiple of 256. A model whose page does not fit in a
   * chunk cannot be registered. */
  uint64_t chunk_bytes;
  /* 0: chunks are handed out in ascending address order. Otherwise each
   * new chunk is drawn uniformly at random from the free chunks with a
   * generator seeded by this value, so physical placement is scattered
   * and reproducible. Logical results never depend on placement. */
  uint64_t placement_seed;
  /* Optional caller-owned device buffer of at least pool_bytes (after
   * rounding), 256-byte aligned; it must outlive the pool. NULL: the pool
   * allocates and owns its buffer. */
  void *device_mem;
  /* Maximum number of simultaneously open requests; 0 means 4096. */
  int32_t max_requests;
  int32_t backing; /* cp_backing */
  /* Cap on the device memory the pool may hold for split-KV partial
   * results (the per-range outputs and lse values a long request's decode
   * merges); 0 means no cap. A decode whose split plan needs more fails
   * with CP_ENOMEM before anything is enqueued or any state changes; the
   * queue and grid schedules with num_splits = 1 need none. */
  uint64_t max_workspace_bytes;
  /* 0: cp_attn_decode_step allocates a new token's pages on the host and
   * passes their page-table entries in the launch. 1: each model has a
   * free-page stack in device memory, and the step's launch pops a new
   * token's pages (one per KV plane) from it and writes their entries into
   * the device page table itself (Section 3.3, control lowering; the
   * per-token path then does no host page bookkeeping). The host refills a
   * stack, with up to a chunk's worth of pages, before a step that would
   * empty it; pages in a stack count against their model's reservations.
   * The host copy of the popped entries is read back, waiting for the
   * device, at the next cp_request_pages, cp_request_close or cp_kv_append;
   * a close also returns stack pages no open reservation can still use.
   * Results do not depend on this setting. A step may open at most 7168
   * pages of one model (requests times planes). */
  int32_t device_pages;
} cp_pool_desc;

/* Create a pool. Errors: CP_EINVAL (page_tokens not in [1, 4096],
 * chunk_bytes not a multiple of 256, fewer than one chunk, an unknown
 * backing, a virtual pool on a device without virtual memory management
 * or with chunk_bytes off its mapping granularity), CP_ENOMEM (device or
 * pinned-host allocation, or the address reservation, failed), CP_EHIP. */
cp_status cp_pool_create(const cp_pool_desc *desc, cp_pool **out);

/* Destroy a pool and free what it owns. CP_ESTATE if requests are still
 * open. The caller must have synchronised every stream used with it. */
cp_status cp_pool_destroy(cp_pool *pool);

typedef struct {
  uint64_t chunks_total;   /* whole chunks in the budget */
  uint64_t chunks_used;    /* chunks currently carved for some model
                              (mapped, for a virtual pool) */
  uint64_t pages_used;     /* pages holding KV of open requests */
  uint64_t pages_reserved; /* pages promised to open requests */
  int32_t requests_open;
  int32_t models;
  uint64_t span_bytes;     /* address range page entries point into */
  int32_t backing;         /* cp_backing */
  int32_t max_models;      /* models the pool can register */
} cp_pool_stats_t;

cp_status cp_pool_stats(cp_pool *pool, cp_pool_stats_t *out);

/* ---------------------------------------------------------------- models */

typedef enum {
  CP_KIND_MLA = 0, /* one latent KV head: row = [latent | rope]; V = latent */
  CP_KIND_GQA = 1  /* n_kv_heads K and V heads; MQA is n_kv_heads = 1 */
} cp_kind;

typedef enum { CP_BF16 = 0 } cp_dtype;

typedef struct {
  int32_t kind;        /* cp_kind */
  int32_t n_q_heads;   /* query heads per layer */
  int32_t n_kv_heads;  /* MLA: must be 1; GQA: divides n_q_heads */
  int32_t head_dim;    /* GQA: K and V width per KV head; MLA: ignored */
  int32_t latent_dim;  /* MLA: latent width (also the V width) */
  int32_t rope_dim;    /* MLA: decoupled rope width; K width = latent + rope */
  float softmax_scale; /* > 0; 0 means 1/sqrt(head_dim) for GQA (required for MLA) */
  int32_t dtype;       /* cp_dtype; only CP_BF16 */
  /* Attention layers whose KV the pool holds, in [1, 1024]; 0 means 1.
   * Each layer has its own KV plane: a request owns one page set per layer,
   * all holding the same token positions, and a decode step reads the
   * plane of the request's current layer (Section 3.2, layer cursor). The
   * geometry above is that of one layer; the budget counts every plane. */
  int32_t n_layers;
} cp_model_desc;

/* Register the KV geometry of one attention layer of a model (Section 2.3
 * C1: models differ in KV layout, KV heads and per-token KV bytes). Sets
 * *model_id. Limits: n_q_heads in [1, 256]; V width in {64, 128, 256, 512};
 * K width a multiple of 8 and at most 1024; per-token bytes at least 128.
 * Errors: CP_EINVAL (geometry outside the limits, page larger than a chunk,
 * too many models: at most 16). */
cp_status cp_model_register(cp_pool *pool, const cp_model_desc *m, int32_t *model_id);

typedef struct {
  int32_t d_k, d_v;          /* K and V width per head */
  int32_t kappa;             /* KV bytes per token */
  int32_t page_bytes;        /* page_tokens * kappa */
  int32_t pages_per_chunk;   /* pages carved from one chunk */
  int32_t row_elems;         /* bf16 elements in one logical row */
  int32_t n_layers;          /* KV planes per request */
} cp_model_info_t;

cp_status cp_model_info(cp_pool *pool, int32_t model_id, cp_model_info_t *out);

/* -------------------------------------------------------------- requests */

/* Admit a request of model_id that will hold at most reserve_tokens tokens
 * (prompt plus generated). Admission reserves ceil(reserve_tokens /
 * page_tokens) pages against the shared budget; it succeeds only if the
 * budget can hold every open reservation of every model at once, so an
 * admitted request is never refused a page later (Section 3.1: admission
 * queues or rejects new requests rather than interrupting active decodes).
 * On a virtual pool the reservation's chunks are mapped here. Sets
 * *req_id. Errors: CP_ENOSPC (budget exhausted: nothing changed, the
 * caller may queue and retry), CP_ENOMEM (a virtual pool could not map the
 * memory: nothing changed), CP_EINVAL. */
cp_status cp_request_open(cp_pool *pool, int32_t model_id, int64_t reserve_tokens, int32_t *req_id);

/* Release a request: its pages go back to its model's slab, chunks that
 * become empty go back to the shared budget, and its reservation ends
 * (Section 3.1: pages are kept until the request finishes). The caller
 * must have synchronised every stream with work on this request. On a
 * virtual pool, a chunk that empties is unmapped, after one device-wide
 * synchronisation per call. */
cp_status cp_request_close(cp_pool *pool, int32_t req_id);

/* Committed tokens of the request: those present in every layer's plane
 * (a token in flight through the layers is not counted until its last
 * layer's decode step). */
cp_status cp_request_len(cp_pool *pool, int32_t req_id, int64_t *ctx_len);

/* The request's layer cursor (Section 3.2): the layer its next decode step
 * reads, in [0, n_layers), and whether a new token is in flight (placed at
 * the first layer's step, committed after the last layer's). */
cp_status cp_request_cursor(cp_pool *pool, int32_t req_id, int32_t *layer, int32_t *in_flight);

/* Copy the request's page-table entries of pages [first, first + count) to
 * host memory, for every layer: ptes is [n_layers][count]. An entry is the
 * byte offset of the page inside the pool's address span, shifted right by
 * 8. For tests and debugging. */
cp_status cp_request_pages(cp_pool *pool, int32_t req_id, int64_t first, int64_t count, uint32_t *ptes);

/* ------------------------------------------------------------------- KV */

/* Append n_new[i] tokens to request req_ids[i], i < n, scattering their KV
 * rows into pool pages through the page table (Section 3.1: attention sees
 * a normal paged interface while physical pages are mapped on demand).
 *
 * rows: device memory, the requests' logical rows packed in call order,
 *   request i contributing n_layers * n_new[i] rows: [n_layers][n_new[i]]
 *   (layer-major; one layer for single-layer models). A logical row is
 *   row_elems bf16 values: MLA [latent | rope]; GQA/MQA [K head 0 .. K head
 *   Hkv-1 | V head 0 .. V head Hkv-1], each head head_dim wide. Rows are
 *   copied bit for bit. The tokens are committed at once in every layer, so
 *   a request with a token in flight (cursor past the first layer) cannot
 *   append (CP_EINVAL).
 * req_ids, n_new: host arrays of n entries; req_ids must be distinct;
 *   n_new[i] >= 0.
 * New pages come from the model's slab, or a fresh chunk of the shared
 *   budget; their page-table entries are written before the copy runs.
 * Errors: CP_EINVAL (unknown or duplicate id, negative count, growth past
 *   the reservation, rows == NULL on a device pool), CP_EHIP. */
cp_status cp_kv_append(cp_pool *pool, int32_t n, const int32_t *req_ids, const int32_t *n_new,
                       const void *rows, void *hip_stream);

/* Batched decode attention over the pool (Section 2.3 C2: attention stays
 * local to the KV and reads all of it at every decode step). Requests may
 * belong to different models. For request i with context n_i >= 1 and every
 * query head h (GQA groups are contiguous: head h reads KV head
 * h / (n_q_heads / n_kv_heads)):
 *     s_j = scale * <q_h, K_j>, j < n_i;  out_h = sum_j softmax(s)_j V_j;
 *     lse_h = ln sum_j exp(s_j)  (natural log).
 * q: device, per request [n_q_heads][d_k] bf16, packed in call order (MLA
 *   queries are the absorbed form: latent part already multiplied through
 *   the key up-projection, rope part post-rotary).
 * out: device, per request [n_q_heads][d_v] bf16, packed in call order.
 * lse: device, per request [n_q_heads] float, packed in call order.
 * req_ids: host array of n distinct ids, n >= 1.
 * Accumulation is fp32; outputs depend only on the logical KV, never on
 * the physical placement of pages (bit-identical across placements). For a
 * multi-layer model, K and V are those of the request's current layer
 * (cp_request_cursor) and the context includes a token in flight; this call
 * does not move the cursor.
 * Errors: CP_EINVAL (unknown or duplicate id, empty context), CP_ESTATE
 * (host-only pool), CP_ENOMEM (workspace growth failed), CP_EHIP. */
cp_status cp_attn_decode(cp_pool *pool, int32_t n, const int32_t *req_ids, const void *q, void *out, float *lse,
                         void *hip_stream);

typedef enum {
  CP_PATH_AUTO = 0, /* matrix cores where many query heads share a KV head, vector otherwise */
  CP_PATH_VALU = 1, /* force the vector (wavefront-reduction) kernel for every model */
  CP_PATH_MFMA = 2  /* force the matrix-core kernel for every model */
} cp_path;

typedef enum {
  /* Persistent grid, one workgroup per CU slot; the launch's pages, in
   * request order, are cut into equal-cost contiguous ranges, one per
   * workgroup, so ragged contexts and mixed models balance to within one
   * page. A request spanning several ranges is merged afterwards. */
  CP_SCHED_BALANCED = 0,
  /* Persistent grid whose workgroups pull (request, KV range) units from a
   * device queue, costliest first. */
  CP_SCHED_QUEUE = 1,
  /* One workgroup per (request, KV range) unit. */
  CP_SCHED_GRID = 2
} cp_schedule;

typedef struct {
  /* Queue and grid schedules: 0 lets the planner split each request's
   * context into page-aligned KV ranges; k >= 1 forces min(k, pages)
   * ranges per request. Must be 0 with the balanced schedule. */
  int32_t num_splits;
  int32_t schedule; /* cp_schedule; opts == NULL means CP_SCHED_BALANCED */
  int32_t path;     /* cp_path */
  int32_t reserved0;
  /* Optional hipEvent_t handles (created with timing enabled) that take
   * the start time of the first and the end time of the last attention
   * kernel of the call, from those launches themselves (no separate
   * marker in the stream); the split merge is not included. */
  void *ev_begin;
  void *ev_end;
} cp_decode_opts;

/* cp_attn_decode with options; opts == NULL behaves like cp_attn_decode. */
cp_status cp_attn_decode_ex(cp_pool *pool, int32_t n, const int32_t *req_ids, const void *q, void *out, float *lse,
                            void *hip_stream, const cp_decode_opts *opts);

/* Size in bytes of the fixed split workspace of cp_attn_decode_noalloc. */
#define CP_NOALLOC_WORKSPACE_BYTES (40u * 1024u * 1024u)

/* cp_attn_decode_ex for callers that cannot allocate device memory: code
 * under HIP graph capture, tight serving loops, and harnesses that forbid
 * allocation. Same arguments, kernels, split plans and results (out and lse
 * bit-identical to cp_attn_decode_ex with the same opts), but the split
 * workspace (the partial outputs and lse values of requests decoded over
 * several KV ranges) is a fixed device array of CP_NOALLOC_WORKSPACE_BYTES
 * that each GPU the library runs on holds until the process ends, instead
 * of the pool's growable workspace: the call makes no hipMalloc or hipFree
 * and no other device allocation. The caller still passes q, out and lse.
 * A plan needing more than that (partial outputs: 2 * n_q_heads * d_v bytes
 * per KV range of each split request, plus 4 * n_q_heads for lse) fails
 * with CP_EINVAL before anything is enqueued; the DeepSeek-V3-shaped batch
 * (8 x 128K tokens, 128 heads) and the 512K-token burst need about 35 MB.
 * The array is shared by every call on one GPU, whichever pool it is on,
 * and keeps the last call's contents (nothing in it needs clearing):
 * noalloc calls on one GPU must not overlap on the device (one stream, or
 * the caller orders them); overlapping calls race on the workspace. */
cp_status cp_attn_decode_noalloc(cp_pool *pool, int32_t n, const int32_t *req_ids, const void *q, void *out,
                                 float *lse, void *hip_stream, const cp_decode_opts *opts);

/* One decode step with single-token appends: the effect of cp_kv_append(pool,
 * n, req_ids, n_new, rows, hip_stream) followed by cp_attn_decode_ex(pool, n,
 * req_ids, q, out, lse, hip_stream, opts), with the same arguments, layouts
 * and results (out and lse bit-identical), but without the append launch
 * and the page-table copy: the attention launches write the new rows and
 * page-table entries themselves. This lowers the per-token host control of
 * the pool's decode step into the device launch (Section 4, control
 * lowering).
 *
 *   n_new   host, n entries, each 0 or 1 (a decode step appends at most the
 *           token just generated).
 *   rows    device, the new logical rows packed in call order (requests with
 *           n_new = 0 contribute none); may be NULL when every n_new is 0.
 *
 * Pages for the new tokens are allocated on the host as in cp_kv_append; the
 * entry of a new page is passed to the launch, and every workgroup that reads
 * a request's last page writes that entry and the new row before reading it.
 *
 * Multi-layer models (Section 3.2, layer-wise pipeline: each batch keeps its
 * own layer cursor, and requests of different models at different layers
 * share one launch): a step serves each request at its current layer and
 * then moves the cursor on. At the first layer, n_new = 1 places a new token
 * (pages of every layer's plane are allocated; a multi-layer model's other
 * planes get their new entries by one page-table copy) and its row of that
 * layer is written; at later layers n_new must be 1 while the token is in
 * flight (its row of that layer) and 0 otherwise. The token is committed
 * after the last layer's step. A single-layer model commits at once, which
 * is the behaviour described above.
 * With device_pages (cp_pool_desc), a new token's pages are popped from the
 * model's device stack inside the launch instead (all planes at the first
 * layer's step).
 * Errors: those of cp_kv_append and cp_attn_decode_ex, plus CP_EINVAL for an
 * n_new other than 0 or 1 or not matching the token in flight. Argument and
 * capacity checks run before any state changes; if the attention launch
 * fails once pages are allocated, the rows are still appended (as by
 * cp_kv_append), the cursors move on, and the error is returned (with
 * device_pages the pool is then unusable: later calls return CP_ESTATE). */
cp_status cp_attn_decode_step(cp_pool *pool, int32_t n, const int32_t *req_ids, const int32_t *n_new,
                              const void *rows, const void *q, void *out, float *lse, void *hip_stream,
                              const cp_decode_opts *opts);

/* One token step through every KV layer of the requests' models in one
 * planned call (Section 3.2, layer-wise pipeline: the layer cursor of each
 * in-flight request is advanced by the launch itself as its layers
 * complete). For each request i and layer l in [0, n_layers(i)) it has the
 * effect of a cp_attn_decode_step at layer l with that layer's query and
 * row, with the same results bit for bit; the work of all layers is spread
 * over one launch per kernel family (KV planes of different layers are
 * independent inputs here: the FFN stage between layers is outside this
 * library).
 *
 *   n_new  host, n entries, each 0 or 1; every request must be at layer 0
 *          with no token in flight (CP_ESTATE otherwise).
 *   rows   device, bf16; for each request with n_new = 1, in call order,
 *          its new token's rows of every layer: [n_layers][row_elems].
 *   q      device, bf16: per request in call order, [n_layers][n_q_heads]
 *          [d_k]; out [n_layers][n_q_heads][d_v] and lse [n_layers]
 *          [n_q_heads] likewise.
 *
 * On the device, the last piece of work of each (request, layer) moves the
 * request's layer cursor on; the one that completes the last layer sets it
 * back to 0 and counts the new token as carried through every layer
 * (cp_request_layer_state). On the host the token is committed when the
 * call returns. New pages come from the host allocator, or from the device
 * stacks (device_pages: one pop per request covers every plane). Errors: as
 * cp_attn_decode_step; the per-request limits of an all-layer launch are
 * request ids below 2^20 and fewer than 4096 layers. If the launch fails
 * after pages were allocated, the pool is unusable (CP_ESTATE). */
cp_status cp_attn_decode_layers(cp_pool *pool, int32_t n, const int32_t *req_ids, const int32_t *n_new,
                                const void *rows, const void *q, void *out, float *lse, void *hip_stream,
                                const cp_decode_opts *opts);

/* The device-side layer state that cp_attn_decode_layers launches drive:
 * the layer cursor (layers of the current all-layer step completed; 0 when
 * none is running) and the tokens carried through every layer since the
 * request was opened. Waits for the device. For tests and monitoring.
 * Errors: CP_EINVAL, CP_ESTATE (host-only pool), CP_EHIP. */
cp_status cp_request_layer_state(cp_pool *pool, int32_t req_id, int32_t *layer, int64_t *tokens);

/* Copy logical rows [start, start + n_tok) of one request out of the pool
 * into dst (device, [n_layers][n_tok][row_elems] bf16), through the same
 * page-table translation that decode uses. Bit-exact inverse of
 * cp_kv_append. Errors: CP_EINVAL (range outside the committed [0,
 * ctx_len)), CP_ESTATE (host-only pool), CP_EHIP. */
cp_status cp_kv_gather(cp_pool *pool, int32_t req_id, int64_t start, int64_t n_tok, void *dst, void *hip_stream);

/* ---------------------------------------------------------------------
 * KV-cache planner (Section 3.1, "KV-cache Planner and Virtualizer",
 * Eq. 1-2): the pool budget for cp_pool_desc.pool_bytes, host only.
 *
 * Request i of a model arrives at A_i with prompt tokens O_p,i, output
 * tokens O_d,i and decode residence time T_i; its active KV at age u is
 * kappa * (O_p,i + O_d,i * u / T_i) for 0 <= u < T_i and 0 otherwise
 * (Eq. 1); the pool demand at time t is the sum over the requests of every
 * model (Eq. 2). The planner draws Poisson arrivals of rate arrival_rate per
 * model over [0, horizon_s), each taking one whole trace record (keeping the
 * correlations between the three quantities), evaluates the demand at n_obs
 * observation times uniform over [W, horizon_s) (W: the longest residence
 * time in any trace), and takes the quantile as the order statistic of rank
 * ceil(quantile * n_obs). The budget is that quantile rounded up to whole
 * chunk_bytes units. Random draws: SplitMix64 (Steele, Lea and Flood, 2014)
 * seeded with `seed`, in the order inter-arrival uniform, record uniform per
 * arrival, model by model, then the observation uniforms.
 * ------------------------------------------------------------------- */
typedef struct {
  double         kappa_bytes;     /* kappa(M): KV bytes per token, > 0 */
  double         arrival_rate;    /* lambda_M: requests per second, > 0 */
  int64_t        n_samples;       /* trace records, >= 1 */
  const int64_t *prompt_tokens;   /* host, n_samples entries, >= 0 */
  const int64_t *output_tokens;   /* host, n_samples entries, >= 0 */
  const double  *service_time_s;  /* host, n_samples entries: residence time T, > 0 */
} cp_plan_model;
typedef struct {
  double   horizon_s;    /* simulated window; must exceed every residence time */
  int64_t  n_obs;        /* observation times, >= 1 */
  double   quantile;     /* provisioning quantile in (0, 1], e.g. 0.95 or 0.99 */
  uint64_t seed;
  uint64_t chunk_bytes;  /* rounding unit of the budget (the pool's allocator chunk) */
} cp_plan_opts;
typedef struct {
  double   quantile_bytes;  /* the demand quantile */
  double   mean_bytes;      /* mean demand over the observations */
  double   max_bytes;       /* largest observed demand */
  uint64_t pool_bytes;      /* quantile_bytes rounded up to whole chunk_bytes */
  int64_t  n_arrivals;      /* simulated requests */
} cp_plan_result;
/* models: host array of n_models descriptors (not retained). Errors:
 * CP_EINVAL (empty or non-positive inputs, horizon not past the longest
 * residence time, more than 1e8 expected arrivals for a model). */
cp_status cp_plan_pool(const cp_plan_model *models, int32_t n_models, const cp_plan_opts *opts, cp_plan_result *out);

#ifdef __cplusplus
}
#endif

#endif /* CROSSPOOL_H */
