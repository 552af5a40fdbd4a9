// Kernel-argument records shared by the host launcher (api.cpp) and the
// kernels (kernels.hip). Everything a launch needs travels by value in the
// kernel-argument segment, so a decode step costs no host-to-device copy.
// Sizes stay well under the 4 KiB argument limit.
#pragma once
#include <stdint.h>

namespace cp {

constexpr int kMaxLaunchModels = 4;   // distinct models in one decode launch
constexpr int kMaxReqPerLaunch = 64;  // requests in one launch (at most one per lane of a wave)
constexpr uint32_t kNoWs = 0xFFFFFFFFu;
// Fixed split workspace of cp_attn_decode_noalloc, per GPU, in bytes.
constexpr uint64_t kNoAllocScratchBytes = 40ull << 20;
constexpr int kMaxScratchDevices = 64;
// Device free-page stacks (pools created with device_pages): entries per
// model; model m's stack is DecodeArgs::stack[m * kStackCap ...].
constexpr int32_t kStackCap = 8192;
// The host refills a stack with up to this many pages (a chunk's worth at
// most) when a step needs more than it holds.
constexpr int32_t kStackRefill = 1024;
enum : int32_t { kSchedBalanced = 0, kSchedQueue = 1, kSchedGrid = 2 };
// Balanced schedule: the fixed work of one piece (page-table and query
// loads, the latency of its first pages under a loaded memory system, the
// end merge and the partial write), in page-cost units (8 KiB of page
// bytes each): measured at about 23K cycles per piece on the narrow kernel,
// which streams about 600 cycles per unit. A request boundary that falls
// inside a workgroup's share is preceded by that much cost on the cost
// line, so the workgroup that runs a second piece there takes
// correspondingly fewer pages. DecReq::unit_begin is the cost position of
// the request's first page.
constexpr uint32_t kPieceFixedCost = 40;

// Decode code paths (GeomK::variant), chosen per model by the host.
//   Vector path (0-7): wavefront reductions; heads per block (16 or 8) and
//     V values per lane (8, 4, 2, 1); any geometry.
//   Small-group vector path (8-13): wavefront reductions for GQA/MHA with
//     1, 2 or 4 query heads per KV head and head_dim 64 or 128.
//   Narrow matrix path (16, 17, 19, 20, 23): 8, 16 or 32 query heads per KV
//     head (MLA latent head, or head_dim 128).
//   Wide matrix path (18, 21, 22): 64 or 128 query heads per KV head; its
//     own kernel (one workgroup per CU, scores split by heads, P.V by
//     columns).
enum : int32_t {
  kV16x8 = 0, kV16x4, kV16x2, kV16x1, kV8x8, kV8x4, kV8x2, kV8x1,
  kS_G1_D64 = 8, kS_G2_D64, kS_G4_D64, kS_G1_D128, kS_G2_D128, kS_G4_D128,
  kM_MLA_G16 = 16, kM_MLA_G32, kM_MLA_G128, kM_D128_G16, kM_D128_G32, kM_D128_G64, kM_D128_G128, kM_D128_G8
};
constexpr bool is_wide_variant(int v) { return v == kM_MLA_G128 || v == kM_D128_G64 || v == kM_D128_G128; }

// One piece of decode work: pages [pg_begin, pg_end) of a request, for one
// head block, writing partial slot `slot` when the request is split; model
// is the request's index into DecodeArgs::geom.
struct Seg {
  uint32_t pg_begin, pg_end, slot, hblk, model;
};

// Per-model geometry as the kernels see it.
struct GeomK {
  int32_t kind;        // 0 MLA, 1 GQA
  int32_t hq, hkv, g;  // g = hq / hkv
  int32_t d_k, d_v, row_elems, page_tokens;
  int32_t page_bytes;
  int32_t variant;     // kernel code path chosen by the host
  float scale_log2;    // softmax scale * log2(e)
  int32_t nb;          // head blocks per KV head (vector path)
  int32_t page_cost;   // relative work of one page (balanced schedule)
  int32_t pool_model;  // the model's id in the pool (its device page stack)
  int32_t layers;      // KV planes of a request of this model
};

// One request of a decode launch.
struct DecReq {
  uint32_t pte_base;  // first page-table entry of the request
  uint32_t ctx_len;   // tokens to attend over (>= 1)
  uint32_t q_off;     // bf16 element offset of the request's queries
  uint32_t o_off;     // bf16 element offset of its outputs
  uint32_t lse_off;   // float offset of its log-sum-exp values
  uint32_t ws_base;   // first partial lse row (kNoWs when the request is not split)
  uint32_t ws_orow;   // partial outputs start at element offset ws_orow * d_v
  uint32_t unit_begin;   // queue/grid: first unit; balanced: cost position of the request's first page
  uint16_t chunk_pages;  // queue/grid: pages per KV range; balanced: first worker of the request
  uint16_t n_chunks;     // KV ranges = partial slots
  uint8_t model;         // index into DecodeArgs::geom
  uint8_t app_flags;     // fused append: kAppRow (the last context token is a new row at
                         // DecodeArgs::rows + app_off), kAppPage (its page is new: app_pte),
                         // kAppPop (its page is new and comes from the model's device
                         // stack, one page per plane; app_pte is then the request id)
  uint16_t n_hblk;       // head blocks per KV range
  uint32_t app_off;      // element offset of the new row in DecodeArgs::rows
  uint32_t app_pte;      // page-table entry of the new row's page when kAppPage is set
};
enum : uint8_t { kAppRow = 1, kAppPage = 2, kAppPop = 4 };

struct DecodeArgs {
  uint8_t *pool;          // written only by the fused append
  uint32_t *pte;          // written only by the fused append (a new page's entry)
  const uint16_t *rows;   // fused append: new logical rows, packed in call order
  const uint16_t *q;
  uint16_t *out;
  float *lse;
  uint16_t *ws_o;     // partial outputs, [row][d_v] bf16, normalised
  float *ws_l;        // partial log-sum-exp, [row], natural log
  uint32_t *queue;    // queue schedule: {next unit, finished workgroups}
  // device page stacks (kAppPop): entries and per-model counts, per-request
  // pop state ((epoch << 1) | done) and per request id {first page-table
  // entry, entries per plane}
  const uint32_t *stack;
  int32_t *stack_top;
  uint32_t *pop_state;
  const uint32_t *req_geo;
  uint32_t epoch;  // this launch's pop epoch (>= 1)
  uint32_t pad0;
  // All-layer launches (cp_attn_decode_layers): a request's layer cursor
  // and the tokens its cursor has carried through every layer (both at
  // index 2 * request id), and per launch entry the pieces finished so far
  // (reset by the last one). ent_tag[r] is request id | layers << 20 for an
  // entry whose completion moves a cursor, 0 otherwise.
  uint32_t *layer_cursor;
  uint32_t *layer_tokens;
  uint32_t *entry_done;
  int32_t n_req, n_units;
  int32_t schedule;     // kSchedBalanced, kSchedQueue or kSchedGrid
  uint32_t total_cost;  // balanced: summed page costs of the launch
  GeomK geom[kMaxLaunchModels];
  DecReq req[kMaxReqPerLaunch];
  uint32_t ent_tag[kMaxReqPerLaunch];
};
constexpr uint32_t kTagLayerShift = 20;

// V columns one merge workgroup covers: 64 lanes of up to four columns
// (d_v is 64, 128, 256 or 512).
constexpr uint32_t merge_block_cols(uint32_t d_v) { return d_v >= 256 ? 256u : d_v; }

struct MergeReq {
  uint32_t block_begin;  // first merge workgroup of this request
  uint32_t hq, d_v, n_chunks;
  uint32_t ws_base, ws_orow, o_off, lse_off;
};

struct MergeArgs {
  const uint16_t *ws_o;
  const float *ws_l;
  uint16_t *out;
  float *lse;
  int32_t n_req, n_blocks, pad0, pad1;  // n_blocks: merge workgroups
  MergeReq req[kMaxReqPerLaunch];
};

struct AppReq {
  uint64_t src_off;    // bf16 element offset of the request's first row in the input
  uint32_t row_begin;  // first grid row of this request in the launch
  uint32_t n_new;
  uint32_t old_len;
  uint32_t pte_base;
  uint32_t model;
  uint32_t pad;
};

struct AppendArgs {
  uint8_t *pool;
  const uint32_t *pte;
  const uint16_t *rows;
  int32_t n_req, total_rows, pad0, pad1;
  GeomK geom[kMaxLaunchModels];
  AppReq req[kMaxReqPerLaunch];
};

struct GatherArgs {
  const uint8_t *pool;
  const uint32_t *pte;
  uint16_t *dst;
  uint32_t pte_base, start, n_tok, pad;
  GeomK geom;
};

// Refill of a device page stack: n entries written at dst[0..n), then the
// model's count set to new_top. The entries travel in the arguments, so the
// host keeps no staging copy alive.
constexpr int32_t kStackPushMax = 640;
struct StackPushArgs {
  uint32_t *dst;
  int32_t *top;
  int32_t n, new_top;
  uint32_t ent[kStackPushMax];
};

static_assert(kMaxReqPerLaunch <= 64, "request lookups search one key per lane");
static_assert(sizeof(StackPushArgs) <= 3072, "stack push arguments too large");
// the argument segment (with the runtime's hidden arguments) stays under 4 KiB
static_assert(sizeof(DecodeArgs) <= 3776, "decode kernel arguments too large");
static_assert(sizeof(MergeArgs) <= 3072, "merge kernel arguments too large");
static_assert(sizeof(AppendArgs) <= 3072, "append kernel arguments too large");

}  // namespace cp
