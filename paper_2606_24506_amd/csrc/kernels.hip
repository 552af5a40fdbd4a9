// gfx950 kernels of the shared KV pool: KV append (scatter through the page
// table), gather (the inverse), decode attention, and the split-KV merge.
//
// Page-internal layouts (one page = page_tokens tokens of one model):
//   MLA      token-major [P][d_k] bf16: a page is the request's logical rows
//            for those tokens, back to back; V is the first d_v of each row.
//   GQA/MQA  head-major [Hkv][ K: P x d | V: P x d ] bf16, so the K (or V)
//            rows of one KV head inside one page are one contiguous block.
// A page starts at pool + (pte << 8).
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <mutex>
#include <type_traits>

#include "decode_mfma.h"
#include "decode_narrow.h"
#include "decode_small.h"
#include "device_common.h"
#include "kargs.h"
#include "schedule.h"

namespace cp {

// ------------------------------------------------------------- append

// One workgroup per appended row; threads copy 16-byte segments.
__global__ __launch_bounds__(256) void kv_append_kernel(const AppendArgs a) {
  const uint32_t row = blockIdx.x;
  const int r = sorted_search(a.n_req, row, [&](int i) { return a.req[i].row_begin; });
  const AppReq &rq = a.req[r];
  const GeomK &g = a.geom[rq.model];
  const uint32_t pos = rq.old_len + (row - rq.row_begin);
  const uint32_t P = (uint32_t)g.page_tokens;
  uint8_t *page = a.pool + ((uint64_t)a.pte[rq.pte_base + pos / P] << 8);
  const uint32_t nseg = (uint32_t)g.row_elems / 8;
  const uint4 *src =
      reinterpret_cast<const uint4 *>(a.rows + rq.src_off + (uint64_t)(row - rq.row_begin) * (uint32_t)g.row_elems);
  for (uint32_t s = threadIdx.x; s < nseg; s += blockDim.x) {
    uint4 v = src[s];
    *reinterpret_cast<uint4 *>(page + row_seg_offset(g, pos % P, s)) = v;
  }
}

hipError_t launch_append(const AppendArgs &a, hipStream_t stream) {
  if (a.total_rows <= 0) return hipSuccess;
  hipLaunchKernelGGL(kv_append_kernel, dim3(a.total_rows), dim3(64), 0, stream, a);
  return hipGetLastError();
}

// ------------------------------------------------- device page stacks

__global__ __launch_bounds__(256) void stack_push_kernel(const StackPushArgs a) {
  for (int32_t i = threadIdx.x; i < a.n; i += blockDim.x) a.dst[i] = a.ent[i];
  if (threadIdx.x == 0) *a.top = a.new_top;
}

hipError_t launch_stack_push(const StackPushArgs &a, hipStream_t stream) {
  hipLaunchKernelGGL(stack_push_kernel, dim3(1), dim3(256), 0, stream, a);
  return hipGetLastError();
}

// ------------------------------------------------------------- gather

__global__ __launch_bounds__(256) void kv_gather_kernel(const GatherArgs a) {
  const uint32_t row = blockIdx.x;
  const GeomK &g = a.geom;
  const uint32_t pos = a.start + row;
  const uint32_t P = (uint32_t)g.page_tokens;
  const uint8_t *page = a.pool + ((uint64_t)a.pte[a.pte_base + pos / P] << 8);
  const uint32_t nseg = (uint32_t)g.row_elems / 8;
  uint4 *dst = reinterpret_cast<uint4 *>(a.dst + (uint64_t)row * (uint32_t)g.row_elems);
  for (uint32_t s = threadIdx.x; s < nseg; s += blockDim.x)
    dst[s] = *reinterpret_cast<const uint4 *>(page + row_seg_offset(g, pos % P, s));
}

hipError_t launch_gather(const GatherArgs &a, hipStream_t stream) {
  if (a.n_tok == 0) return hipSuccess;
  hipLaunchKernelGGL(kv_gather_kernel, dim3(a.n_tok), dim3(64), 0, stream, a);
  return hipGetLastError();
}

// ------------------------------------------------- decode: vector path

typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2_t __attribute__((ext_vector_type(2)));

// Loads DPL consecutive bf16 values of streamed KV as floats (non-temporal:
// KV is read once per call).
template <int DPL>
CP_DEV void load_bf16(const uint8_t *p, float (&v)[DPL]) {
  if constexpr (DPL == 8) {
    const u32x4_t w = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t *>(p));
    uint32_t x[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      v[2 * i] = __uint_as_float(x[i] << 16);
      v[2 * i + 1] = __uint_as_float(x[i] & 0xffff0000u);
    }
  } else if constexpr (DPL == 4) {
    const u32x2_t w = __builtin_nontemporal_load(reinterpret_cast<const u32x2_t *>(p));
    v[0] = __uint_as_float(w.x << 16);
    v[1] = __uint_as_float(w.x & 0xffff0000u);
    v[2] = __uint_as_float(w.y << 16);
    v[3] = __uint_as_float(w.y & 0xffff0000u);
  } else if constexpr (DPL == 2) {
    const uint32_t w = __builtin_nontemporal_load(reinterpret_cast<const uint32_t *>(p));
    v[0] = __uint_as_float(w << 16);
    v[1] = __uint_as_float(w & 0xffff0000u);
  } else {
    v[0] = bf16_to_f32(*reinterpret_cast<const uint16_t *>(p));
  }
}

constexpr int kWaves = 4;
constexpr int kLdsFloats = 16 * 1024 + 4 * 2 * 16 + 64;

// One work unit of the vector path: query heads [h0, h0 + nh) of one KV head
// over the pages of one KV range. Waves take pages round-robin, each with
// its own online-softmax state; the four states are combined at the end in
// a fixed order. Scores live in the log2 domain: s2 = scale*log2(e)*<q, k>.
template <int HB, int DPL>
__device__ __forceinline__ void valu_unit(const DecodeArgs &a, const GeomK &gm, const DecReq &rq, const Seg &sg,
                                          float *lds) {
  const uint32_t chunk = sg.slot, hblk = sg.hblk;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int P = gm.page_tokens;
  const int kvh = (int)hblk / gm.nb, hbi = (int)hblk % gm.nb;
  const int h0 = kvh * gm.g + hbi * HB;
  const int nh = min(HB, gm.g - hbi * HB);
  const int dk = gm.d_k, dv = gm.d_v;

  float *q_s = lds;  // [HB][dk]
  for (int i = threadIdx.x; i < HB * dk; i += blockDim.x) {
    const int h = i / dk, e = i - h * dk;
    q_s[i] = h < nh ? bf16_to_f32(a.q[rq.q_off + (uint32_t)(h0 + h) * dk + e]) : 0.f;
  }
  __syncthreads();

  const uint32_t tok_end = min(rq.ctx_len, sg.pg_end * (uint32_t)P);
  const uint32_t pg_begin = sg.pg_begin;
  const uint32_t pg_end = (tok_end + P - 1) / P;
  const uint64_t head_blk = gm.kind == 0 ? 0 : (uint64_t)2 * P * dk * 2;
  const uint32_t stride = (uint32_t)dk * 2;
  const uint64_t v_off = gm.kind == 0 ? 0 : (uint64_t)P * dk * 2;

  float m[HB], l[HB], acc[HB][DPL];
#pragma unroll
  for (int h = 0; h < HB; ++h) {
    m[h] = -INFINITY;
    l[h] = 0.f;
#pragma unroll
    for (int j = 0; j < DPL; ++j) acc[h][j] = 0.f;
  }

  for (uint32_t pg = pg_begin + wave; pg < pg_end; pg += kWaves) {
    const uint8_t *base = page_ptr(a.pool, a.pte, rq.pte_base, pg) + kvh * head_blk;
    for (int sb = 0; sb < P; sb += 64) {
      const int nvalid = min(min(64, P - sb), (int)tok_end - (int)(pg * P + sb));
      if (nvalid <= 0) break;
      const bool valid = lane < nvalid;
      float s[HB];
#pragma unroll
      for (int h = 0; h < HB; ++h) s[h] = 0.f;
      if (valid) {
        const uint8_t *kr = base + (uint64_t)(sb + lane) * stride;
        for (int e8 = 0; e8 < dk / 8; ++e8) {
          float k[8];
          load_bf16<8>(kr + e8 * 16, k);
#pragma unroll
          for (int h = 0; h < HB; ++h) {
            const float *qh = q_s + h * dk + e8 * 8;
#pragma unroll
            for (int j = 0; j < 8; ++j) s[h] = fmaf(qh[j], k[j], s[h]);
          }
        }
      }
      float pv[HB];
#pragma unroll
      for (int h = 0; h < HB; ++h) {
        const float sv = valid ? s[h] * gm.scale_log2 : -INFINITY;
        const float mn = fmaxf(m[h], wave_max(sv));
        const float alpha = fast_exp2(m[h] - mn);
        const float p = valid ? fast_exp2(sv - mn) : 0.f;
        l[h] = l[h] * alpha + wave_sum(p);
        m[h] = mn;
#pragma unroll
        for (int j = 0; j < DPL; ++j) acc[h][j] *= alpha;
        pv[h] = p;
      }
      const uint8_t *vb = base + v_off + (uint64_t)sb * stride + (uint64_t)lane * DPL * 2;
      for (int t = 0; t < nvalid; ++t) {
        float v[DPL];
        load_bf16<DPL>(vb + (uint64_t)t * stride, v);
#pragma unroll
        for (int h = 0; h < HB; ++h) {
          const float pt = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(pv[h]), t));
#pragma unroll
          for (int j = 0; j < DPL; ++j) acc[h][j] = fmaf(pt, v[j], acc[h][j]);
        }
      }
    }
  }

  // Combine the wave states in wave order.
  __syncthreads();  // q_s no longer needed; reuse LDS
  float *m_s = lds + 16 * 1024;  // [kWaves][HB]
  float *l_s = m_s + kWaves * 16;
  float *acc_s = lds;            // [HB][dv]
  if (lane == 0) {
#pragma unroll
    for (int h = 0; h < HB; ++h) {
      m_s[wave * 16 + h] = m[h];
      l_s[wave * 16 + h] = l[h];
    }
  }
  __syncthreads();
  float M[HB], L[HB], f[HB];
#pragma unroll
  for (int h = 0; h < HB; ++h) {
    float mx = -INFINITY;
    for (int w = 0; w < kWaves; ++w) mx = fmaxf(mx, m_s[w * 16 + h]);
    float sum = 0.f;
    for (int w = 0; w < kWaves; ++w) sum += l_s[w * 16 + h] * fast_exp2(m_s[w * 16 + h] - mx);
    M[h] = mx;
    L[h] = sum;
    f[h] = fast_exp2(m[h] - mx);
  }
  for (int w = 0; w < kWaves; ++w) {
    if (wave == w) {
#pragma unroll
      for (int h = 0; h < HB; ++h)
#pragma unroll
        for (int j = 0; j < DPL; ++j) {
          float *dst = acc_s + h * dv + lane * DPL + j;
          const float x = acc[h][j] * f[h];
          *dst = (w == 0) ? x : *dst + x;
        }
    }
    __syncthreads();
  }
  const bool split = rq.ws_base != kNoWs;
  for (int i = threadIdx.x; i < nh * dv; i += blockDim.x) {
    const int h = i / dv, d = i - h * dv;
    float Lh = 0.f;
#pragma unroll
    for (int hh = 0; hh < HB; ++hh)
      if (hh == h) Lh = L[hh];
    const float o = acc_s[h * dv + d] / Lh;
    const uint32_t qh = (uint32_t)(h0 + h);
    if (split)
      a.ws_o[((uint64_t)rq.ws_orow + (uint64_t)chunk * gm.hq + qh) * dv + d] = (uint16_t)f32_to_bf16(o);
    else
      a.out[rq.o_off + qh * dv + d] = (uint16_t)f32_to_bf16(o);
  }
  if (threadIdx.x < HB && (int)threadIdx.x < nh) {
    float Mh = 0.f, Lh = 1.f;
#pragma unroll
    for (int hh = 0; hh < HB; ++hh)
      if (hh == (int)threadIdx.x) {
        Mh = M[hh];
        Lh = L[hh];
      }
    const float lse = (Mh + fast_log2(Lh)) * kLn2;
    const uint32_t qh = (uint32_t)(h0 + threadIdx.x);
    if (split)
      a.ws_l[(uint64_t)rq.ws_base + (uint64_t)chunk * gm.hq + qh] = lse;
    else
      a.lse[rq.lse_off + qh] = lse;
  }
  __syncthreads();  // LDS is reused by the next unit
}

// Narrow matrix variants: heads per unit, K and V widths, MLA layout,
// tokens per slice, and the stream layout of the 8-wave workgroup (waves
// per stream, ring slots per stream).
constexpr int kNarrowWaves = 8;
template <int V> struct NarrowVar;
template <> struct NarrowVar<kM_MLA_G16> { static constexpr int G = 16, DK = 576, DV = 512, TW = 16, SHARE = 2, NSLOT = 2; static constexpr bool MLA = true; };
template <> struct NarrowVar<kM_MLA_G32> { static constexpr int G = 16, DK = 576, DV = 512, TW = 16, SHARE = 2, NSLOT = 2; static constexpr bool MLA = true; };
template <> struct NarrowVar<kM_D128_G8> { static constexpr int G = 8, DK = 128, DV = 128, TW = 32, SHARE = 2, NSLOT = 2; static constexpr bool MLA = false; };
template <> struct NarrowVar<kM_D128_G16> { static constexpr int G = 16, DK = 128, DV = 128, TW = 32, SHARE = 2, NSLOT = 2; static constexpr bool MLA = false; };
template <> struct NarrowVar<kM_D128_G32> { static constexpr int G = 32, DK = 128, DV = 128, TW = 32, SHARE = 2, NSLOT = 2; static constexpr bool MLA = false; };
template <int V>
using NarrowCfgOf = NarrowCfg<NarrowVar<V>::G, NarrowVar<V>::DK, NarrowVar<V>::DV, NarrowVar<V>::MLA, NarrowVar<V>::TW,
                              kNarrowWaves, NarrowVar<V>::SHARE, NarrowVar<V>::NSLOT>;

template <int V>
constexpr int narrow_lds() { return NarrowCfgOf<V>::LDS; }

constexpr bool has(uint32_t mask, int v) { return (mask >> v) & 1u; }
constexpr uint32_t kValuMask = 0xFFu;
constexpr uint32_t kSmallMask = 0x3F00u;  // variants 8-13

template <int V> struct SmallVar;
template <> struct SmallVar<kS_G1_D64> { static constexpr int G = 1, D = 64; };
template <> struct SmallVar<kS_G2_D64> { static constexpr int G = 2, D = 64; };
template <> struct SmallVar<kS_G4_D64> { static constexpr int G = 4, D = 64; };
template <> struct SmallVar<kS_G1_D128> { static constexpr int G = 1, D = 128; };
template <> struct SmallVar<kS_G2_D128> { static constexpr int G = 2, D = 128; };
template <> struct SmallVar<kS_G4_D128> { static constexpr int G = 4, D = 128; };
template <int V>
constexpr int small_lds() { return SmallCfg<SmallVar<V>::G, SmallVar<V>::D>::LDS; }

// LDS bytes of a kernel covering the variant set `mask`.
constexpr int kernel_lds_bytes(uint32_t mask) {
  int b = 16;
  if (mask & kValuMask) b = kLdsFloats * 4 > b ? kLdsFloats * 4 : b;
#define CP_S(V) if (has(mask, V) && small_lds<V>() > b) b = small_lds<V>();
  CP_S(kS_G1_D64) CP_S(kS_G2_D64) CP_S(kS_G4_D64) CP_S(kS_G1_D128) CP_S(kS_G2_D128) CP_S(kS_G4_D128)
#undef CP_S
#define CP_B(V) if (has(mask, V) && narrow_lds<V>() > b) b = narrow_lds<V>();
  CP_B(kM_MLA_G16) CP_B(kM_MLA_G32) CP_B(kM_D128_G8) CP_B(kM_D128_G16) CP_B(kM_D128_G32)
#undef CP_B
  return b;
}

template <uint32_t MASK>
__device__ __forceinline__ void run_seg(const DecodeArgs &a, const DecReq &rq, const Seg &sg, char *lds) {
  const GeomK &gm = a.geom[sg.model];
#define CP_VCASE(V, HB, DPL)                                        \
  if constexpr (has(MASK, V)) {                                     \
    if (gm.variant == V) {                                          \
      valu_unit<HB, DPL>(a, gm, rq, sg, reinterpret_cast<float *>(lds)); \
      return;                                                       \
    }                                                               \
  }
  CP_VCASE(kV16x8, 16, 8) CP_VCASE(kV16x4, 16, 4) CP_VCASE(kV16x2, 16, 2) CP_VCASE(kV16x1, 16, 1)
  CP_VCASE(kV8x8, 8, 8) CP_VCASE(kV8x4, 8, 4) CP_VCASE(kV8x2, 8, 2) CP_VCASE(kV8x1, 8, 1)
#undef CP_VCASE
#define CP_SCASE(V)                                                                          \
  if constexpr (has(MASK, V)) {                                                              \
    if (gm.variant == V) {                                                                   \
      small_unit<SmallVar<V>::G, SmallVar<V>::D>(a, gm, rq, sg, reinterpret_cast<float *>(lds)); \
      return;                                                                                \
    }                                                                                        \
  }
  CP_SCASE(kS_G1_D64) CP_SCASE(kS_G2_D64) CP_SCASE(kS_G4_D64) CP_SCASE(kS_G1_D128) CP_SCASE(kS_G2_D128)
  CP_SCASE(kS_G4_D128)
#undef CP_SCASE
#define CP_NCASE(V)                                                                          \
  if constexpr (has(MASK, V)) {                                                              \
    if (gm.variant == V) {                                                                   \
      using W = NarrowVar<V>;                                                                \
      narrow_unit<W::G, W::DK, W::DV, W::MLA, W::TW, kNarrowWaves, W::SHARE, W::NSLOT>(a, gm, rq, sg, lds); \
      return;                                                                                \
    }                                                                                        \
  }
  CP_NCASE(kM_MLA_G16) CP_NCASE(kM_MLA_G32) CP_NCASE(kM_D128_G8) CP_NCASE(kM_D128_G16) CP_NCASE(kM_D128_G32)
#undef CP_NCASE
}

// One kernel per variant set of the narrow family; four waves per
// workgroup, LDS sized for the largest variant in the set.
// Vector variants run four waves per workgroup, narrow matrix variants
// eight; the host never mixes the two families in one launch.
template <uint32_t MASK>
constexpr int kernel_waves() { return (MASK & (kValuMask | kSmallMask)) ? 4 : kNarrowWaves; }

template <uint32_t MASK>
__global__ __launch_bounds__(64 * kernel_waves<MASK>()) void decode_kernel(const DecodeArgs a) {
  static_assert(!((MASK & kValuMask) && (MASK & ~kValuMask)) && !((MASK & kSmallMask) && (MASK & ~kSmallMask)),
                "vector, small-group and matrix variants launch separately");
  __shared__ __attribute__((aligned(16))) char lds[kernel_lds_bytes(MASK)];
  __shared__ uint32_t next;
  decode_loop(a, &next, [&](const DecReq &rq, const Seg &sg) { run_seg<MASK>(a, rq, sg, lds); });
}

constexpr uint32_t vbit(int v) { return 1u << v; }
// The variant sets the host launches together: each single variant, and
// the mixed MLA-16 / MQA-32 / GQA-8 batch.
constexpr uint32_t kMixedSmall = vbit(kM_MLA_G16) | vbit(kM_D128_G32) | vbit(kM_D128_G8);
constexpr uint32_t kAllNarrow =
    vbit(kM_MLA_G16) | vbit(kM_MLA_G32) | vbit(kM_D128_G16) | vbit(kM_D128_G32) | vbit(kM_D128_G8);

// Picks the kernel instantiation that covers `mask`. Returns
// hipErrorInvalidValue for a set no instantiation covers (the host keeps
// variants of different workgroup sizes in separate launches).
// ev0 / ev1 (may be null) take the start and end time of the launch.
hipError_t launch_decode(const DecodeArgs &a, int grid, uint32_t mask, hipStream_t stream, hipEvent_t ev0,
                         hipEvent_t ev1) {
  const dim3 g(grid);
#define CP_L(M)                                                                       \
  case M:                                                                             \
    hipExtLaunchKernelGGL((decode_kernel<M>), g, dim3(64 * kernel_waves<M>()), 0, stream, ev0, ev1, 0, a); \
    return hipGetLastError();
  switch (mask) {
    CP_L(vbit(kV16x8)) CP_L(vbit(kV16x4)) CP_L(vbit(kV16x2)) CP_L(vbit(kV16x1))
    CP_L(vbit(kV8x8)) CP_L(vbit(kV8x4)) CP_L(vbit(kV8x2)) CP_L(vbit(kV8x1))
    CP_L(vbit(kM_MLA_G16)) CP_L(vbit(kM_MLA_G32)) CP_L(vbit(kM_D128_G16)) CP_L(vbit(kM_D128_G32))
    CP_L(vbit(kM_D128_G8))
    CP_L(kMixedSmall)
    CP_L(vbit(kS_G1_D64)) CP_L(vbit(kS_G2_D64)) CP_L(vbit(kS_G4_D64)) CP_L(vbit(kS_G1_D128)) CP_L(vbit(kS_G2_D128))
    CP_L(vbit(kS_G4_D128))
    default: break;
  }
#undef CP_L
  if ((mask & ~kValuMask) == 0) {
    hipExtLaunchKernelGGL((decode_kernel<kValuMask>), g, dim3(256), 0, stream, ev0, ev1, 0, a);
    return hipGetLastError();
  }
  if ((mask & ~kSmallMask) == 0) {
    hipExtLaunchKernelGGL((decode_kernel<kSmallMask>), g, dim3(256), 0, stream, ev0, ev1, 0, a);
    return hipGetLastError();
  }
  if ((mask & ~kAllNarrow) == 0) {
    hipExtLaunchKernelGGL((decode_kernel<kAllNarrow>), g, dim3(64 * kNarrowWaves), 0, stream, ev0, ev1, 0, a);
    return hipGetLastError();
  }
  return hipErrorInvalidValue;
}

// Token streams of the narrow kernel for a variant (KV heads a unit covers
// when they split across streams).
int narrow_streams(int variant) {
  switch (variant) {
    case kM_MLA_G16: return NarrowCfgOf<kM_MLA_G16>::NSTREAM;
    case kM_MLA_G32: return NarrowCfgOf<kM_MLA_G32>::NSTREAM;
    case kM_D128_G8: return NarrowCfgOf<kM_D128_G8>::NSTREAM;
    case kM_D128_G16: return NarrowCfgOf<kM_D128_G16>::NSTREAM;
    case kM_D128_G32: return NarrowCfgOf<kM_D128_G32>::NSTREAM;
    default: return 0;
  }
}

// Workgroups of one kernel that fit on a CU at once (LDS-bound).
int decode_wgs_per_cu(uint32_t mask) {
  // small-group vector kernels: two workgroups (eight waves) per CU, so
  // that each SIMD has a second wave to issue while one waits on memory
  if ((mask & kSmallMask) && !(mask & ~kSmallMask)) return 2;
  int b = 16;
  if (mask & 0xFFu) b = kLdsFloats * 4;
#define CP_B(V) if (has(mask, V) && narrow_lds<V>() > b) b = narrow_lds<V>();
  CP_B(kM_MLA_G16) CP_B(kM_MLA_G32) CP_B(kM_D128_G8) CP_B(kM_D128_G16) CP_B(kM_D128_G32)
#undef CP_B
  const int per = (160 * 1024) / (b + 64);
  return per < 1 ? 1 : per;
}

// ------------------------------------------------------------- merge

// Split merge. One workgroup per (split request, query head, block of
// merge_block_cols(d_v) V columns); lane i of every wave covers PER
// consecutive columns of the block. Wave w of the NW waves folds partials
// c = w, w + NW, ... in batches of kMergeUnroll, each batch's lse values and
// outputs loaded together, keeping its own running maximum m_w (log2 domain)
// and rescaling its sums when a batch raises it. The waves then combine in
// wave order with M = max_w m_w:
//   lse = M + ln sum_c exp(lse_c - M),  o = sum_c exp(lse_c - lse) o_c.
// One pass over the partials, so one round trip to memory per batch. The
// partials were written by the decode launch just before and mostly come
// back from the Infinity Cache; the kernel is bound by how many loads it
// keeps in flight, hence whole 8-byte column groups per lane and, for many
// partials, eight waves (NW is the launch's workgroup size / 64).
constexpr int kMergeMaxWaves = 8, kMergeUnroll = 8;

template <int PER>
__device__ __forceinline__ void merge_block(const MergeArgs &a, const MergeReq &rq, uint32_t h, uint32_t db,
                                            float (*part)[256], float *red_m, float *red_l) {
  constexpr float kLog2e = 1.4426950408889634f;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const uint32_t nw = blockDim.x >> 6;
  const uint32_t dv = rq.d_v, n = rq.n_chunks;
  const uint32_t d0 = db * (64 * PER) + lane * PER;
  const uint64_t lrow0 = (uint64_t)rq.ws_base + h;  // lse of chunk c at lrow0 + c * hq
  const uint16_t *obase = a.ws_o + ((uint64_t)rq.ws_orow + h) * dv + d0;
  const uint64_t ostride = (uint64_t)rq.hq * dv;
  float acc[PER], l = 0.f, m = -INFINITY;
#pragma unroll
  for (int j = 0; j < PER; ++j) acc[j] = 0.f;
  // batches of kMergeUnroll partials; only the last may be partial (its
  // test is uniform per wave, and its first partial always exists)
  auto batch = [&](uint32_t c, auto full) {
    float w[kMergeUnroll], x[kMergeUnroll][PER];
#pragma unroll
    for (int u = 0; u < kMergeUnroll; ++u) {
      const uint32_t cc = c + nw * u;
      w[u] = -INFINITY;
#pragma unroll
      for (int j = 0; j < PER; ++j) x[u][j] = 0.f;
      if (decltype(full)::value || cc < n) {
        w[u] = a.ws_l[lrow0 + (uint64_t)cc * rq.hq] * kLog2e;
        const uint16_t *src = obase + (uint64_t)cc * ostride;
        if constexpr (PER == 4) {
          const uint2 v = *reinterpret_cast<const uint2 *>(src);
          x[u][0] = bf16_to_f32(v.x);
          x[u][1] = bf16_to_f32(v.x >> 16);
          x[u][2] = bf16_to_f32(v.y);
          x[u][3] = bf16_to_f32(v.y >> 16);
        } else if constexpr (PER == 2) {
          const uint32_t v = *reinterpret_cast<const uint32_t *>(src);
          x[u][0] = bf16_to_f32(v);
          x[u][1] = bf16_to_f32(v >> 16);
        } else {
          x[u][0] = bf16_to_f32(src[0]);
        }
      }
    }
    float bm = w[0];
#pragma unroll
    for (int u = 1; u < kMergeUnroll; ++u) bm = fmaxf(bm, w[u]);
    if (bm > m) {  // uniform: every lane holds the same lse values
      const float f = fast_exp2(m - bm);  // 0 on the first batch
      l *= f;
#pragma unroll
      for (int j = 0; j < PER; ++j) acc[j] *= f;
      m = bm;
    }
#pragma unroll
    for (int u = 0; u < kMergeUnroll; ++u) {
      const float wu = fast_exp2(w[u] - m);  // 0 for the partials past n
      l += wu;
#pragma unroll
      for (int j = 0; j < PER; ++j) acc[j] = fmaf(wu, x[u][j], acc[j]);
    }
  };
  uint32_t c = wave;
  for (; c + nw * (kMergeUnroll - 1) < n; c += nw * kMergeUnroll) batch(c, std::true_type{});
  if (c < n) batch(c, std::false_type{});
  // combine the waves in order, each rescaled to the block maximum
  if (lane == 0) red_m[wave] = m;
  __syncthreads();
  float M = red_m[0];
  for (uint32_t w2 = 1; w2 < nw; ++w2) M = fmaxf(M, red_m[w2]);
  const float f = m == -INFINITY ? 0.f : fast_exp2(m - M);  // waves without partials add nothing
  if (wave > 0) {
#pragma unroll
    for (int j = 0; j < PER; ++j) part[wave - 1][PER * lane + j] = acc[j] * f;
    if (lane == 0) red_l[wave] = l * f;
  }
  __syncthreads();
  if (wave == 0) {
    float L = l * f;
#pragma unroll
    for (int j = 0; j < PER; ++j) acc[j] *= f;
    for (uint32_t w2 = 1; w2 < nw; ++w2) {
#pragma unroll
      for (int j = 0; j < PER; ++j) acc[j] += part[w2 - 1][PER * lane + j];
      L += red_l[w2];
    }
    const float inv = 1.0f / L;
    uint16_t *dst = a.out + rq.o_off + h * dv + d0;
    if constexpr (PER == 4) {
      *reinterpret_cast<uint2 *>(dst) = bf16x4_bits(acc[0] * inv, acc[1] * inv, acc[2] * inv, acc[3] * inv);
    } else {
#pragma unroll
      for (int j = 0; j < PER; ++j) dst[j] = (uint16_t)f32_to_bf16(acc[j] * inv);
    }
    if (lane == 0 && db == 0) a.lse[rq.lse_off + h] = (M + fast_log2(L)) * kLn2;
  }
}

__global__ __launch_bounds__(64 * kMergeMaxWaves) void merge_kernel(const MergeArgs a) {
  __shared__ float red_m[kMergeMaxWaves], red_l[kMergeMaxWaves];
  __shared__ float part[kMergeMaxWaves - 1][256];
  const uint32_t nblk_total = blockIdx.x;
  const int r = sorted_search(a.n_req, nblk_total, [&](int i) { return a.req[i].block_begin; });
  const MergeReq &rq = a.req[r];
  const uint32_t dblocks = rq.d_v / merge_block_cols(rq.d_v);
  const uint32_t local = nblk_total - rq.block_begin;
  const uint32_t h = local / dblocks, db = local % dblocks;
  const uint32_t per = merge_block_cols(rq.d_v) / 64;
  if (per == 4)
    merge_block<4>(a, rq, h, db, part, red_m, red_l);
  else if (per == 2)
    merge_block<2>(a, rq, h, db, part, red_m, red_l);
  else
    merge_block<1>(a, rq, h, db, part, red_m, red_l);
}

hipError_t launch_merge(const MergeArgs &a, hipStream_t stream) {
  if (a.n_blocks <= 0) return hipSuccess;
  // eight waves when some request has many partials, four otherwise
  int max_n = 0;
  for (int i = 0; i < a.n_req; ++i) max_n = a.req[i].n_chunks > (uint32_t)max_n ? (int)a.req[i].n_chunks : max_n;
  const int waves = max_n >= 8 * kMergeUnroll ? kMergeMaxWaves : 4;
  hipLaunchKernelGGL(merge_kernel, dim3(a.n_blocks), dim3(64 * waves), 0, stream, a);
  return hipGetLastError();
}


// ------------------------------------------------- fixed split workspace

// The split workspace of cp_attn_decode_noalloc: partial outputs and lse
// values of split requests, in a file-scope device array that each GPU the
// library runs on holds until the process ends, so that the call allocates
// no device memory. Nothing in it needs clearing between calls: a launch
// writes every partial slot it plans before its merge reads it. In host
// code this name stands for a host-side placeholder, not device memory; the
// device address comes from scratch_device_address() only.
static __device__ __align__(256) uint8_t scratch[kNoAllocScratchBytes];

// Device address of `scratch` on `device`, which the caller has made
// current. Resolved once per device (each GPU holds its own copy of the
// array at its own address) and kept.
hipError_t scratch_device_address(int device, void **out) {
  static std::mutex mu;
  static void *addr[kMaxScratchDevices] = {};
  if (device < 0 || device >= kMaxScratchDevices) return hipErrorInvalidDevice;
  int cur = -1;
  hipError_t e = hipGetDevice(&cur);
  if (e != hipSuccess) return e;
  if (cur != device) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[device]) {
    void *ptr = nullptr;
    e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!ptr) return hipErrorInvalidSymbol;
    addr[device] = ptr;
  }
  *out = addr[device];
  return hipSuccess;
}

}  // namespace cp
