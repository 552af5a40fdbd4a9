// gfx950 kernels of the shared KV pool: KV append (scatter through the page
// table), gather (the inverse), decode attention, and the split-KV merge.
//
// Page-internal layouts (one page = page_tokens tokens of one model):
//   MLA      token-major [P][d_k] bf16: a page is the request's logical rows
//            for those tokens, back to back; V is the first d_v of each row.
//   GQA/MQA  head-major [Hkv][ K: P x d | V: P x d ] bf16, so the K (or V)
//            rows of one KV head inside one page are one contiguous block.
// A page starts at pool + (pte << 8).
#include <hip/hip_runtime.h>

#include "kargs.h"

namespace cp {

#define CP_DEV __device__ __forceinline__

CP_DEV float bf16_to_f32(uint32_t b) { return __uint_as_float(b << 16); }

// Round to nearest even; quiet NaN stays NaN.
CP_DEV uint32_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return 0x7fc0u;
  u += 0x7fffu + ((u >> 16) & 1u);
  return u >> 16;
}

CP_DEV float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }
CP_DEV float fast_log2(float x) { return __builtin_amdgcn_logf(x); }

constexpr float kLn2 = 0.693147180559945309f;

CP_DEV float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

CP_DEV float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

CP_DEV const uint8_t *page_ptr(const uint8_t *pool, const uint32_t *pte, uint32_t pte_base, uint32_t page) {
  return pool + ((uint64_t)pte[pte_base + page] << 8);
}

// Byte offset, inside a page, of 16-byte segment `seg` of the logical row of
// token slot `slot` (row = [K heads | V heads] for GQA, [latent | rope] for MLA).
CP_DEV uint64_t row_seg_offset(const GeomK &g, uint32_t slot, uint32_t seg) {
  const uint32_t e = seg * 8;  // first bf16 element of the segment
  if (g.kind == 0) return (uint64_t)slot * (uint32_t)(g.d_k * 2) + (uint64_t)e * 2;
  const uint32_t d = (uint32_t)g.d_k, hk = (uint32_t)g.hkv, P = (uint32_t)g.page_tokens;
  const uint64_t head_blk = (uint64_t)2 * P * d * 2;
  if (e < hk * d) {
    const uint32_t kh = e / d, off = e - kh * d;
    return kh * head_blk + (uint64_t)slot * d * 2 + (uint64_t)off * 2;
  }
  const uint32_t e2 = e - hk * d, kh = e2 / d, off = e2 - kh * d;
  return kh * head_blk + (uint64_t)P * d * 2 + (uint64_t)slot * d * 2 + (uint64_t)off * 2;
}

// ------------------------------------------------------------- append

// One workgroup per appended row; threads copy 16-byte segments.
__global__ __launch_bounds__(256) void kv_append_kernel(const AppendArgs a) {
  const uint32_t row = blockIdx.x;
  int r = 0;
  while (r + 1 < a.n_req && a.req[r + 1].row_begin <= row) ++r;
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

// Loads DPL consecutive bf16 values as floats.
template <int DPL>
CP_DEV void load_bf16(const uint8_t *p, float (&v)[DPL]) {
  if constexpr (DPL == 8) {
    uint4 w = *reinterpret_cast<const uint4 *>(p);
    uint32_t x[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      v[2 * i] = __uint_as_float(x[i] << 16);
      v[2 * i + 1] = __uint_as_float(x[i] & 0xffff0000u);
    }
  } else if constexpr (DPL == 4) {
    uint2 w = *reinterpret_cast<const uint2 *>(p);
    v[0] = __uint_as_float(w.x << 16);
    v[1] = __uint_as_float(w.x & 0xffff0000u);
    v[2] = __uint_as_float(w.y << 16);
    v[3] = __uint_as_float(w.y & 0xffff0000u);
  } else if constexpr (DPL == 2) {
    uint32_t w = *reinterpret_cast<const uint32_t *>(p);
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
__device__ void valu_unit(const DecodeArgs &a, const GeomK &gm, const DecReq &rq, uint32_t chunk, uint32_t hblk,
                          float *lds) {
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

  const uint32_t tok_begin = chunk * rq.chunk_pages * (uint32_t)P;
  const uint32_t tok_end = min(rq.ctx_len, tok_begin + (uint32_t)rq.chunk_pages * P);
  const uint32_t pg_begin = chunk * rq.chunk_pages;
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
      a.ws_o[((uint64_t)rq.ws_orow + (uint64_t)chunk * gm.hq + qh) * dv + d] = o;
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

// Vector-path variants: (heads per block, V elements per lane).
enum : int32_t { kV16x8 = 0, kV16x4, kV16x2, kV16x1, kV8x8, kV8x4, kV8x2, kV8x1 };

__device__ void run_unit(const DecodeArgs &a, uint32_t u, float *lds) {
  int r = 0;
  while (r + 1 < a.n_req && a.req[r + 1].unit_begin <= u) ++r;
  const DecReq &rq = a.req[r];
  const GeomK &gm = a.geom[rq.model];
  const uint32_t local = u - rq.unit_begin;
  const uint32_t chunk = local / rq.n_hblk, hblk = local % rq.n_hblk;
  switch (gm.variant) {
    case kV16x8: valu_unit<16, 8>(a, gm, rq, chunk, hblk, lds); break;
    case kV16x4: valu_unit<16, 4>(a, gm, rq, chunk, hblk, lds); break;
    case kV16x2: valu_unit<16, 2>(a, gm, rq, chunk, hblk, lds); break;
    case kV16x1: valu_unit<16, 1>(a, gm, rq, chunk, hblk, lds); break;
    case kV8x8: valu_unit<8, 8>(a, gm, rq, chunk, hblk, lds); break;
    case kV8x4: valu_unit<8, 4>(a, gm, rq, chunk, hblk, lds); break;
    case kV8x2: valu_unit<8, 2>(a, gm, rq, chunk, hblk, lds); break;
    default: valu_unit<8, 1>(a, gm, rq, chunk, hblk, lds); break;
  }
}

__global__ __launch_bounds__(256) void decode_valu_kernel(const DecodeArgs a) {
  __shared__ float lds[kLdsFloats];
  __shared__ uint32_t next;
  if (!a.persistent) {
    run_unit(a, blockIdx.x, lds);
    return;
  }
  for (;;) {
    if (threadIdx.x == 0) next = atomicAdd(&a.queue[0], 1u);
    __syncthreads();
    const uint32_t u = next;
    __syncthreads();
    if (u >= (uint32_t)a.n_units) break;
    run_unit(a, u, lds);
  }
  // The last workgroup to finish resets the queue for the next launch.
  if (threadIdx.x == 0) {
    __threadfence();
    if (atomicAdd(&a.queue[1], 1u) == gridDim.x - 1) {
      atomicExch(&a.queue[0], 0u);
      atomicExch(&a.queue[1], 0u);
    }
  }
}

hipError_t launch_decode_valu(const DecodeArgs &a, int grid, hipStream_t stream) {
  hipLaunchKernelGGL(decode_valu_kernel, dim3(grid), dim3(256), 0, stream, a);
  return hipGetLastError();
}

// ------------------------------------------------------------- merge

// One wave per (split request, query head). Partials are folded in range
// order with a running maximum, which equals
//   lse = M + ln sum_c exp(lse_c - M),  o = sum_c exp(lse_c - lse) o_c.
__global__ __launch_bounds__(64) void merge_kernel(const MergeArgs a) {
  const uint32_t row = blockIdx.x;
  int r = 0;
  while (r + 1 < a.n_req && a.req[r + 1].head_begin <= row) ++r;
  const MergeReq &rq = a.req[r];
  const uint32_t h = row - rq.head_begin;
  const int lane = threadIdx.x;
  const uint32_t dv = rq.d_v;
  const int per = (int)dv / 64;  // 1, 2, 4 or 8
  float acc[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) acc[j] = 0.f;
  float m = -INFINITY, l = 0.f;
  constexpr float kLog2e = 1.4426950408889634f;
  for (uint32_t c = 0; c < rq.n_chunks; ++c) {
    const uint64_t prow = (uint64_t)rq.ws_base + (uint64_t)c * rq.hq + h;
    const float x = a.ws_l[prow] * kLog2e;
    const float mn = fmaxf(m, x);
    const float alpha = fast_exp2(m - mn);
    const float w = fast_exp2(x - mn);
    l = l * alpha + w;
    m = mn;
    const float *src = a.ws_o + ((uint64_t)rq.ws_orow + (uint64_t)c * rq.hq + h) * dv + (uint64_t)lane * per;
#pragma unroll
    for (int j = 0; j < 8; ++j)
      if (j < per) acc[j] = acc[j] * alpha + w * src[j];
  }
  const float inv = 1.0f / l;
  uint16_t *dst = a.out + rq.o_off + h * dv + (uint32_t)lane * per;
#pragma unroll
  for (int j = 0; j < 8; ++j)
    if (j < per) dst[j] = (uint16_t)f32_to_bf16(acc[j] * inv);
  if (lane == 0) a.lse[rq.lse_off + h] = (m + fast_log2(l)) * kLn2;
}

hipError_t launch_merge(const MergeArgs &a, hipStream_t stream) {
  if (a.total_heads <= 0) return hipSuccess;
  hipLaunchKernelGGL(merge_kernel, dim3(a.total_heads), dim3(64), 0, stream, a);
  return hipGetLastError();
}

}  // namespace cp
