// Device helpers shared by the gfx950 kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

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

// Index of the last of n (<= 64) non-decreasing keys key(0..n-1) that is
// <= x, or 0 when none is. The lanes test one key each and a ballot counts
// the passing prefix, so the search costs one load latency instead of a
// chain of dependent scalar loads from the argument segment. key(0) is not
// read; every lane of the wave must take part.
template <class F>
CP_DEV int sorted_search(int n, uint64_t x, F key) {
  const int lane = threadIdx.x & 63;
  const bool le = lane > 0 && lane < n && (uint64_t)key(lane) <= x;
  return __builtin_popcountll(__builtin_amdgcn_ballot_w64(le));
}

CP_DEV const uint8_t *page_ptr(const uint8_t *pool, const uint32_t *pte, uint32_t pte_base, uint32_t page) {
  return pool + ((uint64_t)pte[pte_base + page] << 8);
}

// Byte offset, inside a page, of 16-byte segment `seg` of the logical row of
// token slot `slot` (row = [K heads | V heads] for GQA, [latent | rope] for MLA).
// Four floats rounded to bf16 (nearest even), packed in element order.
CP_DEV uint2 bf16x4_bits(float x0, float x1, float x2, float x3) {
  uint2 pk;
  pk.x = f32_to_bf16(x0) | (f32_to_bf16(x1) << 16);
  pk.y = f32_to_bf16(x2) | (f32_to_bf16(x3) << 16);
  return pk;
}

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

}  // namespace cp
