// Wavefront-reduction decode path for GQA/MHA models with 1, 2 or 4 query
// heads per KV head and head_dim 64 or 128. With so few heads per KV byte
// (at most 4 flop per byte) there is no contraction worth the matrix cores;
// the kernel is built to stream K and V at full width with plain vector
// loads and to keep the vector ALU work per byte small.
//
// Lane layout: a K or V row of one token is D * 2 bytes = LPT lanes x 16
// bytes, so one 16-byte load per lane covers TPI = 64 / LPT consecutive
// tokens of a page (fully coalesced). A wave walks steps of SUB = 16 tokens
// (NI loads for K and NI for V, issued one step ahead):
//   scores   lane (row r, chunk c) forms the partial dot product of its 8
//            K values with the G query heads, and a row reduction (DPP)
//            gives every lane of the row the token's scores;
//   softmax  fp32 online softmax per head over the step's tokens (maximum
//            across the TPI rows by lane swaps), lazily moved reference;
//   P.V      each lane accumulates p(token) * V[token][8 c .. 8 c + 7] for
//            the tokens of its row, so p never leaves the lane.
// At the end the rows are summed by lane swaps, and the four waves of the
// workgroup (which took interleaved steps) are merged through LDS.
#pragma once

#include "decode_mfma.h"

namespace cp {

template <int G, int D>
struct SmallCfg {
  static constexpr int NW = 4;
  static constexpr int LPT = D / 8;     // lanes per token row (16 bytes each)
  static constexpr int TPI = 64 / LPT;  // tokens per load instruction
  static constexpr int SUB = 16;        // tokens per step
  static constexpr int NI = SUB / TPI;  // loads per step, for K and again for V
  static constexpr int LDS = NW * (2 * G + G * D) * 4;  // merge area
  static_assert(D == 64 || D == 128, "head_dim 64 or 128");
  static_assert(G == 1 || G == 2 || G == 4, "1, 2 or 4 query heads per KV head");
};

// Sum over the lanes of one token row (8 or 16 consecutive lanes) by DPP
// moves: swap neighbours, swap pairs, mirror the half rows (pairs lanes of
// the two quads) and, for 16-lane rows, mirror the row.
template <int LPT>
CP_DEV float row_sum(float x) {
  x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0xB1, 0xF, 0xF, false));   // quad_perm [1,0,3,2]
  x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x4E, 0xF, 0xF, false));   // quad_perm [2,3,0,1]
  x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x141, 0xF, 0xF, false));  // row_half_mirror
  if constexpr (LPT == 16)
    x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x140, 0xF, 0xF, false));  // row_mirror
  return x;
}

// Maximum / sum over the TPI token rows of the wave (rows of 8 or 16
// lanes): a rotate by 8 within each 16-lane row for 8-lane rows, then the
// half-row and half-wave swaps.
template <int LPT>
CP_DEV float rows_max(float x) {
  if constexpr (LPT == 8) {
    const float y = __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x128, 0xF, 0xF, false));
    x = x > y ? x : y;  // row_ror:8
  }
  return xor_max_16_32(x);
}
template <int LPT>
CP_DEV float rows_sum(float x) {
  if constexpr (LPT == 8) x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x128, 0xF, 0xF, false));
  return xor_sum_16_32(x);
}

typedef unsigned int u32x4n __attribute__((ext_vector_type(4)));

CP_DEV void unpack8(const u32x4n &u, float (&f)[8]) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    f[2 * i] = bf16_to_f32(u[i] & 0xFFFFu);
    f[2 * i + 1] = bf16_to_f32(u[i] >> 16);
  }
}

// One unit: the query heads of KV head sg.hblk over the pages of one KV
// range (GQA layout: per page and KV head, P K rows then P V rows).
template <int G, int D>
__device__ __forceinline__ void small_unit(const DecodeArgs &a, const GeomK &gm, const DecReq &rq, const Seg &sg,
                                           float *lds) {
  using C = SmallCfg<G, D>;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int r = lane / C::LPT, c = lane % C::LPT;  // token row within a load, 16-byte chunk within the row
  const int P = gm.page_tokens;                     // the host routes only pages of a multiple of 16 tokens here
  const int kvh = (int)sg.hblk;
  const int h0 = kvh * gm.g, hv = gm.g;             // first query head, valid heads (<= G)
  const uint32_t slot = sg.slot;

  // the lane's 8 query values of every head (zero for padded heads)
  float q[G][8];
#pragma unroll
  for (int h = 0; h < G; ++h) {
    const u32x4n u = h < hv ? *reinterpret_cast<const u32x4n *>(a.q + rq.q_off + (uint32_t)(h0 + h) * D + 8 * c)
                            : u32x4n{0u, 0u, 0u, 0u};
    unpack8(u, q[h]);
  }

  const uint32_t tok_begin = sg.pg_begin * (uint32_t)P;
  const uint32_t tok_end = min(rq.ctx_len, sg.pg_end * (uint32_t)P);
  const int nsteps = (int)((tok_end - tok_begin + C::SUB - 1) / C::SUB);
  const uint64_t head_blk = (uint64_t)2 * P * D * 2;
  const int npg = (int)((tok_end + P - 1) / P) - (int)sg.pg_begin;

  // page-table entries of the range, 64 at a time (lane i: page 64 b + i)
  uint32_t pte_lane = 0;
  int pte_batch = -1;
  // Loads of step j: K and V rows of tokens tok_begin + 16 j + TPI i + r.
  auto load_step = [&](int j, u32x4n (&kb)[C::NI], u32x4n (&vb)[C::NI]) __attribute__((always_inline)) {
    const uint32_t t0 = tok_begin + (uint32_t)(C::SUB * j);
    const int sp = (int)(t0 / (uint32_t)P) - (int)sg.pg_begin;  // page within the range
    if ((sp >> 6) != pte_batch) {
      pte_batch = sp >> 6;
      const int pi = 64 * pte_batch + lane;
      pte_lane = pi < npg ? a.pte[rq.pte_base + sg.pg_begin + (uint32_t)pi] : 0u;
    }
    const uint32_t pte = __builtin_amdgcn_readlane(pte_lane, sp & 63);
    const uint8_t *kp = a.pool + ((uint64_t)pte << 8) + (uint64_t)kvh * head_blk +
                        (uint64_t)(t0 % (uint32_t)P) * (D * 2) + (uint64_t)(r * (D * 2) + 16 * c);
#pragma unroll
    for (int i = 0; i < C::NI; ++i) {
      kb[i] = __builtin_nontemporal_load(reinterpret_cast<const u32x4n *>(kp + i * C::TPI * (D * 2)));
      vb[i] = __builtin_nontemporal_load(reinterpret_cast<const u32x4n *>(kp + (uint64_t)P * D * 2 + i * C::TPI * (D * 2)));
    }
  };

  float m[G], lsum[G], o[G][8];
#pragma unroll
  for (int h = 0; h < G; ++h) {
    m[h] = -INFINITY;
    lsum[h] = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) o[h][e] = 0.f;
  }
  const float sl2 = gm.scale_log2;

  auto compute = [&](int j, const u32x4n (&kb)[C::NI], const u32x4n (&vb)[C::NI]) __attribute__((always_inline)) {
    const int valid = min(C::SUB, (int)(tok_end - tok_begin) - C::SUB * j);
    float s[C::NI][G];
#pragma unroll
    for (int i = 0; i < C::NI; ++i) {
      float k[8];
      unpack8(kb[i], k);
#pragma unroll
      for (int h = 0; h < G; ++h) {
        float d = 0.f;
#pragma unroll
        for (int e = 0; e < 8; ++e) d = __builtin_fmaf(q[h][e], k[e], d);
        d = row_sum<C::LPT>(d);
        s[i][h] = C::TPI * i + r < valid ? d : -INFINITY;
      }
    }
    bool bump = false;
    float mt[G];
#pragma unroll
    for (int h = 0; h < G; ++h) {
      float x = s[0][h];
#pragma unroll
      for (int i = 1; i < C::NI; ++i) x = x > s[i][h] ? x : s[i][h];
      mt[h] = rows_max<C::LPT>(x) * sl2;
      bump = bump || mt[h] > m[h] + kLazy;
    }
    if (__builtin_amdgcn_ballot_w64(bump)) {  // the same in every lane
#pragma unroll
      for (int h = 0; h < G; ++h) {
        const float mn = mt[h] > m[h] + kLazy ? mt[h] : m[h];
        const float al = fast_exp2(m[h] - mn);
        m[h] = mn;
        lsum[h] *= al;
#pragma unroll
        for (int e = 0; e < 8; ++e) o[h][e] *= al;
      }
    }
#pragma unroll
    for (int i = 0; i < C::NI; ++i) {
      // rows past the context may hold stale bytes (even NaN): their p is 0
      // and their V is taken as 0, so 0 * V stays 0
      float v[8];
      unpack8(C::TPI * i + r < valid ? vb[i] : u32x4n{0u, 0u, 0u, 0u}, v);
#pragma unroll
      for (int h = 0; h < G; ++h) {
        const float p = fast_exp2(__builtin_fmaf(s[i][h], sl2, -m[h]));
        lsum[h] += p;
#pragma unroll
        for (int e = 0; e < 8; ++e) o[h][e] = __builtin_fmaf(p, v[e], o[h][e]);
      }
    }
  };

  // Steps j = wave, wave + NW, ...: loads one step ahead, two buffers.
  {
    u32x4n ka[C::NI], va[C::NI], kb2[C::NI], vb2[C::NI];
    int j = wave;
    if (j < nsteps) load_step(j, ka, va);
#pragma unroll 1
    while (j < nsteps) {
      if (j + C::NW < nsteps) load_step(j + C::NW, kb2, vb2);
      compute(j, ka, va);
      j += C::NW;
      if (j >= nsteps) break;
      if (j + C::NW < nsteps) load_step(j + C::NW, ka, va);
      compute(j, kb2, vb2);
      j += C::NW;
    }
  }

  // ---- rows summed (each row counted every token of its own once), then
  // the waves merged in wave order through LDS
#pragma unroll
  for (int h = 0; h < G; ++h) {
    lsum[h] = rows_sum<C::LPT>(lsum[h]);
#pragma unroll
    for (int e = 0; e < 8; ++e) o[h][e] = rows_sum<C::LPT>(o[h][e]);
  }
  float *m_s = lds;                      // [NW][G]
  float *l_s = m_s + C::NW * G;          // [NW][G]
  float *o_s = l_s + C::NW * G;          // [NW][G][D]
  if (lane == 0) {
#pragma unroll
    for (int h = 0; h < G; ++h) {
      m_s[wave * G + h] = m[h];
      l_s[wave * G + h] = lsum[h];
    }
  }
  if (r == 0) {
#pragma unroll
    for (int h = 0; h < G; ++h) {
      *reinterpret_cast<f32x4 *>(o_s + (wave * G + h) * D + 8 * c) = f32x4{o[h][0], o[h][1], o[h][2], o[h][3]};
      *reinterpret_cast<f32x4 *>(o_s + (wave * G + h) * D + 8 * c + 4) = f32x4{o[h][4], o[h][5], o[h][6], o[h][7]};
    }
  }
  __syncthreads();
  const bool split = rq.ws_base != kNoWs;
  for (int t = threadIdx.x; t < G * D / 4; t += 64 * C::NW) {
    const int h = (4 * t) / D, d = (4 * t) % D;
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < C::NW; ++w) M = fmaxf(M, m_s[w * G + h]);
    float L = 0.f;
    f32x4 v = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int w = 0; w < C::NW; ++w) {
      const float mw = m_s[w * G + h];
      const float f = mw == -INFINITY ? 0.f : fast_exp2(mw - M);  // a wave without steps adds nothing
      L += l_s[w * G + h] * f;
      v += *reinterpret_cast<const f32x4 *>(o_s + (w * G + h) * D + d) * f;
    }
    if (h < hv) {
      const uint32_t head = (uint32_t)(h0 + h);
      const f32x4 x = v * (1.0f / L);
      const uint2 pk = bf16x4_bits(x[0], x[1], x[2], x[3]);
      if (split) {
        *reinterpret_cast<uint2 *>(a.ws_o + ((uint64_t)rq.ws_orow + (uint64_t)slot * gm.hq + head) * D + d) = pk;
        if (d == 0) a.ws_l[(uint64_t)rq.ws_base + (uint64_t)slot * gm.hq + head] = (M + fast_log2(L)) * kLn2;
      } else {
        *reinterpret_cast<uint2 *>(a.out + rq.o_off + head * D + d) = pk;
        if (d == 0) a.lse[rq.lse_off + head] = (M + fast_log2(L)) * kLn2;
      }
    }
  }
  __syncthreads();  // LDS is reused by the next unit
}

}  // namespace cp
