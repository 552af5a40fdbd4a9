// Generic matrix-core decode path for models with 64 or 128 query heads per
// KV head and separate K and V rows (MQA / GQA groups of 64 or 128 with
// head_dim 128). The 128-head MLA geometry has its own pipelined kernel
// (decode_mla.h). Per token the work is a dense contraction, so the kernel
// keeps the matrix cores busy while streaming KV at HBM speed.
//
// One workgroup of NW waves shares a ring of NBUF tiles of T = 32 tokens
// that stream HBM -> LDS by direct, non-temporal loads. Per tile:
//   scores   wave w owns query heads [w G/NW, (w+1) G/NW): for them it
//            computes S^T[t][h] = sum_d K[t][d] Q[h][d] (mfma 16x16x32 bf16,
//            K rows from LDS as the A operand, Q^T in registers as B), the
//            fp32 online softmax (lazily moved reference maximum), and
//            publishes P^T as bf16 operand fragments;
//   P.V      wave w owns V columns [w DV/NW, (w+1) DV/NW) for every head:
//            O^T[d][h] += sum_t V^T[d][t] P^T[t][h] over the tile's 32 tokens
//            with one mfma 16x16x32 per (column block, head block). The K
//            index of that product runs over the 32 tokens in the order
//            {4q..4q+3, 16+4q..16+4q+3} for lane group q, which is exactly
//            how the two 16-token score accumulators hold them, so the score
//            lanes' P values are the B operand as they stand and V^T comes
//            from two LDS transpose reads.
// Scores and P.V of one tile are separated by a barrier (P and the rescale
// factors cross waves); a second barrier at the top of the next tile
// releases the ring slot.
#pragma once

#include "decode_mfma.h"

namespace cp {

typedef unsigned int u32x4v __attribute__((ext_vector_type(4)));

// NW: waves of the workgroup (4 or 8; with 8, two waves share each SIMD,
// so one's LDS and softmax latencies are the other's issue slots). QL: the
// last QL of the KSTEPS query k-steps are kept in LDS rather than registers.
template <int G, int DK, int DV, bool MLA, int QL, int NW_>
struct WideCfg {
  static constexpr int NW = NW_, T = 32;
  static constexpr int KROW = DK * 2;                // bytes of one K row in HBM
  static constexpr int VROW = MLA ? KROW : DV * 2;   // ... of one V row
  static constexpr int KPITCH = lds_pitch(KROW);     // padded LDS rows: conflict-free reads
  static constexpr int VPITCH = MLA ? KPITCH : lds_pitch(VROW);
  static constexpr int TILE_K = T * KPITCH;
  static constexpr int TILE_V = MLA ? 0 : T * VPITCH;
  static constexpr int TILE = TILE_K + TILE_V;       // LDS bytes of one tile
  static constexpr int NLOADS = (TILE + 1023) / 1024;  // 1 KiB direct loads per tile
  static constexpr int KSTEPS = DK / 32;
  static constexpr int HB = G / 16;                  // head blocks of the KV head
  static constexpr int HBQ = G / (16 * NW);          // head blocks each wave scores
  static constexpr int DBW = DV / (16 * NW);         // V column blocks each wave accumulates
  static constexpr int QR = KSTEPS - QL;             // query k-steps held in registers
  // the query goes to the accumulation registers when it and the P.V
  // accumulators would crowd the architectural file
  static constexpr bool AGPR_Q = NW == 4 && HB * DBW * 4 + HBQ * QR * 4 > 192;
  static constexpr int KA = NW == 8 ? 1 : 2;         // K-fragment read-ahead in k-steps
  static constexpr int PBYTES = HB * 64 * 16;        // P^T fragments of one tile
  static constexpr int QBYTES = NW * HBQ * QL * 1024;  // query fragments kept in LDS
  static constexpr int XBYTES = 4 * NW + G * 4 * 2;  // flags, rescale factors, final m / l
  static constexpr int LDS_LIMIT = 163840;
  static constexpr int NBUF_MAX = (LDS_LIMIT - PBYTES - QBYTES - XBYTES - 64) / TILE;
  static constexpr int NBUF = NBUF_MAX > 8 ? 8 : NBUF_MAX;  // ring depth
  static constexpr int LDS = NBUF * TILE + PBYTES + QBYTES + XBYTES;
  static_assert(NW == 4 || NW == 8, "four or eight waves");
  static_assert(G % 64 == 0 && G <= 128 && HBQ >= 1 && G == 16 * NW * HBQ, "whole head blocks per wave");
  static_assert(DV % (16 * NW) == 0 && DK % 32 == 0, "column blocks must tile the head");
  static_assert(NBUF >= 3, "ring too shallow");
  static_assert(QL >= 0 && QL < KSTEPS, "some query k-steps stay in registers");
  static_assert(TILE % 16 == 0, "tiles are whole 16-byte chunks");
};

// One unit: every query head of KV head `kvh` over the pages of one KV range.
template <int G, int DK, int DV, bool MLA, int QL, int NW>
__device__ __forceinline__ void wide_unit(const DecodeArgs &a, const GeomK &gm, const DecReq &rq, const Seg &sg,
                                          char *lds) {
  using C = WideCfg<G, DK, DV, MLA, QL, NW>;
  constexpr int GW = G / NW;  // query heads one wave scores
  const uint32_t kvh = sg.hblk, slot = sg.slot;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // uniform: lets wave-derived values live in SGPRs
  const int col = lane & 15, quad = lane >> 4;
  const int P = gm.page_tokens;  // the host routes only pages of a multiple of 32 tokens here
  const int tpp = P / C::T;        // tiles per page
  const int h_kv = (int)kvh * G;   // first query head of this KV head

  char *const ring = lds;
  char *const pbuf = lds + C::NBUF * C::TILE;
  char *const qbuf = pbuf + C::PBYTES;                                  // [wave][hb][QL][lane] query fragments
  int *const flags = reinterpret_cast<int *>(qbuf + C::QBYTES);        // [NW] rescale needed, per score wave
  float *const alpha_x = reinterpret_cast<float *>(flags + NW);         // [G] rescale factor of this tile
  float *const ml_x = alpha_x + G;                                      // [G] final: l, after m in alpha_x

  // Q^T operand fragments of this wave's score heads: lane holds head
  // (h_kv + G/4 * wave + 16 hb + col), dims 32 c + 8 quad .. +7.
  // The last QL k-steps go to this wave's part of the LDS query area instead.
  bf16x8 qf[C::HBQ][C::QR];
  char *const qmine = qbuf + wave * (C::HBQ * QL * 1024);
#pragma unroll
  for (int hb = 0; hb < C::HBQ; ++hb) {
    const uint16_t *qrow = a.q + rq.q_off + (uint32_t)(h_kv + GW * wave + 16 * hb + col) * DK + 8 * quad;
#pragma unroll
    for (int c = 0; c < C::QR; ++c) {
      qf[hb][c] = *reinterpret_cast<const bf16x8 *>(qrow + 32 * c);
      // the query lives in the accumulation registers, which the matrix
      // cores read directly as their B operand; the P.V accumulators take
      // the architectural registers
      if constexpr (C::AGPR_Q) asm volatile("" : "+a"(qf[hb][c]));
    }
#pragma unroll
    for (int c = 0; c < QL; ++c)
      *reinterpret_cast<bf16x8 *>(qmine + ((hb * QL + c) * 64 + lane) * 16) =
          *reinterpret_cast<const bf16x8 *>(qrow + 32 * (C::QR + c));
  }

  const uint32_t tok_end = min(rq.ctx_len, sg.pg_end * (uint32_t)P);
  const uint32_t pg_begin = sg.pg_begin;
  const int npg = (int)((tok_end + P - 1) / P) - (int)pg_begin;
  const int last_tok = npg > 0 ? (int)tok_end - (int)((pg_begin + (uint32_t)npg - 1) * (uint32_t)P) : 0;
  const int ntiles = npg > 0 ? (npg - 1) * tpp + (last_tok + C::T - 1) / C::T : 0;
  const uint64_t kv_head_bytes = MLA ? 0 : (uint64_t)2 * P * DK * 2;

  // Page-table entries of the segment, 64 at a time (lane i: page 64 b + i).
  uint32_t pte_lane = 0;
  int pte_batch = -1;
  auto load_ptes = [&](int batch) {
    const int sp = batch * 64 + lane;
    pte_lane = sp < npg ? a.pte[rq.pte_base + pg_begin + (uint32_t)sp] : 0u;
    pte_batch = batch;
    // Wait here, visibly to the compiler: the tile loads are inline asm it
    // cannot count, so a wait it placed at the first use of pte_lane would
    // be a full vmcnt(0) in every tile, draining the KV loads in flight.
    // This drains them once per 64 pages instead.
    __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
  };
  // Direct loads of a tile into its ring slot. Load i of the tile covers
  // LDS bytes [1024 i, 1024 i + 1024) of the slot. Wave w issues a
  // contiguous range of loads, in groups of up to four per M0 write
  // (dma_group); the groups are spread over the tile's work so that an M0
  // write rarely finds the previous group still queued. Lanes on a row's
  // pad fetch the row's last 16 bytes again (same cache line, never read
  // back); lanes past the tile are masked off.
  constexpr int LBASE = C::NLOADS / NW, LREM = C::NLOADS % NW;
  constexpr int MY_MAX = LBASE + (LREM ? 1 : 0);  // loads of the busiest wave
  constexpr int NGRP = (MY_MAX + 3) / 4;          // M0 groups per wave and tile
  const int my_loads = LBASE + (wave < LREM ? 1 : 0);
  const int my_first = wave * LBASE + min(wave, LREM);
  // per-lane global offsets of this wave's loads, biased for dma_group
  // (MLA tiles are K rows only, whose offsets fit 16 bits: two per register)
  constexpr bool PACK = C::TILE_V == 0 && C::TILE <= 65536;
  uint32_t voff[NGRP][PACK ? 2 : 4];
#pragma unroll
  for (int g = 0; g < NGRP; ++g)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int o = (my_first + 4 * g + j) * 1024 + lane * 16;
      uint32_t gofs;
      if (C::TILE_V == 0 || o < C::TILE_K) {
        const int oc = o < C::TILE_K ? o : 0;
        const int row = oc / C::KPITCH, w = oc - row * C::KPITCH;
        gofs = (uint32_t)(row * C::KROW + (w < C::KROW ? w : C::KROW - 16));
      } else {
        const int o2 = o < C::TILE ? o - C::TILE_K : 0;
        const int row = o2 / C::VPITCH, w = o2 - row * C::VPITCH;
        gofs = (uint32_t)(P * DK * 2 + row * C::VROW + (w < C::VROW ? w : C::VROW - 16));
      }
      if constexpr (PACK)
        voff[g][j / 2] = (j & 1) ? (voff[g][j / 2] | (gofs << 16)) : gofs;
      else
        voff[g][j] = gofs + kDmaBias - 1024u * j;
    }
  auto group_offsets = [&](int g, uint32_t (&v)[4]) {
#pragma unroll
    for (int j = 0; j < 4; ++j)
      v[j] = PACK ? ((voff[g][j / 2] >> (16 * (j & 1))) & 0xFFFFu) + kDmaBias - 1024u * j : voff[g][PACK ? 0 : j];
  };
  // Source base of tile k (lowered by kDmaBias) and its slot.
  auto tile_src = [&](int k) -> uint64_t {
    const int sp = k / tpp;
    if ((sp >> 6) != pte_batch) load_ptes(sp >> 6);
    const uint32_t pte = __builtin_amdgcn_readlane(pte_lane, sp & 63);
    return uniform_ptr(a.pool + ((uint64_t)pte << 8) + kvh * kv_head_bytes + (uint64_t)(k % tpp) * C::T * C::KROW -
                       kDmaBias);
  };
  // Group g of this wave's loads of tile k, whose source base is sb.
  auto issue_group = [&](int k, uint64_t sb, int g) {
    const int n = min(4, my_loads - 4 * g);
    if (n <= 0) return;
    const int first = my_first + 4 * g;
    const uint32_t lb = __builtin_amdgcn_readfirstlane(lds_addr(ring + (k % C::NBUF) * C::TILE) + first * 1024);
    // a partial last load of the tile goes alone, with the lanes past the
    // tile masked off
    const bool tail = C::TILE % 1024 != 0 && first + n == C::NLOADS;
    const int nf = tail ? n - 1 : n;
    uint32_t vo[4];
    group_offsets(g, vo);
    if (nf == 4) dma_group<4>(sb, vo, lb);
    else if (nf == 3) dma_group<3>(sb, vo, lb);
    else if (nf == 2) dma_group<2>(sb, vo, lb);
    else if (nf == 1) dma_group<1>(sb, vo, lb);
    if (tail && (C::NLOADS - 1) * 1024 + lane * 16 < C::TILE) {
      const uint32_t last[4] = {vo[nf] + 1024u * nf, 0u, 0u, 0u};
      dma_group<1>(sb, last, lb + nf * 1024);
    }
  };
  auto issue_all = [&](int k) {
    const uint64_t sb = tile_src(k);
#pragma unroll
    for (int g = 0; g < NGRP; ++g) issue_group(k, sb, g);
  };

  float m[C::HBQ], lsum[C::HBQ];
  f32x4 o[C::DBW][C::HB];
#pragma unroll
  for (int hb = 0; hb < C::HBQ; ++hb) {
    m[hb] = -INFINITY;
    lsum[hb] = 0.f;
  }
#pragma unroll
  for (int db = 0; db < C::DBW; ++db)
#pragma unroll
    for (int hb = 0; hb < C::HB; ++hb) o[db][hb] = f32x4{0.f, 0.f, 0.f, 0.f};
  const float sl2 = gm.scale_log2;

  if (ntiles > 0) load_ptes(0);
  for (int k = 0; k < C::NBUF - 1 && k < ntiles; ++k) issue_all(k);

#pragma unroll 1
  for (int k = 0; k < ntiles; ++k) {
    // own loads of tile k have landed once at most the later tiles' remain
    const int later = min(C::NBUF - 2, ntiles - 1 - k);
    if (later <= 0)
      wait_vm<0>();
    else if (my_loads == MY_MAX) {
      if (later == 1) wait_vm<MY_MAX>(); else if (later == 2) wait_vm<2 * MY_MAX>(); else wait_vm<3 * MY_MAX>();
    } else {
      if (later == 1) wait_vm<MY_MAX - 1>(); else if (later == 2) wait_vm<2 * (MY_MAX - 1)>(); else wait_vm<3 * (MY_MAX - 1)>();
    }
    __syncthreads();  // tile k visible to all waves; tile k-1's slot and P area are free
    // loads of tile k + NBUF - 1 into the slot tile k-1 left: group 0 now,
    // the others during the score and P.V products
    const int kn = k + C::NBUF - 1;
    const bool more = kn < ntiles;
    const uint64_t sbn = more ? tile_src(kn) : 0;
    if (more) issue_group(kn, sbn, 0);

    char *tb = ring + (k % C::NBUF) * C::TILE;
    const int t0 = (int)((pg_begin + (uint32_t)(k / tpp)) * P) + (k % tpp) * C::T;
    const int valid = min(C::T, (int)tok_end - t0);
    char *vt = MLA ? tb : tb + C::TILE_K;
    if (valid < C::T) {
      // rows past the context may hold stale bytes: zero their V part so that
      // 0 * V stays 0 (their scores are masked to -inf below)
      const int nz = (C::T - valid) * (DV * 2 / 16);
      for (int i = threadIdx.x; i < nz; i += 64 * NW) {
        const int row = valid + i / (DV * 2 / 16), pc = i % (DV * 2 / 16);
        *reinterpret_cast<uint4 *>(vt + row * C::VPITCH + pc * 16) = make_uint4(0, 0, 0, 0);
      }
    }

    // ---- scores of this wave's heads, both 16-token slices
    f32x4 s[2][C::HBQ];
#pragma unroll
    for (int sl = 0; sl < 2; ++sl)
#pragma unroll
      for (int hb = 0; hb < C::HBQ; ++hb) s[sl][hb] = f32x4{0.f, 0.f, 0.f, 0.f};
    {
      const char *kr0 = tb + col * C::KPITCH + quad * 16;
      const char *kr1 = kr0 + 16 * C::KPITCH;
      // K fragments (k-step c, slice sl) are read KA k-steps ahead of
      // their products
      constexpr int KA = C::KA, NK = C::KSTEPS;
      bf16x8 kf[KA + 1][2];
#pragma unroll
      for (int c = 0; c < KA; ++c) {
        kf[c][0] = *reinterpret_cast<const bf16x8 *>(kr0 + 64 * c);
        kf[c][1] = *reinterpret_cast<const bf16x8 *>(kr1 + 64 * c);
      }
#pragma unroll
      for (int c = 0; c < NK; ++c) {
        if (c + KA < NK) {
          kf[(c + KA) % (KA + 1)][0] = *reinterpret_cast<const bf16x8 *>(kr0 + 64 * (c + KA));
          kf[(c + KA) % (KA + 1)][1] = *reinterpret_cast<const bf16x8 *>(kr1 + 64 * (c + KA));
        }
        if (NGRP > 1 && c == NK / 2 && more) issue_group(kn, sbn, 1);
#pragma unroll
        for (int hb = 0; hb < C::HBQ; ++hb) {
          const bf16x8 qv = c < C::QR ? qf[hb][c < C::QR ? c : 0]
                                      : *reinterpret_cast<const bf16x8 *>(
                                            qmine + ((hb * QL + (c - C::QR)) * 64 + lane) * 16);
#pragma unroll
          for (int sl = 0; sl < 2; ++sl)
            s[sl][hb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[c % (KA + 1)][sl], qv, s[sl][hb], 0, 0, 0);
        }
      }
    }
    // ---- online softmax per head (lane owns head column col; rows 4 quad + r).
    // Scores stay unscaled: the scale (positive) is applied to the column
    // maximum and folded into the exponent's fma.
    if (valid < C::T) {
#pragma unroll
      for (int sl = 0; sl < 2; ++sl)
#pragma unroll
        for (int hb = 0; hb < C::HBQ; ++hb)
#pragma unroll
          for (int r = 0; r < 4; ++r)
            if (16 * sl + 4 * quad + r >= valid) s[sl][hb][r] = -INFINITY;
    }
    bool bump = false;
    float mt[C::HBQ];
#pragma unroll
    for (int hb = 0; hb < C::HBQ; ++hb) {
      float x = s[0][hb][0];
#pragma unroll
      for (int sl = 0; sl < 2; ++sl)
#pragma unroll
        for (int r = 0; r < 4; ++r) x = x > s[sl][hb][r] ? x : s[sl][hb][r];
      x = xor_max_16_32(x) * sl2;
      mt[hb] = x;
      bump = bump || x > m[hb] + kLazy;
    }
    const bool any_bump = __builtin_amdgcn_ballot_w64(bump) != 0;
    if (any_bump) {
#pragma unroll
      for (int hb = 0; hb < C::HBQ; ++hb) {
        const float mn = mt[hb] > m[hb] + kLazy ? mt[hb] : m[hb];
        const float al = fast_exp2(m[hb] - mn);
        m[hb] = mn;
        lsum[hb] *= al;
        if (quad == 0) alpha_x[GW * wave + 16 * hb + col] = al;
      }
    }
    if (lane == 0) flags[wave] = any_bump ? 1 : 0;
#pragma unroll
    for (int hb = 0; hb < C::HBQ; ++hb) {
      bf16x8 pk;
      float ps = 0.f;
#pragma unroll
      for (int sl = 0; sl < 2; ++sl)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          // the row sum takes p in fp32; only the P.V operand is rounded to bf16
          const float p = fast_exp2(__builtin_fmaf(s[sl][hb][r], sl2, -m[hb]));
          ps += p;
          pk[4 * sl + r] = (__bf16)p;
        }
      lsum[hb] += ps;
      *reinterpret_cast<bf16x8 *>(pbuf + ((wave * C::HBQ + hb) * 64 + lane) * 16) = pk;
    }
    __syncthreads();  // P^T fragments, rescale factors and zeroed rows are visible

    // ---- rescale this wave's accumulators where a score wave moved its reference
    {
      int fl[NW];
      int any = 0;
#pragma unroll
      for (int w2 = 0; w2 < NW; ++w2) any |= fl[w2] = flags[w2];
      if (any != 0) {
#pragma unroll
        for (int hb = 0; hb < C::HB; ++hb) {
          if (fl[hb / C::HBQ]) {
            const float al = alpha_x[16 * hb + col];
#pragma unroll
            for (int db = 0; db < C::DBW; ++db) o[db][hb] *= al;
          }
        }
      }
    }
    if (more) {
#pragma unroll
      for (int g = 2; g < NGRP; ++g) issue_group(kn, sbn, g);
    }
    // ---- P.V for this wave's V columns, every head block
    {
      const int vrow = 4 * quad + (col >> 2);  // V row this lane supplies to the transpose read
      const char *vr0 = vt + vrow * C::VPITCH + 8 * (col & 3) + 32 * (wave * C::DBW);
      const char *vr1 = vr0 + 16 * C::VPITCH;
      constexpr int DH = C::DBW > 4 ? C::DBW / 2 : C::DBW;  // column blocks per pass
#pragma unroll
      for (int pass = 0; pass < C::DBW / DH; ++pass) {
        bf16x8 vf[DH];
#pragma unroll
        for (int j = 0; j < DH; ++j) {
          const int db = pass * DH + j;
          const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
              (__attribute__((address_space(3))) s16x4 *)(vr0 + 32 * db));
          const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
              (__attribute__((address_space(3))) s16x4 *)(vr1 + 32 * db));
          vf[j] = __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
        }
#pragma unroll
        for (int hb = 0; hb < C::HB; ++hb) {
          const bf16x8 pf = *reinterpret_cast<const bf16x8 *>(pbuf + (hb * 64 + lane) * 16);
#pragma unroll
          for (int j = 0; j < DH; ++j) {
            const int db = pass * DH + j;
            o[db][hb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf[j], pf, o[db][hb], 0, 0, 0);
          }
        }
      }
    }
  }

  // ---- final: score waves publish m and l; every wave normalises its columns
#pragma unroll
  for (int hb = 0; hb < C::HBQ; ++hb) {
    lsum[hb] = xor_sum_16_32(lsum[hb]);
  }
  __syncthreads();  // last tile's P area is no longer read
  if (quad == 0) {
#pragma unroll
    for (int hb = 0; hb < C::HBQ; ++hb) {
      alpha_x[GW * wave + 16 * hb + col] = m[hb];
      ml_x[GW * wave + 16 * hb + col] = lsum[hb];
    }
  }
  __syncthreads();
  const bool split = rq.ws_base != kNoWs;
#pragma unroll
  for (int hb = 0; hb < C::HB; ++hb) {
    const uint32_t head = (uint32_t)(h_kv + 16 * hb + col);
    const float inv = 1.0f / ml_x[16 * hb + col];
#pragma unroll
    for (int db = 0; db < C::DBW; ++db) {
      const int d = (DV / NW) * wave + 16 * db + 4 * quad;
      const f32x4 v = o[db][hb] * inv;
      uint16_t *dst = split ? a.ws_o + ((uint64_t)rq.ws_orow + (uint64_t)slot * gm.hq + head) * DV + d
                            : a.out + rq.o_off + head * DV + d;
      *reinterpret_cast<uint2 *>(dst) = bf16x4_bits(v[0], v[1], v[2], v[3]);
    }
  }
  if (quad == 0) {
#pragma unroll
    for (int hb = 0; hb < C::HBQ; ++hb) {
      const uint32_t head = (uint32_t)(h_kv + GW * wave + 16 * hb + col);
      const float lse = (m[hb] + fast_log2(lsum[hb])) * kLn2;
      if (split)
        a.ws_l[(uint64_t)rq.ws_base + (uint64_t)slot * gm.hq + head] = lse;
      else
        a.lse[rq.lse_off + head] = lse;
    }
  }
  __syncthreads();  // LDS is reused by the next unit
}

}  // namespace cp
