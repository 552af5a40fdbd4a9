// Cooperative matrix-core decode path for 16 or 32 query heads per KV head
// (MLA latent head; MQA/GQA with head_dim 128): the four waves of a
// workgroup share each tile of T = 16 * NS tokens, and tiles stream into a
// ring of NBUF LDS buffers so that NBUF - 1 tiles are in flight while one is
// used (a double buffer of large tiles would leave the memory pipe idle for
// one latency per tile).
//
// Per tile: wave w < NS computes S^T = K Q^T for tokens 16w .. 16w+15 and
// every head (mfma 16x16x32) and publishes its slice maximum per head; all
// waves take the tile maximum (same values, same decisions); the S waves
// publish P^T = exp2(S^T - m) of their slices as bf16 fragments; finally
// every wave accumulates O^T[its quarter of the V columns] += V^T P^T over
// the tile (mfma 16x16x16, V^T from the LDS transpose read).
// Each K and V byte is read from LDS once, no wave repeats another's work,
// and at the end of a segment every wave writes its own columns: there is no
// cross-wave merge. The softmax reference moves lazily as in the per-wave
// path (decode_mfma.h).
#pragma once

#include "decode_mfma.h"

namespace cp {

template <int HBW, int DK, int DV, bool MLA, int NS, int NBUF_>
struct CoopCfg {
  static constexpr int NW = 4, T = 16 * NS, NBUF = NBUF_;  // waves, tile tokens, ring buffers
  static constexpr int KROW = DK * 2;
  static constexpr int VROW = MLA ? KROW : DV * 2;
  static constexpr int KPITCH = KROW + 16;
  static constexpr int VPITCH = MLA ? KPITCH : VROW + 16;
  static constexpr int TILE_K = T * KPITCH;
  static constexpr int TILE_V = MLA ? 0 : T * VPITCH;
  static constexpr int TILE_USED = TILE_K + TILE_V;
  static constexpr int DMA_WAVE = (TILE_USED + 1024 * NW - 1) / (1024 * NW);
  static constexpr int TILE = DMA_WAVE * NW * 1024;
  static constexpr int BUF = (NBUF * TILE + 1) / 2;  // the ring spans the kernel's two LDS buffers
  static constexpr int KSTEPS = DK / 32;
  static constexpr int NBLK = DV / 16;
  static constexpr int NBW = NBLK / NW;  // V column blocks per wave
  static constexpr int HEADS = 16 * HBW;
  static constexpr int KB = KSTEPS % 6 == 0 ? 6 : (KSTEPS % 4 == 0 ? 4 : 2);
  static constexpr int VB = NBW >= 8 ? 4 : NBW;
  static_assert(BUF <= kLdsBuf, "tile does not fit");
  static_assert(NBLK % NW == 0 && NBW % VB == 0 && KSTEPS % KB == 0, "uneven split");
  static_assert(HBW <= 2, "exchange area holds two head blocks");
  static_assert(DMA_WAVE * (NBUF - 1) <= 48, "too many loads in flight per wave");
  static_assert(NS >= 1 && NS <= NW, "one S wave per slice");
};

// LDS exchange area (inside `red`): slice maxima [NW][HEADS], row sums
// [NW][HEADS], and P^T fragments [NW][HBW][64 lanes] of 8 bytes.
constexpr int kXm = 0, kXl = 4 * 64, kXp = 8 * 64;

template <int N>
CP_DEV void wait_tiles(int n) {  // wait until at most n tiles of N loads each are outstanding
  if (n <= 0)
    wait_vm<0>();
  else if (n == 1)
    wait_vm<N>();
  else
    wait_vm<2 * N>();
}

template <int HBW, int DK, int DV, bool MLA, int NS, int NBUF>
__device__ __forceinline__ void coop_unit(const DecodeArgs &a, const GeomK &gm, const DecReq &rq, const Seg &sg,
                                          char *buf0, char *buf1, float *red) {
  using C = CoopCfg<HBW, DK, DV, MLA, NS, NBUF>;
  static_assert(NBUF <= 3, "wait_tiles covers up to two tiles in flight");
  const uint32_t kvh = sg.hblk, slot = sg.slot;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int col = lane & 15, quad = lane >> 4;
  const int P = gm.page_tokens;  // the host routes only 64-token pages here
  const int tpp = P / C::T;        // tiles per page
  const int h0 = (int)kvh * C::HEADS;
  float *m_x = red + kXm, *l_x = red + kXl;
  s16x4 *p_x = reinterpret_cast<s16x4 *>(red + kXp);

  // Q^T fragments: lane holds head (h0 + 16*hb + col), dims 32c + 8*quad .. +7.
  bf16x8 qf[HBW][C::KSTEPS];
#pragma unroll
  for (int hb = 0; hb < HBW; ++hb)
#pragma unroll
    for (int c = 0; c < C::KSTEPS; ++c)
      qf[hb][c] = *reinterpret_cast<const bf16x8 *>(a.q + rq.q_off + (uint32_t)(h0 + 16 * hb + col) * DK +
                                                   32 * c + 8 * quad);

  const uint32_t tok_end = min(rq.ctx_len, sg.pg_end * (uint32_t)P);
  const uint32_t pg_begin = sg.pg_begin;
  const int npg = (int)((tok_end + P - 1) / P) - (int)pg_begin;
  const int last_tok = npg > 0 ? (int)tok_end - (int)((pg_begin + (uint32_t)npg - 1) * (uint32_t)P) : 0;
  const int ntiles = npg > 0 ? (npg - 1) * tpp + (last_tok + C::T - 1) / C::T : 0;
  const uint64_t kv_head_bytes = MLA ? 0 : (uint64_t)2 * P * DK * 2;

  uint32_t pte_lane = 0;
  int pte_batch = -1;
  auto load_ptes = [&](int batch) {
    const int sp = batch * 64 + lane;
    pte_lane = sp < npg ? a.pte[rq.pte_base + pg_begin + (uint32_t)sp] : 0u;
    pte_batch = batch;
  };
  // Direct loads of tile k into its ring slot; each wave fetches a quarter.
  char *const ring = buf0;  // NBUF * TILE bytes across the two kernel buffers
  (void)buf1;
  auto issue = [&](int k) {
    char *dst = ring + (k % NBUF) * C::TILE;
    const int sp = k / tpp;  // page within the segment
    if ((sp >> 6) != pte_batch) load_ptes(sp >> 6);
    const uint32_t pte = __builtin_amdgcn_readlane(pte_lane, sp & 63);
    const uint64_t sbase = uniform_ptr(a.pool + ((uint64_t)pte << 8) + kvh * kv_head_bytes +
                                       (uint64_t)(k % tpp) * C::T * C::KROW);
    const uint32_t ldsb = lds_addr(dst);
#pragma unroll
    for (int i = 0; i < C::DMA_WAVE; ++i) {
      const int inst = wave * C::DMA_WAVE + i;
      const int o = inst * 1024 + lane * 16;
      // pad lanes and lanes past the tile refetch the start of a row
      uint32_t off;
      if (C::TILE_V == 0 || o < C::TILE_K) {
        const int oc = o < C::TILE_K ? o : 0;
        const int row = oc / C::KPITCH, w = oc - row * C::KPITCH;
        off = (uint32_t)(row * C::KROW + (w < C::KROW ? w : 0));
      } else {
        const int o2 = o < C::TILE_USED ? o - C::TILE_K : 0;
        const int row = o2 / C::VPITCH, w = o2 - row * C::VPITCH;
        off = (uint32_t)(P * DK * 2 + row * C::VROW + (w < C::VROW ? w : 0));  // V rows follow the P K rows
      }
      dma16_sbase(sbase, off, __builtin_amdgcn_readfirstlane(ldsb + inst * 1024));
    }
  };

  float m[HBW], lsum[HBW];
  f32x4 o[HBW][C::NBW];
#pragma unroll
  for (int hb = 0; hb < HBW; ++hb) {
    m[hb] = -INFINITY;
    lsum[hb] = 0.f;
#pragma unroll
    for (int nb = 0; nb < C::NBW; ++nb) o[hb][nb] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  const float sl2 = gm.scale_log2;
  const int vrow_l = 4 * quad + (col >> 2);  // V row this lane supplies to a transpose read
  const int va = col & 3;

  auto compute = [&](int k) {
    char *tb = ring + (k % NBUF) * C::TILE;
    const int valid = min(C::T, (int)tok_end - (int)((pg_begin + (uint32_t)(k / tpp)) * P) - (k % tpp) * C::T);
    const char *kt = tb;
    char *vt = MLA ? tb : tb + C::TILE_K;
    if (valid < C::T) {
      // rows past the context may hold stale bytes: zero their V part
      const int nz = (C::T - valid) * (DV * 2 / 16);
      for (int i = threadIdx.x; i < nz; i += 64 * C::NW) {
        const int row = valid + i / (DV * 2 / 16), pc = i % (DV * 2 / 16);
        *reinterpret_cast<uint4 *>(vt + row * C::VPITCH + pc * 16) = make_uint4(0, 0, 0, 0);
      }
    }
    // S^T of this wave's 16-token slice, K fragments pipelined in batches
    const bool swave = wave < NS;
    // NACC independent accumulators per head block break the dependent MFMA
    // chain over the K steps (a chain runs at MFMA latency, not throughput)
    constexpr int NACC = C::KSTEPS % 3 == 0 ? 3 : 2;
    f32x4 s[HBW], sacc[NACC][HBW];
#pragma unroll
    for (int hb = 0; hb < HBW; ++hb) {
      s[hb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int u = 0; u < NACC; ++u) sacc[u][hb] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
    if (swave) {
      const char *kr = kt + (16 * wave + col) * C::KPITCH + quad * 16;
      constexpr int KB = C::KB, NKB = C::KSTEPS / KB;
      bf16x8 kf[2][KB];
#pragma unroll
      for (int j = 0; j < KB; ++j) kf[0][j] = *reinterpret_cast<const bf16x8 *>(kr + 64 * j);
#pragma unroll
      for (int b = 0; b < NKB; ++b) {
        if (b + 1 < NKB) {
#pragma unroll
          for (int j = 0; j < KB; ++j)
            kf[(b + 1) & 1][j] = *reinterpret_cast<const bf16x8 *>(kr + 64 * ((b + 1) * KB + j));
        }
#pragma unroll
        for (int j = 0; j < KB; ++j) {
          const int u = (b * KB + j) % NACC;
#pragma unroll
          for (int hb = 0; hb < HBW; ++hb)
            sacc[u][hb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[b & 1][j], qf[hb][b * KB + j], sacc[u][hb], 0, 0, 0);
        }
        __builtin_amdgcn_sched_barrier(0);
      }
#pragma unroll
      for (int hb = 0; hb < HBW; ++hb) {
        s[hb] = sacc[0][hb];
#pragma unroll
        for (int u = 1; u < NACC; ++u) s[hb] += sacc[u][hb];
      }
    }
    // slice maxima -> tile maxima (identical in every wave)
#pragma unroll
    for (int hb = 0; hb < HBW; ++hb) {
      float x = -INFINITY;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float v = 16 * wave + 4 * quad + r < valid ? s[hb][r] * sl2 : -INFINITY;
        s[hb][r] = v;
        x = fmaxf(x, v);
      }
      x = fmaxf(x, __shfl_xor(x, 16, 64));
      x = fmaxf(x, __shfl_xor(x, 32, 64));
      if (swave && quad == 0) m_x[wave * C::HEADS + 16 * hb + col] = x;
    }
    __syncthreads();
    bool bump = false;
    float mt[HBW];
#pragma unroll
    for (int hb = 0; hb < HBW; ++hb) {
      float x = m_x[16 * hb + col];
#pragma unroll
      for (int w2 = 1; w2 < NS; ++w2) x = fmaxf(x, m_x[w2 * C::HEADS + 16 * hb + col]);
      mt[hb] = x;
      bump = bump || x > m[hb] + kLazy;
    }
    if (__builtin_amdgcn_ballot_w64(bump)) {
#pragma unroll
      for (int hb = 0; hb < HBW; ++hb) {
        const float mn = mt[hb] > m[hb] + kLazy ? mt[hb] : m[hb];
        const float alpha = fast_exp2(m[hb] - mn);
        m[hb] = mn;
        lsum[hb] *= alpha;
#pragma unroll
        for (int nb = 0; nb < C::NBW; ++nb) o[hb][nb] *= alpha;
      }
    }
    // P^T of this slice: fp32 into the row sum, bf16 to the exchange area
#pragma unroll
    for (int hb = 0; hb < HBW; ++hb) {
      s16x4 pk;
      float ps = 0.f;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float p = fast_exp2(s[hb][r] - m[hb]);
        ps += p;
        pk[r] = __builtin_bit_cast(short, (__bf16)p);
      }
      if (swave) {
        lsum[hb] += ps;
        p_x[(wave * HBW + hb) * 64 + lane] = pk;
      }
    }
    __syncthreads();
    // O^T[this wave's columns] += V^T P^T over the tile's slices
#pragma unroll
    for (int sl = 0; sl < NS; ++sl) {
      s16x4 pf[HBW];
#pragma unroll
      for (int hb = 0; hb < HBW; ++hb) pf[hb] = p_x[(sl * HBW + hb) * 64 + lane];
      const char *vr = vt + (16 * sl + vrow_l) * C::VPITCH + 8 * va + 32 * (wave * C::NBW);
      constexpr int VB = C::VB, NVB = C::NBW / VB;
      s16x4 vf[2][VB];
#pragma unroll
      for (int j = 0; j < VB; ++j)
        vf[0][j] = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4 *)(vr + 32 * j));
#pragma unroll
      for (int b = 0; b < NVB; ++b) {
        if (b + 1 < NVB) {
#pragma unroll
          for (int j = 0; j < VB; ++j)
            vf[(b + 1) & 1][j] = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                (__attribute__((address_space(3))) s16x4 *)(vr + 32 * ((b + 1) * VB + j)));
        }
#pragma unroll
        for (int j = 0; j < VB; ++j)
#pragma unroll
          for (int hb = 0; hb < HBW; ++hb)
            o[hb][b * VB + j] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(vf[b & 1][j], pf[hb], o[hb][b * VB + j], 0, 0, 0);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
  };

  // Ring of NBUF tiles: tiles k+1 .. k+NBUF-1 stream in while tile k is
  // used; the slot of tile k+NBUF-1 was released by the barrier that closed
  // tile k-1.
  if (ntiles > 0) load_ptes(0);
  for (int k = 0; k < NBUF - 1 && k < ntiles; ++k) issue(k);
#pragma unroll 1
  for (int k = 0; k < ntiles; ++k) {
    if (k + NBUF - 1 < ntiles) issue(k + NBUF - 1);
    wait_tiles<C::DMA_WAVE>(min(NBUF - 1, ntiles - 1 - k));
    __syncthreads();  // every wave's share of tile k has landed
    compute(k);
    __syncthreads();  // tile k's slot and the exchange area are free again
  }

  // Row sums: lanes hold a quarter of the slice, waves a quarter of the tile.
#pragma unroll
  for (int hb = 0; hb < HBW; ++hb) {
    float x = lsum[hb];
    x += __shfl_xor(x, 16, 64);
    x += __shfl_xor(x, 32, 64);
    if (quad == 0) l_x[wave * C::HEADS + 16 * hb + col] = x;
  }
  __syncthreads();
  const bool split = rq.ws_base != kNoWs;
#pragma unroll
  for (int hb = 0; hb < HBW; ++hb) {
    float L = 0.f;
#pragma unroll
    for (int w2 = 0; w2 < C::NW; ++w2) L += l_x[w2 * C::HEADS + 16 * hb + col];
    const uint32_t head = (uint32_t)(h0 + 16 * hb + col);
    const float inv = 1.0f / L;
#pragma unroll
    for (int nb = 0; nb < C::NBW; ++nb) {
      const int d = 16 * (wave * C::NBW + nb) + 4 * quad;
      const f32x4 v = o[hb][nb] * inv;
      if (split) {
        *reinterpret_cast<f32x4 *>(a.ws_o + ((uint64_t)rq.ws_orow + (uint64_t)slot * gm.hq + head) * DV + d) = v;
      } else {
        uint2 pk;
        pk.x = f32_to_bf16(v[0]) | (f32_to_bf16(v[1]) << 16);
        pk.y = f32_to_bf16(v[2]) | (f32_to_bf16(v[3]) << 16);
        *reinterpret_cast<uint2 *>(a.out + rq.o_off + head * DV + d) = pk;
      }
    }
    if (wave == 0 && quad == 0) {
      const float lse = (m[hb] + fast_log2(L)) * kLn2;
      if (split)
        a.ws_l[(uint64_t)rq.ws_base + (uint64_t)slot * gm.hq + head] = lse;
      else
        a.lse[rq.lse_off + head] = lse;
    }
  }
  __syncthreads();  // the exchange area is reused by the next segment
}

}  // namespace cp
