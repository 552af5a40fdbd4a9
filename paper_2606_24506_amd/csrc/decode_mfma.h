// Matrix-core decode path for models whose query heads share a KV head in
// groups of 16 or more (MLA latent head; MQA/GQA with g >= 16), where the
// per-KV-head work is a real dense contraction.
//
// Per 16-token slice of a KV tile, with heads h of one 16-head block:
//   S^T[t][h]  = sum_d K[t][d] Q[h][d]          (mfma 16x16x32 bf16; A = K
//                                                rows from LDS, B = Q^T held
//                                                in registers)
//   P = exp2(S^T * scale*log2e - m)              (fp32 online softmax; m, l per
//                                                head; rounded to bf16 for PV)
//   O^T[d][h] += sum_t V^T[d][t] P^T[t][h]      (mfma 16x16x16 bf16; A = V^T
//                                                via the LDS transpose read,
//                                                B = P^T straight from the S^T
//                                                accumulator layout)
// so every lane owns one head column throughout and the softmax rescale is
// lane-local. KV tiles stream HBM -> LDS with direct LDS loads (no VGPR
// staging), double-buffered; 16-byte chunks of each row are XOR-swizzled by
// (row mod 8) to spread LDS banks.
#pragma once

#include <hip/hip_runtime.h>

#include "device_common.h"
#include "kargs.h"

namespace cp {

typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

constexpr int kLdsBuf = 77824;  // bytes per KV buffer (two buffers)
constexpr int kRedFloats = 1536;  // reduction / exchange floats
constexpr float kLazy = 8.0f;  // log2 headroom before the softmax reference moves

// Direct HBM -> LDS load of 16 bytes per lane: lane i writes
// lds_base + 16 * i. Issued through inline asm so the compiler does not
// insert a full vmcnt wait before every LDS read; completion is awaited with
// wait_vm<N>() below. KV is streamed once per call, so the loads carry the
// non-temporal policy (nt): on MI355X this lifts page-scattered reads from
// about 4.7 to about 6.8 TB/s.
// M0 is set inside the same statement; nothing else in these kernels uses it.
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
CP_DEV void dma16(const void *g, uint32_t lds_base) {
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off nt" ::"v"(g), "s"(lds_base) : "memory", "m0");
}
// Same with a wave-uniform base address in SGPRs and a 32-bit per-lane
// byte offset.
CP_DEV void dma16_sbase(uint64_t sbase, uint32_t voff, uint32_t lds_base) {
  asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1 nt" ::"v"(voff), "s"(sbase), "s"(lds_base)
               : "memory", "m0");
}

// A pointer known to be the same in every lane, moved to scalar registers.
CP_DEV uint64_t uniform_ptr(const void *p) {
  const uint64_t v = (uint64_t)(uintptr_t)p;
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(v >> 32));
  return ((uint64_t)hi << 32) | lo;
}
#pragma clang diagnostic pop

template <int N>
CP_DEV void wait_vm() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

CP_DEV uint32_t lds_addr(const void *p) { return (uint32_t)(uintptr_t)p; }

template <int HBW, int WPT, int NW, int DK, int DV, int T, bool MLA>
struct MfmaCfg {
  static constexpr int KROW = DK * 2;  // bytes of one K row in HBM
  static constexpr int VROW = MLA ? KROW : DV * 2;
  static constexpr int KPITCH = KROW + 16;  // ... and in LDS
  static constexpr int VPITCH = MLA ? KPITCH : VROW + 16;
  static constexpr int TILE_K = T * KPITCH;
  static constexpr int TILE_V = MLA ? 0 : T * VPITCH;
  static constexpr int TILE_USED = TILE_K + TILE_V;
  static constexpr int DMA_WAVE = (TILE_USED + 1024 * WPT - 1) / (1024 * WPT);  // direct loads per wave per tile
  static constexpr int TILE = DMA_WAVE * WPT * 1024;  // LDS bytes of one tile
  static constexpr int GROUPS = NW / WPT;             // independent tile streams per workgroup
  static constexpr int NSUB = T / 16;
  static constexpr int KSTEPS = DK / 32;
  static constexpr int NBLK = DV / 16;
  static constexpr int HEADS = 16 * HBW * WPT;  // query heads per KV head
  static constexpr int BUF = GROUPS * TILE;     // bytes of one of the two KV buffers
  // LDS fragment batches of the software pipelines (smaller when 8 waves
  // share a SIMD pair and registers are scarce)
  static constexpr int KB = KSTEPS % 6 == 0 && NW < 8 ? 6 : (KSTEPS % 3 == 0 ? 3 : 2);
  static constexpr int VB = NW < 8 ? 8 : 4;
  static_assert(KSTEPS % KB == 0 && NBLK % VB == 0, "batches must tile the steps");
  static_assert(BUF <= kLdsBuf, "tile does not fit");
  static_assert(GROUPS == 1 || WPT == 1, "streams of several waves need their own barriers");
  static_assert(DMA_WAVE <= 24, "too many loads in flight per wave");
};

// One unit: the heads of KV head `kvh` over the pages of one KV range.
// Waves form GROUPS tile streams of WPT waves; a stream takes every
// GROUPS-th page of the range, and its WPT waves split the head blocks.
template <int HBW, int WPT, int NW, int DK, int DV, int T, bool MLA>
__device__ __forceinline__ void mfma_unit(const DecodeArgs &a, const GeomK &gm, const DecReq &rq, const Seg &sg,
                                          char *buf0, char *buf1, float *red) {
  const uint32_t kvh = sg.hblk, chunk = sg.slot;
  using C = MfmaCfg<HBW, WPT, NW, DK, DV, T, MLA>;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int grp = wave / WPT, wig = wave % WPT;
  const int col = lane & 15, quad = lane >> 4;
  const int P = gm.page_tokens;
  const int h_wave = (int)kvh * C::HEADS + wig * 16 * HBW;  // first head of this wave

  // Q^T fragments: lane holds head (h_wave + 16*hb + col), dims 32c + 8*quad .. +7.
  bf16x8 qf[HBW][C::KSTEPS];
#pragma unroll
  for (int hb = 0; hb < HBW; ++hb)
#pragma unroll
    for (int c = 0; c < C::KSTEPS; ++c)
      qf[hb][c] = *reinterpret_cast<const bf16x8 *>(a.q + rq.q_off + (uint32_t)(h_wave + 16 * hb + col) * DK +
                                                   32 * c + 8 * quad);

  const uint32_t tok_end = min(rq.ctx_len, sg.pg_end * (uint32_t)P);
  const uint32_t pg_begin = sg.pg_begin;
  const uint32_t pg_end = (tok_end + P - 1) / P;
  const int tpp = P / T;  // tiles per page
  // The segment's tiles in page-major order; stream grp takes tiles grp,
  // grp + GROUPS, ... so streams differ by at most one tile of work.
  const int npg = (int)pg_end - (int)pg_begin;
  const int last_tok = npg > 0 ? (int)tok_end - (int)((pg_end - 1) * (uint32_t)P) : 0;
  const int seg_tiles = npg > 0 ? (npg - 1) * tpp + (last_tok + T - 1) / T : 0;
  const int ntiles = seg_tiles > grp ? (seg_tiles - grp + C::GROUPS - 1) / C::GROUPS : 0;
  const uint64_t kv_head_bytes = MLA ? 0 : (uint64_t)2 * P * DK * 2;
  char *const tb0 = buf0 + grp * C::TILE;
  char *const tb1 = buf1 + grp * C::TILE;

  // Page-table entries of the segment's pages, 64 at a time: lane i holds
  // the entry of page (64 * batch + i). Loading them ahead of the tile loop
  // keeps vector loads of the page table (and the full vmcnt wait the
  // compiler puts after them) out of the per-tile path.
  uint32_t pte_lane = 0;
  int pte_batch = -1;
  auto load_ptes = [&](int batch) {
    const int sp = batch * 64 + lane;  // page index within the segment
    pte_lane = sp < npg ? a.pte[rq.pte_base + pg_begin + (uint32_t)sp] : 0u;
    pte_batch = batch;
  };

  // Issue the direct loads of tile k into tile buffer `dst`.
  auto issue = [&](int k, char *dst) {
    const int t = grp + C::GROUPS * k;  // tile within the segment
    const int sp = t / tpp;
    if ((sp >> 6) != pte_batch) load_ptes(sp >> 6);
    const uint32_t t0 = (uint32_t)(t % tpp) * T;
    const uint32_t pte = __builtin_amdgcn_readlane(pte_lane, sp & 63);
    // uniform base of the KV head's block in this page; K rows of the tile
    // start t0 rows in, V rows P rows after the K rows (GQA layout)
    const uint8_t *base = a.pool + ((uint64_t)pte << 8) + kvh * kv_head_bytes + (uint64_t)t0 * C::KROW;
    const uint32_t ldsb = lds_addr(dst);
    const uint64_t sbase = uniform_ptr(base);
#pragma unroll
    for (int i = 0; i < C::DMA_WAVE; ++i) {
      const int inst = wig * C::DMA_WAVE + i;
      const int o = inst * 1024 + lane * 16;  // byte offset inside the LDS tile
      // Lanes that land on a row's 16-byte pad, or past the tile, fetch the
      // first 16 bytes of a row they already cover (same cache lines), so
      // every load is issued by all lanes without branches.
      uint32_t off;
      if (C::TILE_V == 0 || o < C::TILE_K) {
        const int oc = o < C::TILE_K ? o : 0;
        const int row = oc / C::KPITCH, w = oc - row * C::KPITCH;
        off = (uint32_t)(row * C::KROW + (w < C::KROW ? w : 0));
      } else {
        const int o2 = o < C::TILE_USED ? o - C::TILE_K : 0;
        const int row = o2 / C::VPITCH, w = o2 - row * C::VPITCH;
        off = (uint32_t)(P * DK * 2 + row * C::VROW + (w < C::VROW ? w : 0));
      }
      dma16_sbase(sbase, off, __builtin_amdgcn_readfirstlane(ldsb + inst * 1024));
    }
  };

  float m[HBW], lsum[HBW];
  f32x4 o[HBW][C::NBLK];
#pragma unroll
  for (int hb = 0; hb < HBW; ++hb) {
    m[hb] = -INFINITY;
    lsum[hb] = 0.f;
#pragma unroll
    for (int nb = 0; nb < C::NBLK; ++nb) o[hb][nb] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  const float sl2 = gm.scale_log2;

  auto compute = [&](int k, char *tb) {
    const int t = grp + C::GROUPS * k;  // tile within the segment
    const int t0 = (int)((pg_begin + (uint32_t)(t / tpp)) * P) + (t % tpp) * T;  // first token of the tile
    const int valid = min(T, (int)tok_end - t0);
    const char *kt = tb;
    char *vt = MLA ? tb : tb + C::TILE_K;
    if (valid < T) {
      // rows past the context may hold stale bytes: zero their V part so
      // that 0 * V stays 0 in the PV product
      const int nz = (T - valid) * (DV * 2 / 16);
      for (int i = wig * 64 + lane; i < nz; i += 64 * WPT) {
        const int row = valid + i / (DV * 2 / 16), pc = i % (DV * 2 / 16);
        *reinterpret_cast<uint4 *>(vt + row * C::VPITCH + pc * 16) = make_uint4(0, 0, 0, 0);
      }
      if (WPT > 1) __syncthreads();
    }
    // One 16-token slice at a time: S^T, online softmax, then PV.
    const int vrow_l = 4 * quad + (col >> 2);  // V row this lane supplies to the transpose read
    const int va = col & 3;
#pragma unroll 1
    for (int sub = 0; sub < C::NSUB; ++sub) {
      // NACC independent accumulators break the dependent MFMA chain
      constexpr int NACC = C::KSTEPS % 3 == 0 ? 3 : 2;
      f32x4 s[HBW], sacc[NACC][HBW];
#pragma unroll
      for (int hb = 0; hb < HBW; ++hb)
#pragma unroll
        for (int u = 0; u < NACC; ++u) sacc[u][hb] = f32x4{0.f, 0.f, 0.f, 0.f};
      {
        // K fragments in batches of KB: batch b+1 is read while batch b
        // feeds the matrix cores.
        const char *kr = kt + (sub * 16 + col) * C::KPITCH + quad * 16;
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
      }
#pragma unroll
      for (int hb = 0; hb < HBW; ++hb) {
        s[hb] = sacc[0][hb];
#pragma unroll
        for (int u = 1; u < NACC; ++u) s[hb] += sacc[u][hb];
      }
      // Online softmax; lane owns head column `col`, tokens sub*16 + 4*quad + r.
      // The reference maximum m only moves when the slice maximum exceeds it
      // by more than kLazy (log2 units), so p <= 2^kLazy and the accumulator
      // rescale (a pass over every O register) is rare. Numerator and
      // denominator always share the same reference, so the result is the
      // same softmax.
      bool bump = false;
      float mt[HBW];
#pragma unroll
      for (int hb = 0; hb < HBW; ++hb) {
        float x = -INFINITY;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int tk = sub * 16 + 4 * quad + r;
          const float v = tk < valid ? s[hb][r] * sl2 : -INFINITY;
          s[hb][r] = v;
          x = fmaxf(x, v);
        }
        x = fmaxf(x, __shfl_xor(x, 16, 64));
        x = fmaxf(x, __shfl_xor(x, 32, 64));
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
          for (int nb = 0; nb < C::NBLK; ++nb) o[hb][nb] *= alpha;
        }
      }
      s16x4 pf[HBW];
#pragma unroll
      for (int hb = 0; hb < HBW; ++hb) {
        float ps = 0.f;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          // the row sum takes p in fp32; only the PV operand is rounded to bf16
          const float p = fast_exp2(s[hb][r] - m[hb]);
          ps += p;
          pf[hb][r] = __builtin_bit_cast(short, (__bf16)p);
        }
        lsum[hb] += ps;
      }
      // O^T += V^T P^T; the transpose read gives lane (4a+b) of each 16-lane
      // quarter column (4a+b) of four V rows supplied by lanes a, 4+a, 8+a, 12+a.
      const char *vr = vt + (sub * 16 + vrow_l) * C::VPITCH + 8 * va;
      {
        // V^T fragments in batches of VB, software-pipelined like K.
        constexpr int VB = C::VB, NVB = C::NBLK / VB;
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
    }
  };

  // Double-buffered tile loop: tile k+1 streams in while tile k is used.
  if (ntiles > 0) {
    load_ptes(0);
    issue(0, tb0);
  }
#pragma unroll 1
  for (int k = 0; k < ntiles; ++k) {
    char *cur = (k & 1) ? tb1 : tb0;
    if (k + 1 < ntiles) {
      issue(k + 1, (k & 1) ? tb0 : tb1);
      wait_vm<C::DMA_WAVE>();
    } else {
      wait_vm<0>();
    }
    if (WPT > 1) __syncthreads();
    compute(k, cur);
    if (WPT > 1) __syncthreads();
  }

  // Row sums: each lane holds a quarter of its head's tokens.
#pragma unroll
  for (int hb = 0; hb < HBW; ++hb) {
    lsum[hb] += __shfl_xor(lsum[hb], 16, 64);
    lsum[hb] += __shfl_xor(lsum[hb], 32, 64);
  }
  const bool split = rq.ws_base != kNoWs;

  if constexpr (C::GROUPS == 1) {
    // The workgroup's waves own disjoint heads: write straight from registers.
#pragma unroll
    for (int hb = 0; hb < HBW; ++hb) {
      const uint32_t head = (uint32_t)(h_wave + 16 * hb + col);
      const float inv = 1.0f / lsum[hb];
      const float lse = (m[hb] + fast_log2(lsum[hb])) * kLn2;
#pragma unroll
      for (int nb = 0; nb < C::NBLK; ++nb) {
        const int d = 16 * nb + 4 * quad;
        const f32x4 v = o[hb][nb] * inv;
        if (split) {
          float *dst = a.ws_o + ((uint64_t)rq.ws_orow + (uint64_t)chunk * gm.hq + head) * DV + d;
          *reinterpret_cast<f32x4 *>(dst) = v;
        } else {
          uint2 pk;
          pk.x = f32_to_bf16(v[0]) | (f32_to_bf16(v[1]) << 16);
          pk.y = f32_to_bf16(v[2]) | (f32_to_bf16(v[3]) << 16);
          *reinterpret_cast<uint2 *>(a.out + rq.o_off + head * DV + d) = pk;
        }
      }
      if (quad == 0) {
        if (split)
          a.ws_l[(uint64_t)rq.ws_base + (uint64_t)chunk * gm.hq + head] = lse;
        else
          a.lse[rq.lse_off + head] = lse;
      }
    }
    return;
  }

  // Several streams hold partial states of the same heads: combine them in
  // stream order through LDS. red: m[GROUPS][HEADS], l[GROUPS][HEADS].
  constexpr int HD = C::HEADS;
  float *m_s = red, *l_s = red + 4 * 128;
  __syncthreads();
  if (quad == 0) {
#pragma unroll
    for (int hb = 0; hb < HBW; ++hb) {
      const int hl = wig * 16 * HBW + 16 * hb + col;  // head within the KV head
      m_s[grp * HD + hl] = m[hb];
      l_s[grp * HD + hl] = lsum[hb];
    }
  }
  __syncthreads();
  float f[HBW], Lt[HBW];
#pragma unroll
  for (int hb = 0; hb < HBW; ++hb) {
    const int hl = wig * 16 * HBW + 16 * hb + col;
    float M = -INFINITY;
    for (int g2 = 0; g2 < C::GROUPS; ++g2) M = fmaxf(M, m_s[g2 * HD + hl]);
    float L = 0.f;
    for (int g2 = 0; g2 < C::GROUPS; ++g2) L += l_s[g2 * HD + hl] * fast_exp2(m_s[g2 * HD + hl] - M);
    f[hb] = fast_exp2(m[hb] - M);
    Lt[hb] = L;
    if (grp == 0 && quad == 0) {
      red[8 * 128 + hl] = M;
      red[8 * 128 + 128 + hl] = L;
    }
  }
  constexpr int PAD = DV + 4;
  float *acc = reinterpret_cast<float *>(buf0);  // [HEADS][DV + 4]
  static_assert(C::GROUPS == 1 || HD * PAD * 4 <= C::BUF, "merge buffer does not fit in the KV buffer");
  for (int g2 = 0; g2 < C::GROUPS; ++g2) {
    if (grp == g2) {
#pragma unroll
      for (int hb = 0; hb < HBW; ++hb) {
        const int hl = wig * 16 * HBW + 16 * hb + col;
#pragma unroll
        for (int nb = 0; nb < C::NBLK; ++nb) {
          f32x4 *dst = reinterpret_cast<f32x4 *>(acc + hl * PAD + 16 * nb + 4 * quad);
          const f32x4 v = o[hb][nb] * f[hb];
          *dst = (g2 == 0) ? v : *dst + v;
        }
      }
    }
    __syncthreads();
  }
  (void)Lt;
  // Normalise and write, four consecutive values per thread.
  const uint32_t h_base = kvh * HD;
  for (int i = threadIdx.x; i < HD * DV / 4; i += 64 * NW) {
    const int hl = (4 * i) / DV, d = (4 * i) % DV;
    const float inv = 1.0f / red[8 * 128 + 128 + hl];
    const f32x4 v = *reinterpret_cast<const f32x4 *>(acc + hl * PAD + d) * inv;
    const uint32_t head = h_base + hl;
    if (split) {
      *reinterpret_cast<f32x4 *>(a.ws_o + ((uint64_t)rq.ws_orow + (uint64_t)chunk * gm.hq + head) * DV + d) = v;
    } else {
      uint2 pk;
      pk.x = f32_to_bf16(v[0]) | (f32_to_bf16(v[1]) << 16);
      pk.y = f32_to_bf16(v[2]) | (f32_to_bf16(v[3]) << 16);
      *reinterpret_cast<uint2 *>(a.out + rq.o_off + head * DV + d) = pk;
    }
  }
  for (int hl = threadIdx.x; hl < HD; hl += 64 * NW) {
    const float lse = (red[8 * 128 + hl] + fast_log2(red[8 * 128 + 128 + hl])) * kLn2;
    const uint32_t head = h_base + hl;
    if (split)
      a.ws_l[(uint64_t)rq.ws_base + (uint64_t)chunk * gm.hq + head] = lse;
    else
      a.lse[rq.lse_off + head] = lse;
  }
  __syncthreads();
}

}  // namespace cp
