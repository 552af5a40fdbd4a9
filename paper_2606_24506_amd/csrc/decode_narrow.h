// Matrix-core decode path for 8 to 32 query heads per KV head (MLA-16/32
// on one latent head; MQA and GQA groups with head_dim 128). Per KV byte
// there are only 8-32 flops here, so the kernel is built to hide memory and
// LDS latency rather than to feed the matrix cores: a workgroup of NW = 8
// waves (two per SIMD, so one wave's stalls are the other's issue slots)
// forms NW / SHARE token streams. A stream walks its own slices of TW
// tokens through a private ring of NSLOT LDS slots with its own online
// softmax; streams only meet when the unit ends. With SHARE = 2 the two
// waves of a stream both compute the (cheap) scores of every slice and each
// accumulates P.V for half of the V columns, which halves the accumulator
// registers so that two waves fit a SIMD; every K byte is then read from
// LDS twice and every V byte once.
//
// Per slice and 16-head block (a group of 8 heads is padded to 16):
//   S^T[t][h] = sum_d K[t][d] Q[h][d]    mfma 16x16x32 bf16 (K rows from LDS
//                                       as A, Q^T in registers as B; two or
//                                       three independent accumulator chains)
//   fp32 online softmax with a lazily moved reference maximum
//   O^T[d][h] += sum_t V^T[d][t] P^T[t][h]
//       TW = 16: mfma 16x16x16 bf16, B = P^T as the score lanes hold it;
//       TW = 32: mfma 16x16x32 bf16 with the token index ordered
//                {4q..4q+3, 16+4q..16+4q+3} for lane group q, so the two
//                score accumulators form B as they stand.
// Streams split a unit's work by KV head when the model's KV heads are a
// multiple of the stream count (each stream then owns whole heads), and by
// token slices otherwise (slice j goes to stream j mod NSTREAM, and the
// partial softmax states are merged through LDS at the end of the unit).
#pragma once

#include "decode_mfma.h"

namespace cp {

// G: query heads one unit handles (a model group of 8 is padded to 16; an
// MLA group of 32 runs as two units of 16, since 32 heads x 512 columns of
// accumulators would not leave registers for the rest).
template <int G, int DK, int DV, bool MLA, int TW, int NW, int SHARE, int NSLOT>
struct NarrowCfg {
  static constexpr int HBW = (G + 15) / 16;          // 16-head blocks
  static constexpr int HEADS = 16 * HBW;             // head columns, padded
  static constexpr int KROW = DK * 2;
  static constexpr int VROW = MLA ? KROW : DV * 2;
  static constexpr int KPITCH = lds_pitch(KROW);     // padded rows: conflict-free LDS reads
  static constexpr int VPITCH = MLA ? KPITCH : lds_pitch(VROW);
  static constexpr int SK = TW * KPITCH;
  static constexpr int SV = MLA ? 0 : TW * VPITCH;
  static constexpr int SLICE = SK + SV;              // LDS bytes of one slice
  static constexpr int NSTREAM = NW / SHARE;
  static constexpr int NLOADS = (SLICE + 1023) / 1024;          // 1 KiB direct loads per slice
  static constexpr int LOADS_M = (NLOADS + SHARE - 1) / SHARE;  // ... issued by one stream member
  static constexpr int NGRP = (LOADS_M + 3) / 4;                // M0 groups per member and slice
  static constexpr int RING = NSTREAM * NSLOT * SLICE;
  static constexpr int KSTEPS = DK / 32;
  static constexpr int NBLK = DV / 16;
  static constexpr int NBLKW = NBLK / SHARE;         // V column blocks one member accumulates
  static constexpr int NSL = TW / 16;                // 16-token sub-slices
  static constexpr int NACC = KSTEPS % 3 == 0 ? 3 : 2;  // independent score chains
  static constexpr bool AGPR_Q = HBW * KSTEPS * 4 >= 64;  // the query goes to accumulation registers
  static constexpr int VB = NBLKW >= 8 ? 8 : NBLKW;  // V^T fragments per prefetch batch
  static constexpr int OPITCH = DV + 8;              // merge area row pitch (floats; 2 mod 8 16-byte chunks)
  static constexpr int MERGE = HEADS * OPITCH * 4 + 2 * NSTREAM * HEADS * 4;
  static constexpr int LDS = RING > MERGE ? RING : MERGE;
  static_assert(G >= 8 && G <= 32, "8 to 32 heads per unit");
  static_assert(TW == 16 || TW == 32, "slices of 16 or 32 tokens");
  static_assert(SHARE == 1 || SHARE == 2, "one or two waves per stream");
  static_assert(NSLOT == 1 || NSLOT == 2, "one or two ring slots");
  static_assert(SHARE == 1 || NSLOT == 2, "shared streams prefetch");
  static_assert(KSTEPS % NACC == 0 && NBLK % SHARE == 0 && NBLKW % VB == 0, "blocking");
  static_assert(LDS <= 163840, "LDS budget");
};

template <int G, int DK, int DV, bool MLA, int TW, int NW, int SHARE, int NSLOT>
__device__ __forceinline__ void narrow_unit(const DecodeArgs &a, const GeomK &gm, const DecReq &rq, const Seg &sg,
                                            char *lds) {
  using C = NarrowCfg<G, DK, DV, MLA, TW, NW, SHARE, NSLOT>;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int stream = wave % C::NSTREAM, member = wave / C::NSTREAM;
  const int col = lane & 15, quad = lane >> 4;
  const int P = gm.page_tokens;  // the host routes only pages of a multiple of TW tokens here
  const int spp = P / TW;        // slices per page
  const uint32_t slot = sg.slot;
  // Work split: KV heads across streams, or token slices across streams. A
  // group wider than one unit (gm.nb blocks of C::HEADS heads) takes gm.nb
  // units per KV range.
  const bool head_par = gm.hkv % C::NSTREAM == 0;
  const int nsub = gm.nb;
  const int kvh = head_par ? C::NSTREAM * (int)sg.hblk + stream : (int)sg.hblk / nsub;
  const int sub = head_par ? 0 : (int)sg.hblk % nsub;
  const int h0 = kvh * gm.g + sub * C::HEADS;           // first query head of the unit
  const int hv = min(C::HEADS, gm.g - sub * C::HEADS);  // valid heads (fewer when padded)
  const int nb0 = member * C::NBLKW;                     // first V column block of this wave

  const uint32_t tok_begin = sg.pg_begin * (uint32_t)P;
  const uint32_t tok_end = min(rq.ctx_len, sg.pg_end * (uint32_t)P);
  const int nslices = (int)((tok_end - tok_begin + TW - 1) / TW);
  const int first = head_par ? 0 : stream;      // this stream's first slice
  const int step = head_par ? 1 : C::NSTREAM;   // ... and the stride between its slices
  const int mine = nslices > first ? (nslices - first + step - 1) / step : 0;
  // iterations of the loop: the same in every wave when streams share
  // barriers (then streams with fewer slices idle through the last ones)
  const int iters = SHARE == 1 ? mine : (head_par ? nslices : (nslices + C::NSTREAM - 1) / C::NSTREAM);
  const uint64_t kv_head_bytes = MLA ? 0 : (uint64_t)2 * P * DK * 2;
  char *const ring = lds + stream * (NSLOT * C::SLICE);
  const int npg = (int)((tok_end + P - 1) / P) - (int)sg.pg_begin;

  // Page-table entries of the unit, 64 at a time (lane i: page 64 b + i).
  uint32_t pte_lane = 0;
  int pte_batch = -1;
  auto load_ptes = [&](int batch) {
    const int sp = batch * 64 + lane;
    pte_lane = sp < npg ? a.pte[rq.pte_base + sg.pg_begin + (uint32_t)sp] : 0u;
    pte_batch = batch;
    // visible to the compiler, which cannot count the inline-asm slice
    // loads: otherwise it would drain them before every use of pte_lane
    __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
  };
  // This member's loads of a slice are [ld0, ld0 + nld); load j covers LDS
  // bytes [1024 j, 1024 j + 1024) of the slot. Per-lane source offsets are
  // biased for dma_group; pad lanes refetch the row's last 16 bytes; the
  // lanes of a partial last load past the slice are masked off.
  const int ld0 = member * C::LOADS_M;
  const int nld = min(C::LOADS_M, C::NLOADS - ld0);
  uint32_t voff[C::NGRP][4];
#pragma unroll
  for (int g = 0; g < C::NGRP; ++g)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int o = (ld0 + 4 * g + j) * 1024 + lane * 16;
      uint32_t gofs;
      if (C::SV == 0 || o < C::SK) {
        const int oc = o < C::SK ? o : 0;
        const int row = oc / C::KPITCH, w = oc - row * C::KPITCH;
        gofs = (uint32_t)(row * C::KROW + (w < C::KROW ? w : C::KROW - 16));
      } else {
        const int o2 = o < C::SLICE ? o - C::SK : 0;
        const int row = o2 / C::VPITCH, w = o2 - row * C::VPITCH;
        gofs = (uint32_t)(P * DK * 2 + row * C::VROW + (w < C::VROW ? w : C::VROW - 16));
      }
      voff[g][j] = gofs + kDmaBias - 1024u * j;
    }
  // Issues this member's loads of the stream's i-th slice into slot i % NSLOT.
  auto issue = [&](int i) {
    const int sl = first + step * i;  // slice within the unit
    const int sp = sl / spp;          // page within the unit
    if ((sp >> 6) != pte_batch) load_ptes(sp >> 6);
    const uint32_t pte = __builtin_amdgcn_readlane(pte_lane, sp & 63);
    const uint64_t sb = uniform_ptr(a.pool + ((uint64_t)pte << 8) + (uint64_t)kvh * kv_head_bytes +
                                    (uint64_t)(sl % spp) * TW * C::KROW - kDmaBias);
    const uint32_t lb = lds_addr(ring + (i % NSLOT) * C::SLICE) + 1024 * ld0;
#pragma unroll
    for (int g = 0; g < C::NGRP; ++g) {
      const int n = min(4, nld - 4 * g);
      // a partial last load of the slice goes alone, lanes past it masked
      const bool tail = C::SLICE % 1024 != 0 && ld0 + 4 * g + n == C::NLOADS;
      const int nf = n - (tail ? 1 : 0);
      if (nf == 4) dma_group<4>(sb, voff[g], lb + 4096 * g);
      else if (nf == 3) dma_group<3>(sb, voff[g], lb + 4096 * g);
      else if (nf == 2) dma_group<2>(sb, voff[g], lb + 4096 * g);
      else if (nf == 1) dma_group<1>(sb, voff[g], lb + 4096 * g);
      if (tail && (C::NLOADS - 1) * 1024 + lane * 16 < C::SLICE) {
        const uint32_t t[4] = {voff[g][nf] + 1024u * nf, 0u, 0u, 0u};
        dma_group<1>(sb, t, lb + 4096 * g + 1024 * nf);
      }
    }
  };

  float m[C::HBW], lsum[C::HBW];
  f32x4 o[C::HBW][C::NBLKW];
#pragma unroll
  for (int hb = 0; hb < C::HBW; ++hb) {
    m[hb] = -INFINITY;
    lsum[hb] = 0.f;
#pragma unroll
    for (int nb = 0; nb < C::NBLKW; ++nb) o[hb][nb] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  const float sl2 = gm.scale_log2;
  const int vrow = 4 * quad + (col >> 2);  // V row this lane supplies to a transpose read
  const int vcol = 8 * (col & 3) + 32 * nb0;

  // Unit start. The query is staged through LDS: its Q^T operand fragments
  // (lane holds head h0 + 16 hb + col, dims 32 c + 8 quad .. +7) are copied
  // by direct loads into a second ring slot in fragment order (fragment
  // f = hb KSTEPS + c at byte 1024 f + 16 lane). When the streams share the
  // unit's heads, one copy in stream 0's slot serves the workgroup and
  // every wave copies every NW-th fragment; when each stream owns a KV head
  // (and so its own h0), each stream copies its query into its own slot.
  // Those loads read 16 rows of 64 bytes each, which the address unit
  // serves a row at a time, so one copy per workgroup (or stream) instead
  // of one per wave keeps them from delaying the first slice. The
  // page-table wait of the first slice's issue covers the copy; the slot is
  // free until the loop's first barrier, by which point every wave has read
  // its fragments.
  constexpr int NQF = C::HBW * C::KSTEPS;
  static_assert(NQF * 1024 <= C::SLICE, "the query fits one ring slot");
  static_assert(NSLOT == 2, "the query is staged in the second ring slot");
  char *const qstage = (head_par ? ring : lds) + C::SLICE;
  {
    const int qw = head_par ? member : wave, nqw = head_par ? SHARE : NW;  // this copier, copiers
    const uint64_t qb = uniform_ptr(a.q + rq.q_off + (uint32_t)h0 * DK) - kDmaBias;
    for (int f = qw; f < NQF; f += nqw) {
      const int hb = f / C::KSTEPS, c = f - hb * C::KSTEPS, hh = 16 * hb + col;
      const uint32_t o[4] = {(uint32_t)((hh < hv ? hh : 0) * DK + 32 * c + 8 * quad) * 2 + kDmaBias, 0u, 0u, 0u};
      dma_group<1>(qb, o, lds_addr(qstage + 1024 * f));
    }
  }
  if (mine > 0) issue(0);
  else wait_vm<0>();
  __syncthreads();  // the query copy is visible to every wave
  bf16x8 qf[C::HBW][C::KSTEPS];
#pragma unroll
  for (int hb = 0; hb < C::HBW; ++hb)
#pragma unroll
    for (int c = 0; c < C::KSTEPS; ++c)
      qf[hb][c] = *reinterpret_cast<const bf16x8 *>(qstage + 1024 * (hb * C::KSTEPS + c) + 16 * lane);
#pragma unroll
  for (int hb = 0; hb < C::HBW; ++hb)
#pragma unroll
    for (int c = 0; c < C::KSTEPS; ++c) {
      if (16 * hb + col >= hv) qf[hb][c] = bf16x8{};
      // a long query lives in the accumulation registers, which the matrix
      // cores read directly as the B operand; that leaves the architectural
      // registers to the accumulators and to fragment prefetch. Either way
      // the reads complete here, before the slot is refilled.
      if constexpr (C::AGPR_Q) asm volatile("" : "+a"(qf[hb][c]));
      else asm volatile("" : "+v"(qf[hb][c]));
    }

#pragma unroll 1
  for (int i = 0; i < iters; ++i) {
    const bool active = i < mine;
    if constexpr (NSLOT == 1) {
      if (active) issue(i);
      wait_vm<0>();
    } else if constexpr (SHARE == 1) {
      // slice i+1 goes to the slot of slice i-1, whose reads this wave has
      // finished, before waiting for slice i
      if (i + 1 < mine) {
        issue(i + 1);
        wait_vm<C::NLOADS>();
      } else {
        wait_vm<0>();
      }
    } else {
      wait_vm<0>();
      __syncthreads();  // both members' loads of slice i landed; slot of slice i-1 free
      if (i + 1 < mine) issue(i + 1);
    }
    if (!active) continue;
    char *kt = ring + (i % NSLOT) * C::SLICE;
    char *vt = MLA ? kt : kt + C::SK;
    const int s = first + step * i;
    const int valid = min(TW, (int)(tok_end - tok_begin) - s * TW);
    if (valid < TW) {
      // rows past the context may hold stale bytes: their scores are masked
      // to -inf, and this wave's V columns of them are zeroed so that
      // 0 * V stays 0 (each member zeroes only the columns it reads)
      constexpr int CH = C::NBLKW * 2;  // 16-byte chunks of this member's columns per row
      for (int z = lane; z < (TW - valid) * CH; z += 64) {
        const int row = valid + z / CH, pc = z % CH;
        *reinterpret_cast<uint4 *>(vt + row * C::VPITCH + 32 * nb0 + pc * 16) = make_uint4(0, 0, 0, 0);
      }
    }

    // ---- scores: C::NSL sub-slices x C::HBW head blocks
    f32x4 sv[C::NSL][C::HBW];
#pragma unroll
    for (int u = 0; u < C::NSL; ++u) {
      f32x4 acc[C::NACC][C::HBW];
#pragma unroll
      for (int j = 0; j < C::NACC; ++j)
#pragma unroll
        for (int hb = 0; hb < C::HBW; ++hb) acc[j][hb] = f32x4{0.f, 0.f, 0.f, 0.f};
      const char *kr = kt + (16 * u + col) * C::KPITCH + quad * 16;
      // K fragments in batches of six, read ahead of their products (the
      // scheduler would otherwise wait a full LDS latency per k-step)
      constexpr int KB = C::KSTEPS % 6 == 0 ? 6 : C::KSTEPS;
#pragma unroll
      for (int b = 0; b < C::KSTEPS / KB; ++b) {
        bf16x8 kf[KB];
#pragma unroll
        for (int c = 0; c < KB; ++c) kf[c] = *reinterpret_cast<const bf16x8 *>(kr + 64 * (b * KB + c));
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int c = 0; c < KB; ++c)
#pragma unroll
          for (int hb = 0; hb < C::HBW; ++hb) {
            const int cc = b * KB + c;
            acc[cc % C::NACC][hb] =
                __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[c], qf[hb][cc], acc[cc % C::NACC][hb], 0, 0, 0);
          }
      }
#pragma unroll
      for (int hb = 0; hb < C::HBW; ++hb) {
        f32x4 t = acc[0][hb];
#pragma unroll
        for (int j = 1; j < C::NACC; ++j) t += acc[j][hb];
        sv[u][hb] = t;
      }
    }
    // ---- online softmax (lane owns head column col; rows 16 u + 4 quad + r)
    // (scores stay unscaled: the positive scale goes onto the column maximum
    // and into the exponent's fma)
    if (valid < TW) {
#pragma unroll
      for (int u = 0; u < C::NSL; ++u)
#pragma unroll
        for (int hb = 0; hb < C::HBW; ++hb)
#pragma unroll
          for (int r = 0; r < 4; ++r)
            if (16 * u + 4 * quad + r >= valid) sv[u][hb][r] = -INFINITY;
    }
    bool bump = false;
    float mt[C::HBW];
#pragma unroll
    for (int hb = 0; hb < C::HBW; ++hb) {
      float x = sv[0][hb][0];
#pragma unroll
      for (int u = 0; u < C::NSL; ++u)
#pragma unroll
        for (int r = 0; r < 4; ++r) x = x > sv[u][hb][r] ? x : sv[u][hb][r];
      x = xor_max_16_32(x) * sl2;
      mt[hb] = x;
      bump = bump || x > m[hb] + kLazy;
    }
    if (__builtin_amdgcn_ballot_w64(bump)) {
#pragma unroll
      for (int hb = 0; hb < C::HBW; ++hb) {
        const float mn = mt[hb] > m[hb] + kLazy ? mt[hb] : m[hb];
        const float al = fast_exp2(m[hb] - mn);
        m[hb] = mn;
        lsum[hb] *= al;
#pragma unroll
        for (int nb = 0; nb < C::NBLKW; ++nb) o[hb][nb] *= al;
      }
    }
    // ---- P (fp32 into the row sums, bf16 as the P.V operand) and O^T += V^T P^T
    if constexpr (TW == 16) {
      s16x4 pf[C::HBW];
#pragma unroll
      for (int hb = 0; hb < C::HBW; ++hb) {
        float ps = 0.f;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float p = fast_exp2(__builtin_fmaf(sv[0][hb][r], sl2, -m[hb]));
          ps += p;
          pf[hb][r] = __builtin_bit_cast(short, (__bf16)p);
        }
        lsum[hb] += ps;
      }
      const char *vr = vt + vrow * C::VPITCH + vcol;
      // V^T fragments in batches of VB, the next batch read while this one
      // feeds the matrix cores
      constexpr int NVB = C::NBLKW / C::VB;
      s16x4 vf[2][C::VB];
#pragma unroll
      for (int j = 0; j < C::VB; ++j)
        vf[0][j] = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4 *)(vr + 32 * j));
#pragma unroll
      for (int b = 0; b < NVB; ++b) {
        if (b + 1 < NVB) {
#pragma unroll
          for (int j = 0; j < C::VB; ++j)
            vf[(b + 1) & 1][j] = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                (__attribute__((address_space(3))) s16x4 *)(vr + 32 * ((b + 1) * C::VB + j)));
        }
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int j = 0; j < C::VB; ++j)
#pragma unroll
          for (int hb = 0; hb < C::HBW; ++hb)
            o[hb][b * C::VB + j] =
                __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(vf[b & 1][j], pf[hb], o[hb][b * C::VB + j], 0, 0, 0);
        __builtin_amdgcn_sched_barrier(0);
      }
    } else {
      bf16x8 pf[C::HBW];
#pragma unroll
      for (int hb = 0; hb < C::HBW; ++hb) {
        float ps = 0.f;
#pragma unroll
        for (int u = 0; u < 2; ++u)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const float p = fast_exp2(__builtin_fmaf(sv[u][hb][r], sl2, -m[hb]));
            ps += p;
            pf[hb][4 * u + r] = (__bf16)p;
          }
        lsum[hb] += ps;
      }
      const char *vr0 = vt + vrow * C::VPITCH + vcol;
      const char *vr1 = vr0 + 16 * C::VPITCH;
      bf16x8 vf[C::NBLKW];
#pragma unroll
      for (int nb = 0; nb < C::NBLKW; ++nb) {
        const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4 *)(vr0 + 32 * nb));
        const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4 *)(vr1 + 32 * nb));
        vf[nb] = __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
      }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int nb = 0; nb < C::NBLKW; ++nb)
#pragma unroll
        for (int hb = 0; hb < C::HBW; ++hb)
          o[hb][nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf[nb], pf[hb], o[hb][nb], 0, 0, 0);
    }
  }

  // ---- unit end
#pragma unroll
  for (int hb = 0; hb < C::HBW; ++hb) {
    lsum[hb] = xor_sum_16_32(lsum[hb]);
  }
  const bool split = rq.ws_base != kNoWs;
  auto write_out = [&](int hh, int d, const f32x4 &v) {  // hh: head within the unit
    const uint32_t head = (uint32_t)(h0 + hh);
    uint16_t *dst = split ? a.ws_o + ((uint64_t)rq.ws_orow + (uint64_t)slot * gm.hq + head) * DV + d
                          : a.out + rq.o_off + head * DV + d;
    *reinterpret_cast<uint2 *>(dst) = bf16x4_bits(v[0], v[1], v[2], v[3]);
  };
  auto write_lse = [&](int hh, float lse) {
    const uint32_t head = (uint32_t)(h0 + hh);
    if (split)
      a.ws_l[(uint64_t)rq.ws_base + (uint64_t)slot * gm.hq + head] = lse;
    else
      a.lse[rq.lse_off + head] = lse;
  };
  if (head_par) {
    // this stream owns whole heads; each member writes its V columns
#pragma unroll
    for (int hb = 0; hb < C::HBW; ++hb) {
      const int hh = 16 * hb + col;
      if (hh < hv) {
        const float inv = 1.0f / lsum[hb];
#pragma unroll
        for (int nb = 0; nb < C::NBLKW; ++nb) write_out(hh, 16 * (nb0 + nb) + 4 * quad, o[hb][nb] * inv);
        if (member == 0 && quad == 0) write_lse(hh, (m[hb] + fast_log2(lsum[hb])) * kLn2);
      }
    }
    __syncthreads();  // keep the waves together for the next unit
    return;
  }
  // token slices were split over the streams: merge their softmax states.
  // Every stream writes its rescaled partial output to a region of its own
  // (or, when those do not fit, the streams add into one region in turn).
  constexpr bool PAR = C::NSTREAM * C::HEADS * C::OPITCH * 4 + 2 * C::NSTREAM * C::HEADS * 4 <= C::LDS;
  constexpr int NREG = PAR ? C::NSTREAM : 1;
  float *const macc = reinterpret_cast<float *>(lds);            // [NREG][HEADS][OPITCH]
  float *const m_x = macc + NREG * C::HEADS * C::OPITCH;         // [NSTREAM][HEADS]
  float *const l_x = m_x + C::NSTREAM * C::HEADS;                // [NSTREAM][HEADS]
  __syncthreads();  // every stream is done with its ring
  if (member == 0 && quad == 0) {
#pragma unroll
    for (int hb = 0; hb < C::HBW; ++hb) {
      m_x[stream * C::HEADS + 16 * hb + col] = m[hb];
      l_x[stream * C::HEADS + 16 * hb + col] = lsum[hb];
    }
  }
  __syncthreads();
  float f[C::HBW];
#pragma unroll
  for (int hb = 0; hb < C::HBW; ++hb) {
    const int hh = 16 * hb + col;
    float M = -INFINITY;
#pragma unroll
    for (int s2 = 0; s2 < C::NSTREAM; ++s2) M = fmaxf(M, m_x[s2 * C::HEADS + hh]);
    // a stream without slices has m = -inf and contributes nothing
    f[hb] = m[hb] == -INFINITY ? 0.f : fast_exp2(m[hb] - M);
  }
  auto put = [&](float *region, bool add) {
#pragma unroll
    for (int hb = 0; hb < C::HBW; ++hb)
#pragma unroll
      for (int nb = 0; nb < C::NBLKW; ++nb) {
        f32x4 *dst = reinterpret_cast<f32x4 *>(region + (16 * hb + col) * C::OPITCH + 16 * (nb0 + nb) + 4 * quad);
        const f32x4 v = o[hb][nb] * f[hb];
        *dst = add ? *dst + v : v;
      }
  };
  if constexpr (PAR) {
    put(macc + stream * C::HEADS * C::OPITCH, false);
    __syncthreads();
  } else {
    for (int s2 = 0; s2 < C::NSTREAM; ++s2) {
      if (stream == s2) put(macc, s2 > 0);
      __syncthreads();
    }
  }
  // normalise and write: thread t takes head t / TPH and the 16-byte column
  // chunks t % TPH + TPH j (conflict-free LDS reads, coalesced stores); the
  // head's merged m and l are formed once
  {
    constexpr int TPH = 64 * NW / C::HEADS;  // threads per head
    constexpr int NCH = DV / 4 / TPH;        // 16-byte chunks per thread
    static_assert(NCH >= 1 && (DV / 4) % TPH == 0, "whole chunks per thread");
    const int hh = threadIdx.x / TPH, ci = threadIdx.x % TPH;
    float M = -INFINITY, L = 0.f;
#pragma unroll
    for (int s2 = 0; s2 < C::NSTREAM; ++s2) M = fmaxf(M, m_x[s2 * C::HEADS + hh]);
#pragma unroll
    for (int s2 = 0; s2 < C::NSTREAM; ++s2) {
      const float ms = m_x[s2 * C::HEADS + hh];
      L += ms == -INFINITY ? 0.f : l_x[s2 * C::HEADS + hh] * fast_exp2(ms - M);
    }
    const float inv = 1.0f / L;
#pragma unroll 1
    for (int j = 0; j < NCH; ++j) {
      const int d = 4 * (ci + TPH * j);
      f32x4 v = *reinterpret_cast<const f32x4 *>(macc + hh * C::OPITCH + d);
#pragma unroll
      for (int r = 1; r < NREG; ++r) v += *reinterpret_cast<const f32x4 *>(macc + (r * C::HEADS + hh) * C::OPITCH + d);
      if (hh < hv) write_out(hh, d, v * inv);
    }
    if (hh < hv && ci == 0) write_lse(hh, (M + fast_log2(L)) * kLn2);
  }
  __syncthreads();  // LDS is reused by the next unit
}

}  // namespace cp
