// Matrix-core decode path for DeepSeek-V3-shaped MLA (section 2.2's latent
// attention): 128 query heads read one latent KV head whose 576-element rows
// hold the 512-element value part first and the 64-element rotary part last.
// Per token that is about 240 flop per KV byte, so streaming KV at HBM speed
// needs the matrix cores busy most of the time; the kernel is built around
// keeping them fed.
//
// Eight waves (two per SIMD) share the tile stream; tiles are T = 32 tokens.
//   scores  wave w owns query heads [16 w, 16 w + 16): S^T[t][h] =
//           sum_d K[t][d] Q[h][d] with mfma 16x16x32 bf16 (K rows from LDS as
//           the A operand, the wave's query fragments in registers as B),
//           then the fp32 online softmax with a lazily moved reference, and
//           P^T published to LDS as bf16 operand fragments;
//   P.V     wave w owns value columns [64 w, 64 w + 64) for all 128 heads:
//           O^T[d][h] += sum_t V^T[d][t] P^T[t][h]. The token index of that
//           product runs {4q..4q+3, 16+4q..16+4q+3} for lane group q, which
//           is how the score accumulators hold P, and V^T comes from LDS
//           transpose reads.
// Software pipeline: iteration k computes the scores and softmax of tile k
// and the P.V product of tile k-1, with one workgroup barrier per tile.
// P^T and the rescale factors are double-buffered by tile parity, so a wave
// may publish tile k's while another still multiplies tile k-1's, and the two
// waves of a SIMD drift apart within the iteration: one's softmax and LDS
// waits are the other's matrix-core issue slots. (Fixed opposite orders for
// the two waves, and wave priorities, measured no better.)
//
// LDS (160 KiB): a ring of four value tiles (32 rows of 1024 bytes), a ring
// of three rotary tiles (32 rows of 128 bytes: the rotary part is only read
// by the scores of its own tile, one iteration less than the value part),
// two P^T buffers of 8 KiB and two rescale records. Rows carry no padding:
// 16-byte chunk g of row r is stored at chunk g ^ (2r mod 16) in a value
// row and at g ^ (r & 6) in a rotary row, which keeps the K operand reads
// (16 rows x 16 bytes per lane group) and the V transpose reads free of
// bank conflicts. The direct HBM -> LDS loads apply the permutation through
// their per-lane source addresses, so every load writes one contiguous
// KiB (a rotary load: half a KiB) of LDS.
//
// Registers are the binding limit (the P.V accumulators and the query
// fragments take 200 of a wave's 256), so per-lane constants are formed
// where they are used, from the lane index counted afresh each iteration:
// the compiler can neither hoist them out of the loop nor keep them in
// scratch memory, whose reloads would make it wait for every load in
// flight, tile loads included.
#pragma once

#include "decode_mfma.h"

namespace cp {

struct MlaCfg {
  static constexpr int G = 128, DK = 576, DV = 512, NW = 8, T = 32;
  static constexpr int KROW = DK * 2;          // bytes of one KV row in HBM
  static constexpr int MROW = DV * 2;          // value part: one value-ring row
  static constexpr int RROW = KROW - MROW;     // rotary part: one rotary-ring row
  static constexpr int MSLOT = T * MROW;       // 32 KiB
  static constexpr int RSLOT = T * RROW;       // 4 KiB
  static constexpr int NM = 4, NR = 3;         // ring depths
  static constexpr int HB = G / 16;            // head blocks
  static constexpr int DBW = DV / (16 * NW);   // value column blocks per wave
  static constexpr int KSTEPS = DK / 32;       // score k-steps
  static constexpr int KMAIN = DV / 32;        // ... of them in the value part
  static constexpr int PBYTES = HB * 64 * 16;  // P^T fragments of one tile
  static constexpr int XFLAGS = 16;             // rescale record: one flag byte per score wave,
  static constexpr int XBYTES = XFLAGS + 4 * G;  // then alpha[G]
  static constexpr int OFF_R = NM * MSLOT;
  static constexpr int OFF_P = OFF_R + NR * RSLOT;
  static constexpr int OFF_X = OFF_P + 2 * PBYTES;
  static constexpr int LDS = OFF_X + 2 * XBYTES;
  static_assert(MROW == 1024 && RROW == 128, "one direct load per value row, eight rotary rows per load");
  static_assert(NW * 4 == T, "each of the first NW / 2 waves loads eight value rows and eight rotary rows");
  static_assert(HB == NW && DBW == 4, "one score head block and four value column blocks per wave");
  static_assert(LDS + 16 <= 163840, "LDS budget");
};

// Swizzles: position of 16-byte chunk g of row r.
CP_DEV int mla_vswz(int r) { return (2 * r) & 15; }
CP_DEV int mla_rswz(int r) { return r & 6; }

// Lane index and its mfma coordinates, counted afresh by the lane-count
// instructions at every use: the compiler can neither hoist them nor keep
// the thread index alive across the loop for them.
struct LaneIds {
  int lane, col, quad;
};
CP_DEV LaneIds lane_ids() {
  int t;
  asm volatile("v_mbcnt_lo_u32_b32 %0, -1, 0\n\tv_mbcnt_hi_u32_b32 %0, -1, %0" : "=v"(t));
  return LaneIds{t, t & 15, t >> 4};
}

__device__ __forceinline__ void mla_unit(const DecodeArgs &a, const GeomK &gm, const DecReq &rq, const Seg &sg,
                                         char *lds) {
  using C = MlaCfg;
  constexpr int NW = C::NW, T = C::T;
  const uint32_t slot = sg.slot;
  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const LaneIds L0 = lane_ids();
  const int col = L0.col, quad = L0.quad;
  const int P = gm.page_tokens;  // the host routes only pages of a multiple of 32 tokens here
  const int tpp = P / T;
  const int h0 = (int)sg.hblk * C::G;  // first query head of the (single) KV head

  char *const vring = lds;
  char *const rring = lds + C::OFF_R;
  char *const pbuf = lds + C::OFF_P;
  char *const xbuf = lds + C::OFF_X;

  const uint32_t tok_end = min(rq.ctx_len, sg.pg_end * (uint32_t)P);
  const uint32_t pg_begin = sg.pg_begin;
  const int npg = (int)((tok_end + P - 1) / P) - (int)pg_begin;
  const int last_tok = npg > 0 ? (int)tok_end - (int)((pg_begin + (uint32_t)npg - 1) * (uint32_t)P) : 0;
  const int ntiles = npg > 0 ? (npg - 1) * tpp + (last_tok + T - 1) / T : 0;

  // Page-table entries of the segment, 64 at a time (lane i: page 64 b + i).
  uint32_t pte_lane = 0;
  int pte_batch = -1;
  auto load_ptes = [&](int batch) {
    const int sp = batch * 64 + lane_ids().lane;
    pte_lane = sp < npg ? a.pte[rq.pte_base + pg_begin + (uint32_t)sp] : 0u;
    pte_batch = batch;
    // a visible wait: the tile loads are inline asm the compiler cannot
    // count, so its own wait at the first use would drain them every tile
    __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
  };
  // Source base of tile k, lowered by kDmaBias.
  auto tile_src = [&](int k) -> uint64_t {
    const int sp = k / tpp;
    if ((sp >> 6) != pte_batch) load_ptes(sp >> 6);
    const uint32_t pte = __builtin_amdgcn_readlane(pte_lane, sp & 63);
    return uniform_ptr(a.pool + ((uint64_t)pte << 8) + (uint64_t)(k % tpp) * T * C::KROW - kDmaBias);
  };

  // Direct loads, all issued by the first half of the waves, which wait at
  // the barrier for the second half anyway: wave w < 4 loads value rows
  // 8w .. 8w+7 (two groups of four loads, one M0 write each) and rotary
  // rows 8w .. 8w+7 (one load). Per-lane source offsets (within the tile)
  // place chunk (lane ^ swizzle) of the row at LDS chunk `lane`.
  const bool loader = wave < NW / 2;
  auto issue_value = [&](const LaneIds &L, int k, uint64_t sb, int g) {
    const uint32_t lb =
        __builtin_amdgcn_readfirstlane(lds_addr(vring + (k % C::NM) * C::MSLOT) + wave * 8192 + g * 4096);
    uint32_t vo[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int r = 8 * wave + 4 * g + j;
      vo[j] = (uint32_t)(r * C::KROW + 16 * (L.lane ^ mla_vswz(r))) + kDmaBias - 1024u * j;
    }
    dma_group<4>(sb, vo, lb);
  };
  auto issue_rope = [&](const LaneIds &L, int k, uint64_t sb) {
    const uint32_t lb = __builtin_amdgcn_readfirstlane(lds_addr(rring + (k % C::NR) * C::RSLOT) + wave * 1024);
    const int r = 8 * wave + (L.lane >> 3);
    const uint32_t vo[4] = {(uint32_t)(r * C::KROW + C::MROW + 16 * ((L.lane & 7) ^ mla_rswz(r))) + kDmaBias, 0u, 0u,
                            0u};
    dma_group<1>(sb, vo, lb);
  };
  auto issue_tile = [&](const LaneIds &L, int k, uint64_t sb) {
    issue_value(L, k, sb, 0);
    issue_value(L, k, sb, 1);
    issue_rope(L, k, sb);
  };

  // K operand read addresses of tile k (slice 0; slice 1 is 16 rows
  // further): value k-step 4a + b of row col sits at kva[b] + 256 a, kept
  // for the tile's value slot and moved on by one slot per tile; rotary
  // k-step c of row col at kra ^ (64 c), formed per tile.
  uint32_t kva[4];
  {
    const int s = mla_vswz(col);
#pragma unroll
    for (int b = 0; b < 4; ++b)
      kva[b] = lds_addr(vring) + (uint32_t)(col * C::MROW + 64 * (b ^ (s >> 2)) + 16 * (quad ^ (s & 3)));
  }
  static_assert((C::MSLOT & (C::MSLOT - 1)) == 0 && C::NM == 4, "value slots rotate by masking");

  float m = -INFINITY, lsum = 0.f;
  f32x4 o[C::DBW][C::HB];
#pragma unroll
  for (int db = 0; db < C::DBW; ++db)
#pragma unroll
    for (int hb = 0; hb < C::HB; ++hb) o[db][hb] = f32x4{0.f, 0.f, 0.f, 0.f};
  const float sl2 = gm.scale_log2;

  if (ntiles > 0) load_ptes(0);
  if (loader) {
    for (int k = 0; k < 2 && k < ntiles; ++k) issue_tile(L0, k, tile_src(k));
  }

  // Q^T operand fragments of this wave's heads: lane holds head
  // (h0 + 16 wave + col), dims 32 c + 8 quad .. +7.
  bf16x8 qf[C::KSTEPS];
  {
    const uint16_t *qrow = a.q + rq.q_off + (uint32_t)(h0 + 16 * wave + col) * C::DK + 8 * quad;
#pragma unroll
    for (int c = 0; c < C::KSTEPS; ++c) qf[c] = *reinterpret_cast<const bf16x8 *>(qrow + 32 * c);
  }

  // P.V of tile kp: pv_load issues the LDS reads of its rescale flags, the
  // wave's V^T fragments and the first P^T fragments; pv_mma applies the
  // rescale its score waves asked for and runs the products, reading each
  // later P^T fragment two head blocks ahead.
  struct PvRegs {
    uint64_t fl;  // flag bytes of the score waves (the same in every lane)
    bf16x8 vf[C::DBW];
    bf16x8 pf[2];
  };
  auto pv_load = [&](const LaneIds &L, int kp, PvRegs &r) {
    const int lane = L.lane, col = L.col, quad = L.quad;
    r.fl = *reinterpret_cast<const uint64_t *>(xbuf + (kp & 1) * C::XBYTES);
    // this lane supplies value row vr (and vr + 16), bytes 8 (col & 3) of
    // each column block of the wave's columns
    const int vr = 4 * quad + (col >> 2);
    const int vsw = mla_vswz(vr), vch = 8 * wave + ((col >> 1) & 1);
    const char *vt = vring + (kp % C::NM) * C::MSLOT + vr * C::MROW + 8 * (col & 1);
#pragma unroll
    for (int db = 0; db < C::DBW; ++db) {
      const char *p0 = vt + 16 * ((vch + 2 * db) ^ vsw);
      const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4 *)p0);
      const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
          (__attribute__((address_space(3))) s16x4 *)(p0 + 16 * C::MROW));
      r.vf[db] = __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
    }
    const char *pt = pbuf + (kp & 1) * C::PBYTES + lane * 16;
    r.pf[0] = *reinterpret_cast<const bf16x8 *>(pt);
    r.pf[1] = *reinterpret_cast<const bf16x8 *>(pt + 1024);
  };
  auto pv_mma = [&](const LaneIds &L, int kp, PvRegs &r) {
    const int lane = L.lane, col = L.col;
    const uint64_t fl = ((uint64_t)__builtin_amdgcn_readfirstlane((uint32_t)(r.fl >> 32)) << 32) |
                        __builtin_amdgcn_readfirstlane((uint32_t)r.fl);
    if (fl != 0) {
      const float *alpha = reinterpret_cast<const float *>(xbuf + (kp & 1) * C::XBYTES + C::XFLAGS);
#pragma unroll
      for (int hb = 0; hb < C::HB; ++hb) {
        if ((fl >> (8 * hb)) & 0xFF) {
          const float al = alpha[16 * hb + col];
#pragma unroll
          for (int db = 0; db < C::DBW; ++db) o[db][hb] *= al;
        }
      }
    }
    const char *pt = pbuf + (kp & 1) * C::PBYTES + lane * 16;
    bf16x8 pn = r.pf[0];
#pragma unroll
    for (int hb = 0; hb < C::HB; ++hb) {
      const bf16x8 pf = pn;
      pn = r.pf[(hb + 1) & 1];
      if (hb + 2 < C::HB) r.pf[hb & 1] = *reinterpret_cast<const bf16x8 *>(pt + (hb + 2) * 1024);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int db = 0; db < C::DBW; ++db)
        o[db][hb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(r.vf[db], pf, o[db][hb], 0, 0, 0);
    }
  };

  // Every load so far (query, page table) is complete before the tile loop,
  // as far as the compiler can see: it then places no wait of its own inside
  // the loop, where one would also drain the tile loads in flight.
  __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);

#pragma unroll 1
  for (int k = 0; k <= ntiles && ntiles > 0; ++k) {
    // own loads of tile k have landed once at most tile k+1's remain
    if (loader) {
      if (k + 1 < ntiles)
        wait_vm<9>();
      else if (k < ntiles)
        wait_vm<0>();
    }
    // tile k visible; P^T and rescale record of tile k-1 complete; the value
    // slot of tile k-2 and the rotary slot of tile k-1 are free
    __syncthreads();
    const LaneIds L = lane_ids();
    const int lane = L.lane, col = L.col, quad = L.quad;
    const int kn = k + 2;
    const bool more = loader && kn < ntiles;
    const uint64_t sbn = more ? tile_src(kn) : 0;
    if (more) issue_value(L, kn, sbn, 0);

    if (k < ntiles) {
      char *vt = vring + (k % C::NM) * C::MSLOT;
      const int t0 = (int)((pg_begin + (uint32_t)(k / tpp)) * P) + (k % tpp) * T;
      const int valid = min(T, (int)tok_end - t0);
      if (valid < T) {
        // value rows past the context may hold stale bytes: zero them so
        // that 0 * V stays 0 in the next iteration's P.V (their scores are
        // masked to -inf below)
        const int nz = (T - valid) * (C::MROW / 16);
        uint32_t z;  // a zero formed here, not a zero vector kept through the loop
        asm volatile("v_mov_b32 %0, 0" : "=v"(z));
        for (int i = wave * 64 + lane; i < nz; i += 64 * NW)
          *reinterpret_cast<uint4 *>(vt + valid * C::MROW + i * 16) = make_uint4(z, z, z, z);
      }

      // ---- scores of this wave's 16 heads, one 16-token slice after the other
      const uint32_t kra = lds_addr(rring + (k % C::NR) * C::RSLOT) +
                           (uint32_t)(col * C::RROW + 64 * (mla_rswz(col) >> 2) + 16 * (quad ^ (mla_rswz(col) & 3)));
      f32x4 s[2] = {f32x4{0.f, 0.f, 0.f, 0.f}, f32x4{0.f, 0.f, 0.f, 0.f}};
      auto kread = [&](int c, int sl) -> bf16x8 {
        const uint32_t ad = c < C::KMAIN ? kva[c & 3] + 256 * (c >> 2) + sl * 16 * C::MROW
                                         : (kra ^ (64 * (c - C::KMAIN))) + sl * 16 * C::RROW;
        return *reinterpret_cast<const bf16x8 *>(lds + (ad - lds_addr(lds)));
      };
      // K fragments are read KD products ahead; the scheduling barriers keep
      // the compiler from sinking the reads back to their uses
      constexpr int KD = 4;
#pragma unroll
      for (int sl = 0; sl < 2; ++sl) {
        bf16x8 kf[KD + 1];
#pragma unroll
        for (int c = 0; c < KD; ++c) kf[c] = kread(c, sl);
#pragma unroll
        for (int c = 0; c < C::KSTEPS; ++c) {
          if (c + KD < C::KSTEPS) kf[(c + KD) % (KD + 1)] = kread(c + KD, sl);
          if (sl == 0 && c == 6 && more) issue_value(L, kn, sbn, 1);
          if (sl == 1 && c == 0 && more) issue_rope(L, kn, sbn);
          __builtin_amdgcn_sched_barrier(0);
          s[sl] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[c % (KD + 1)], qf[c], s[sl], 0, 0, 0);
        }
      }
      // ---- online softmax (lane: head col, tokens 16 sl + 4 quad + r).
      // Scores stay unscaled; the (positive) scale is applied to the
      // maximum and folded into the exponent's fma.
      if (valid < T) {
#pragma unroll
        for (int sl = 0; sl < 2; ++sl)
#pragma unroll
          for (int r = 0; r < 4; ++r)
            if (16 * sl + 4 * quad + r >= valid) s[sl][r] = -INFINITY;
      }
      float x = s[0][0];
#pragma unroll
      for (int sl = 0; sl < 2; ++sl)
#pragma unroll
        for (int r = 0; r < 4; ++r) x = __builtin_fmaxf(x, s[sl][r]);
      const float mt = xor_max_16_32(x) * sl2;
      const bool bump = mt > m + kLazy;
      const bool any_bump = __builtin_amdgcn_ballot_w64(bump) != 0;
      char *xw = xbuf + (k & 1) * C::XBYTES;
      if (any_bump) {
        const float mn = bump ? mt : m;
        const float al = fast_exp2(m - mn);
        m = mn;
        lsum *= al;
        if (quad == 0) reinterpret_cast<float *>(xw + C::XFLAGS)[16 * wave + col] = al;
      }
      if (lane == 0) reinterpret_cast<uint8_t *>(xw)[wave] = any_bump ? 1 : 0;
      bf16x8 pk;
      float ps = 0.f;
#pragma unroll
      for (int sl = 0; sl < 2; ++sl)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          // the row sum takes p in fp32; only the P.V operand is rounded to bf16
          const float p = fast_exp2(__builtin_fmaf(s[sl][r], sl2, -m));
          ps += p;
          pk[4 * sl + r] = (__bf16)p;
        }
      lsum += ps;
      *reinterpret_cast<bf16x8 *>(pbuf + (k & 1) * C::PBYTES + (wave * 64 + lane) * 16) = pk;
      // the next tile's slots
      const uint32_t vbase = lds_addr(vring);
#pragma unroll
      for (int b = 0; b < 4; ++b) kva[b] = vbase + ((kva[b] - vbase + C::MSLOT) & (C::NM * C::MSLOT - 1));
    }

    if (k >= 1) {
      PvRegs pr;
      pv_load(L, k - 1, pr);
      pv_mma(L, k - 1, pr);
    }
  }

  // ---- final: score waves publish m and l; every wave normalises its columns
  {
  const LaneIds Lf = lane_ids();
  const int col = Lf.col, quad = Lf.quad;
  lsum = xor_sum_16_32(lsum);
  __syncthreads();  // every wave is past its last P.V: the rescale records are free
  float *const m_x = reinterpret_cast<float *>(xbuf + C::XFLAGS);
  float *const l_x = reinterpret_cast<float *>(xbuf + C::XBYTES + C::XFLAGS);
  if (quad == 0) {
    m_x[16 * wave + col] = m;
    l_x[16 * wave + col] = lsum;
  }
  __syncthreads();
  const bool split = rq.ws_base != kNoWs;
#pragma unroll
  for (int hb = 0; hb < C::HB; ++hb) {
    const uint32_t head = (uint32_t)(h0 + 16 * hb + col);
    const float inv = 1.0f / l_x[16 * hb + col];
#pragma unroll
    for (int db = 0; db < C::DBW; ++db) {
      const int d = (C::DV / NW) * wave + 16 * db + 4 * quad;
      const f32x4 v = o[db][hb] * inv;
      uint16_t *dst = split ? a.ws_o + ((uint64_t)rq.ws_orow + (uint64_t)slot * gm.hq + head) * C::DV + d
                            : a.out + rq.o_off + head * C::DV + d;
      *reinterpret_cast<uint2 *>(dst) = bf16x4_bits(v[0], v[1], v[2], v[3]);
    }
  }
  if (quad == 0) {
    const uint32_t head = (uint32_t)(h0 + 16 * wave + col);
    const float lse = (m + fast_log2(lsum)) * kLn2;
    if (split)
      a.ws_l[(uint64_t)rq.ws_base + (uint64_t)slot * gm.hq + head] = lse;
    else
      a.lse[rq.lse_off + head] = lse;
  }
  }
  __syncthreads();  // LDS is reused by the next unit
}

}  // namespace cp
