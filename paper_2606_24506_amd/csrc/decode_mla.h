// Matrix-core decode path for DeepSeek-V3-shaped MLA (section 2.2's latent
// attention): 128 query heads read one latent KV head whose 576-element rows
// hold the 512-element value part first and the 64-element rotary part last.
// Per token that is about 240 flop per KV byte, so streaming KV at HBM speed
// needs the matrix cores busy most of the time; the kernel is built around
// keeping them fed.
//
// Eight waves, two per SIMD, with different jobs; tiles are T = 32 tokens.
//   score waves 0..3 (the older wave of each SIMD, which the hardware issues
//           for first): wave w scores heads [32 w, 32 w + 32), S^T[t][h] =
//           sum_d K[t][d] Q[h][d] with mfma 16x16x32 bf16 (K rows from LDS as
//           the A operand, feeding the wave's two head blocks of query
//           fragments held in registers as B), then runs the fp32 online
//           softmax with a lazily moved reference and publishes P^T to LDS
//           as bf16 operand fragments; it also accumulates P.V for value
//           column block w (16 columns) of all 128 heads.
//   P.V waves 4..7: wave 4 + j accumulates O^T[d][h] += sum_t V^T[d][t]
//           P^T[t][h] for column blocks 4 + 7 j .. 4 + 7 j + 6 of all 128
//           heads, and issues the direct HBM -> LDS tile loads, all of a
//           tile right after the barrier that frees its slot (the loads
//           need the lead time). The token index of that product runs
//           {4q..4q+3, 16+4q..16+4q+3} for lane group q, which is how the
//           score accumulators hold P; V^T comes from LDS transpose reads.
// Software pipeline with one workgroup barrier per tile: iteration k runs
// the scores and softmax of tile k and the P.V product of tile k-1 (a score
// wave's eight P.V products go between its score products), with P^T and
// the rescale records double-buffered by tile parity. On every SIMD the
// score wave's softmax and its waits for K fragments are the P.V wave's
// matrix-core issue slots, and each K fragment read from LDS feeds two
// products.
//
// LDS (160 KiB): a ring of four value tiles (32 rows of 1024 bytes), a ring
// of three rotary tiles (32 rows of 128 bytes: the rotary part is only read
// by the scores of its own tile, one iteration less than the value part),
// two P^T buffers of 8 KiB and two rescale records. Rows carry no padding:
// 16-byte chunk g of row r is stored at chunk g ^ (2r mod 16) in a value
// row and at g ^ (r & 6) in a rotary row, which keeps the K operand reads
// (16 rows x 16 bytes per lane group) and the V transpose reads free of
// bank conflicts. The direct loads apply the permutation through their
// per-lane source addresses, so every load writes one contiguous KiB (a
// rotary load: half a KiB) of LDS.
//
// Registers are the binding limit: a score wave holds 144 registers of
// query fragments and 32 of accumulators, a P.V wave 224 of accumulators.
// Per-lane constants are formed where they are used, from the lane index
// counted afresh each iteration: the compiler can neither hoist them out of
// the loop nor keep them in scratch memory, whose reloads would make it
// wait for every load in flight, tile loads included.
#pragma once

#include <type_traits>

#include "decode_mfma.h"

namespace cp {

struct MlaCfg {
  static constexpr int G = 128, DK = 576, DV = 512, NW = 8, T = 32;
  static constexpr int NSW = 4;                // score waves; the others multiply P.V
  static constexpr int HB = G / 16;            // head blocks
  static constexpr int SHB = HB / NSW;         // head blocks scored per score wave
  static constexpr int DB = DV / 16;           // value column blocks
  static constexpr int PDB = (DB - NSW) / (NW - NSW);  // column blocks per P.V wave (a score wave: one)
  static constexpr int KROW = DK * 2;          // bytes of one KV row in HBM
  static constexpr int MROW = DV * 2;          // value part: one value-ring row
  static constexpr int RROW = KROW - MROW;     // rotary part: one rotary-ring row
  static constexpr int MSLOT = T * MROW;       // 32 KiB
  static constexpr int RSLOT = T * RROW;       // 4 KiB
  static constexpr int NM = 4, NR = 3;         // ring depths
  static constexpr int KSTEPS = DK / 32;       // score k-steps
  static constexpr int KMAIN = DV / 32;        // ... of them in the value part
  static constexpr int LOADS = 9;              // direct loads per loading wave and tile
  static constexpr int PBYTES = HB * 64 * 16;  // P^T fragments of one tile
  static constexpr int XFLAGS = 16;             // rescale record: one flag byte per head block,
  static constexpr int XBYTES = XFLAGS + 4 * G;  // then alpha[G]
  static constexpr int OFF_R = NM * MSLOT;
  static constexpr int OFF_P = OFF_R + NR * RSLOT;
  static constexpr int OFF_X = OFF_P + 2 * PBYTES;
  static constexpr int LDS = OFF_X + 2 * XBYTES;
  static_assert(MROW == 1024 && RROW == 128, "one direct load per value row, eight rotary rows per load");
  static_assert((NW - NSW) * 8 == T, "each loading wave loads eight value rows and eight rotary rows");
  static_assert(SHB == 2 && NSW + (NW - NSW) * PDB == DB, "work split");
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

// V^T operand fragment of value column block b of a tile slot: this lane
// supplies value rows vr and vr + 16, bytes 8 (col & 3) of the block.
CP_DEV bf16x8 mla_vfrag(const char *vslot, const LaneIds &L, int b) {
  const int vr = 4 * L.quad + (L.col >> 2);
  const char *p0 = vslot + vr * MlaCfg::MROW + 8 * (L.col & 1) + 16 * ((2 * b + ((L.col >> 1) & 1)) ^ mla_vswz(vr));
  const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4 *)p0);
  const s16x4 hi =
      __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4 *)(p0 + 16 * MlaCfg::MROW));
  return __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
}

// Flag bytes of a rescale record, the same in every lane.
CP_DEV uint64_t mla_flags(const char *xrec) {
  const uint64_t f = *reinterpret_cast<const uint64_t *>(xrec);
  // the builtin returns a signed int: both halves are zero-extended
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)f);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(f >> 32));
  return ((uint64_t)hi << 32) | lo;
}

__device__ __forceinline__ void mla_unit(const DecodeArgs &a, const GeomK &gm, const DecReq &rq, const Seg &sg,
                                         char *lds) {
  using C = MlaCfg;
  constexpr int T = C::T;
  const uint32_t slot = sg.slot;
  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int P = gm.page_tokens;  // the host routes only pages of a multiple of 32 tokens here
  const int tpp = P / T;
  const int h0 = (int)sg.hblk * C::G;

  char *const vring = lds;
  char *const rring = lds + C::OFF_R;
  char *const pbuf = lds + C::OFF_P;
  char *const xbuf = lds + C::OFF_X;

  const uint32_t tok_end = min(rq.ctx_len, sg.pg_end * (uint32_t)P);
  const uint32_t pg_begin = sg.pg_begin;
  const int npg = (int)((tok_end + P - 1) / P) - (int)pg_begin;
  const int last_tok = npg > 0 ? (int)tok_end - (int)((pg_begin + (uint32_t)npg - 1) * (uint32_t)P) : 0;
  const int ntiles = npg > 0 ? (npg - 1) * tpp + (last_tok + T - 1) / T : 0;
  // tokens of tile k inside the piece
  auto tile_valid = [&](int k) {
    const int t0 = (int)((pg_begin + (uint32_t)(k / tpp)) * P) + (k % tpp) * T;
    return min(T, (int)tok_end - t0);
  };
  const bool split = rq.ws_base != kNoWs;
  float *const l_x = reinterpret_cast<float *>(xbuf + C::XBYTES + C::XFLAGS);
  const float sl2 = gm.scale_log2;

  if (wave < C::NSW) {
    // ================================================================ score wave
    const int w = wave;
    const LaneIds L0 = lane_ids();
    // Q^T operand fragments of the wave's head blocks 2w + i: lane holds
    // head (h0 + 16 (2w + i) + col), dims 32 c + 8 quad .. +7.
    bf16x8 qf[C::SHB][C::KSTEPS];
#pragma unroll
    for (int i = 0; i < C::SHB; ++i) {
      const uint16_t *qrow = a.q + rq.q_off + (uint32_t)(h0 + 16 * (C::SHB * w + i) + L0.col) * C::DK + 8 * L0.quad;
#pragma unroll
      for (int c = 0; c < C::KSTEPS; ++c) qf[i][c] = *reinterpret_cast<const bf16x8 *>(qrow + 32 * c);
    }
    // K operand read addresses of tile k (slice 0; slice 1 is 16 rows
    // further): value k-step 4a + b of row col sits at kva[b] + 256 a, kept
    // for the tile's value slot and moved on by one slot per tile; rotary
    // k-step c of row col at kra ^ (64 c), formed per tile.
    uint32_t kva[4];
    {
      const int s = mla_vswz(L0.col);
#pragma unroll
      for (int b = 0; b < 4; ++b)
        kva[b] = lds_addr(vring) + (uint32_t)(L0.col * C::MROW + 64 * (b ^ (s >> 2)) + 16 * (L0.quad ^ (s & 3)));
    }
    static_assert((C::MSLOT & (C::MSLOT - 1)) == 0 && C::NM == 4, "value slots rotate by masking");
    float m[C::SHB], lsum[C::SHB];
#pragma unroll
    for (int i = 0; i < C::SHB; ++i) m[i] = -INFINITY, lsum[i] = 0.f;
    f32x4 os[C::HB];  // column block w of every head block
#pragma unroll
    for (int hb = 0; hb < C::HB; ++hb) os[hb] = f32x4{0.f, 0.f, 0.f, 0.f};
    // the query loads are complete before the tile loop, as far as the
    // compiler can see, so it places no wait of its own inside the loop
    __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);

    // One iteration: the scores and softmax of tile k (HAS_S) and the P.V
    // share of tile k-1 (HAS_PV). The share's operands are read at the top
    // and its eight products go between the score products, one every nine.
    auto iter = [&](int k, auto has_s, auto has_pv) {
      constexpr bool HAS_S = decltype(has_s)::value, HAS_PV = decltype(has_pv)::value;
      // tile k visible; P^T and rescale record of tile k-1 complete; the
      // P^T buffer and record of tile k free
      __syncthreads();
      const LaneIds L = lane_ids();
      const int lane = L.lane, col = L.col, quad = L.quad;
      const int kp = k - 1;
      bf16x8 vf, pf[2];
      const char *pt = pbuf + (kp & 1) * C::PBYTES + lane * 16;
      if constexpr (HAS_PV) {
        const char *xr = xbuf + (kp & 1) * C::XBYTES;
        const uint64_t fl = mla_flags(xr);
        if (fl != 0) {
          const float *alpha = reinterpret_cast<const float *>(xr + C::XFLAGS);
#pragma unroll
          for (int hb = 0; hb < C::HB; ++hb)
            if ((fl >> (8 * hb)) & 0xFF) os[hb] *= alpha[16 * hb + col];
        }
        vf = mla_vfrag(vring + (kp % C::NM) * C::MSLOT, L, w);
        pf[0] = *reinterpret_cast<const bf16x8 *>(pt);
        pf[1] = *reinterpret_cast<const bf16x8 *>(pt + 1024);
      }
      // P.V share product of head block hb, then the read of hb + 2's P^T
      auto pv_step = [&](int hb) {
        os[hb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, pf[hb & 1], os[hb], 0, 0, 0);
        if (hb + 2 < C::HB) pf[hb & 1] = *reinterpret_cast<const bf16x8 *>(pt + (hb + 2) * 1024);
      };
      if constexpr (HAS_S) {
        const int valid = tile_valid(k);
        const uint32_t kra = lds_addr(rring + (k % C::NR) * C::RSLOT) +
                             (uint32_t)(col * C::RROW + 64 * (mla_rswz(col) >> 2) + 16 * (quad ^ (mla_rswz(col) & 3)));
        f32x4 s[C::SHB][2];
#pragma unroll
        for (int i = 0; i < C::SHB; ++i) s[i][0] = s[i][1] = f32x4{0.f, 0.f, 0.f, 0.f};
        auto kread = [&](int c, int sl) -> bf16x8 {
          const uint32_t ad = c < C::KMAIN ? kva[c & 3] + 256 * (c >> 2) + sl * 16 * C::MROW
                                           : (kra ^ (64 * (c - C::KMAIN))) + sl * 16 * C::RROW;
          return *reinterpret_cast<const bf16x8 *>(lds + (ad - lds_addr(lds)));
        };
        // K fragments are read KD fragments (2 KD products) ahead; the
        // scheduling barriers keep the compiler from sinking the reads back
        // to their uses
        constexpr int KD = 3;
#pragma unroll
        for (int sl = 0; sl < 2; ++sl) {
          bf16x8 kf[KD + 1];
#pragma unroll
          for (int c = 0; c < KD; ++c) kf[c] = kread(c, sl);
#pragma unroll
          for (int c = 0; c < C::KSTEPS; ++c) {
            if (c + KD < C::KSTEPS) kf[(c + KD) % (KD + 1)] = kread(c + KD, sl);
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int i = 0; i < C::SHB; ++i)
              s[i][sl] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[c % (KD + 1)], qf[i][c], s[i][sl], 0, 0, 0);
            if (HAS_PV && (c & 3) == 1 && c < 16) pv_step(4 * sl + (c >> 2));
          }
        }
        // ---- online softmax (lane: head col of each block, tokens 16 sl +
        // 4 quad + r). Scores stay unscaled; the (positive) scale is applied
        // to the maximum and folded into the exponent's fma. The reference
        // of a head moves when its new maximum passes it by kLazy, which
        // happens iff some lane's own maximum does: the lanes test their
        // own, and only a tile where one passes takes the head's maximum
        // across lanes.
        char *xw = xbuf + (k & 1) * C::XBYTES;
#pragma unroll
        for (int i = 0; i < C::SHB; ++i) {
          const int hb = C::SHB * w + i;
          if (valid < T) {
#pragma unroll
            for (int sl = 0; sl < 2; ++sl)
#pragma unroll
              for (int r = 0; r < 4; ++r)
                if (16 * sl + 4 * quad + r >= valid) s[i][sl][r] = -INFINITY;
          }
          float x = s[i][0][0];
#pragma unroll
          for (int sl = 0; sl < 2; ++sl)
#pragma unroll
            for (int r = 0; r < 4; ++r) x = __builtin_fmaxf(x, s[i][sl][r]);
          const bool any_bump = __builtin_amdgcn_ballot_w64(x * sl2 > m[i] + kLazy) != 0;
          if (any_bump) {
            const float mt = xor_max_16_32(x) * sl2;
            const float mn = mt > m[i] + kLazy ? mt : m[i];
            const float al = fast_exp2(m[i] - mn);
            m[i] = mn;
            lsum[i] *= al;
            if (quad == 0) reinterpret_cast<float *>(xw + C::XFLAGS)[16 * hb + col] = al;
          }
          if (lane == 0) reinterpret_cast<uint8_t *>(xw)[hb] = any_bump ? 1 : 0;
          bf16x8 pk;
          float ps = 0.f;
#pragma unroll
          for (int sl = 0; sl < 2; ++sl)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              // the row sum takes p in fp32; only the P.V operand is rounded to bf16
              const float p = fast_exp2(__builtin_fmaf(s[i][sl][r], sl2, -m[i]));
              ps += p;
              pk[4 * sl + r] = (__bf16)p;
            }
          lsum[i] += ps;
          *reinterpret_cast<bf16x8 *>(pbuf + (k & 1) * C::PBYTES + (hb * 64 + lane) * 16) = pk;
        }
        // the next tile's value slot
        const uint32_t vbase = lds_addr(vring);
#pragma unroll
        for (int b = 0; b < 4; ++b) kva[b] = vbase + ((kva[b] - vbase + C::MSLOT) & (C::NM * C::MSLOT - 1));
      } else if constexpr (HAS_PV) {
#pragma unroll
        for (int hb = 0; hb < C::HB; ++hb) pv_step(hb);
      }
    };
    using Yes = std::integral_constant<bool, true>;
    using No = std::integral_constant<bool, false>;
    if (ntiles > 0) {
      iter(0, Yes{}, No{});
#pragma unroll 1
      for (int k = 1; k < ntiles; ++k) iter(k, Yes{}, Yes{});
      iter(ntiles, No{}, Yes{});
    }

    // ---- final: publish the row sums; normalise column block w
    const LaneIds Lf = lane_ids();
#pragma unroll
    for (int i = 0; i < C::SHB; ++i) lsum[i] = xor_sum_16_32(lsum[i]);
    __syncthreads();  // every wave is past its last P.V: the rescale records are free
    if (Lf.quad == 0) {
#pragma unroll
      for (int i = 0; i < C::SHB; ++i) l_x[16 * (C::SHB * w + i) + Lf.col] = lsum[i];
    }
    __syncthreads();
#pragma unroll
    for (int hb = 0; hb < C::HB; ++hb) {
      const uint32_t head = (uint32_t)(h0 + 16 * hb + Lf.col);
      const f32x4 v = os[hb] * (1.0f / l_x[16 * hb + Lf.col]);
      const int d = 16 * w + 4 * Lf.quad;
      uint16_t *dst = split ? a.ws_o + ((uint64_t)rq.ws_orow + (uint64_t)slot * gm.hq + head) * C::DV + d
                            : a.out + rq.o_off + head * C::DV + d;
      *reinterpret_cast<uint2 *>(dst) = bf16x4_bits(v[0], v[1], v[2], v[3]);
    }
    if (Lf.quad == 0) {
#pragma unroll
      for (int i = 0; i < C::SHB; ++i) {
        const uint32_t head = (uint32_t)(h0 + 16 * (C::SHB * w + i) + Lf.col);
        const float lse = (m[i] + fast_log2(lsum[i])) * kLn2;
        if (split)
          a.ws_l[(uint64_t)rq.ws_base + (uint64_t)slot * gm.hq + head] = lse;
        else
          a.lse[rq.lse_off + head] = lse;
      }
    }
  } else {
    // ================================================================ P.V wave
    const int j = wave - C::NSW;
    const int b0 = C::NSW + C::PDB * j;  // first column block
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
    // Direct loads: P.V wave j loads value rows 8j .. 8j+7 (two groups of
    // four loads, one M0 write each) and rotary rows 8j .. 8j+7 (one load).
    // Per-lane source offsets (within the tile) place chunk (lane ^ swizzle)
    // of the row at LDS chunk `lane`.
    auto issue_value = [&](int k, uint64_t sb, int g) {
      const int lane = lane_ids().lane;
      const uint32_t lb =
          __builtin_amdgcn_readfirstlane(lds_addr(vring + (k % C::NM) * C::MSLOT) + j * 8192 + g * 4096);
      uint32_t vo[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int r = 8 * j + 4 * g + q;
        vo[q] = (uint32_t)(r * C::KROW + 16 * (lane ^ mla_vswz(r))) + kDmaBias - 1024u * q;
      }
      dma_group<4>(sb, vo, lb);
    };
    auto issue_rope = [&](int k, uint64_t sb) {
      const int lane = lane_ids().lane;
      const uint32_t lb = __builtin_amdgcn_readfirstlane(lds_addr(rring + (k % C::NR) * C::RSLOT) + j * 1024);
      const int r = 8 * j + (lane >> 3);
      const uint32_t vo[4] = {(uint32_t)(r * C::KROW + C::MROW + 16 * ((lane & 7) ^ mla_rswz(r))) + kDmaBias, 0u,
                              0u, 0u};
      dma_group<1>(sb, vo, lb);
    };

    f32x4 op[C::PDB][C::HB];
#pragma unroll
    for (int i = 0; i < C::PDB; ++i)
#pragma unroll
      for (int hb = 0; hb < C::HB; ++hb) op[i][hb] = f32x4{0.f, 0.f, 0.f, 0.f};

    if (ntiles > 0) {
      load_ptes(0);
      for (int k = 0; k < 2 && k < ntiles; ++k) {
        const uint64_t sb = tile_src(k);
        issue_value(k, sb, 0);
        issue_value(k, sb, 1);
        issue_rope(k, sb);
      }
    }

#pragma unroll 1
    for (int k = 0; k <= ntiles && ntiles > 0; ++k) {
      // own loads of tile k have landed once at most tile k+1's remain
      if (k + 1 < ntiles)
        wait_vm<C::LOADS>();
      else if (k < ntiles)
        wait_vm<0>();
      // tile k visible; P^T and rescale record of tile k-1 complete; the
      // value slot of tile k-2 and the rotary slot of tile k-1 are free
      __syncthreads();
      const int kn = k + 2;
      const bool more = kn < ntiles;
      const uint64_t sbn = more ? tile_src(kn) : 0;
      if (more) {
        issue_value(kn, sbn, 0);
        issue_value(kn, sbn, 1);
        issue_rope(kn, sbn);
      }
      if (k < ntiles) {
        const int valid = tile_valid(k);
        if (valid < T) {
          // value rows past the context may hold stale bytes: zero them so
          // that 0 * V stays 0 in the next iteration's P.V (their scores are
          // masked to -inf)
          char *vt = vring + (k % C::NM) * C::MSLOT;
          const int nz = (T - valid) * (C::MROW / 16);
          uint32_t z;  // a zero formed here, not a zero vector kept through the loop
          asm volatile("v_mov_b32 %0, 0" : "=v"(z));
          for (int i = j * 64 + lane_ids().lane; i < nz; i += 64 * (C::NW - C::NSW))
            *reinterpret_cast<uint4 *>(vt + valid * C::MROW + i * 16) = make_uint4(z, z, z, z);
        }
      }
      if (k >= 1) {
        // ---- P.V of tile k-1: apply the rescales the score waves asked
        // for, then the products, in four passes of two head blocks (V^T
        // fragments read once per pass, P^T fragments once)
        const int kp = k - 1;
        const LaneIds L = lane_ids();
        const char *xr = xbuf + (kp & 1) * C::XBYTES;
        const uint64_t fl = mla_flags(xr);
        if (fl != 0) {
          const float *alpha = reinterpret_cast<const float *>(xr + C::XFLAGS);
#pragma unroll
          for (int hb = 0; hb < C::HB; ++hb) {
            if ((fl >> (8 * hb)) & 0xFF) {
              const float ah = alpha[16 * hb + L.col];
#pragma unroll
              for (int i = 0; i < C::PDB; ++i) op[i][hb] *= ah;
            }
          }
        }
        const char *vs = vring + (kp % C::NM) * C::MSLOT;
        const char *pt = pbuf + (kp & 1) * C::PBYTES + L.lane * 16;
        constexpr int PH = 2;  // head blocks per pass
#pragma unroll
        for (int ps = 0; ps < C::HB / PH; ++ps) {
          bf16x8 pf[PH];
#pragma unroll
          for (int h = 0; h < PH; ++h) pf[h] = *reinterpret_cast<const bf16x8 *>(pt + (PH * ps + h) * 1024);
          bf16x8 vf[2];
          vf[0] = mla_vfrag(vs, L, b0);
#pragma unroll
          for (int i = 0; i < C::PDB; ++i) {
            if (i + 1 < C::PDB) vf[(i + 1) & 1] = mla_vfrag(vs, L, b0 + i + 1);
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int h = 0; h < PH; ++h)
              op[i][PH * ps + h] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf[i & 1], pf[h], op[i][PH * ps + h], 0, 0, 0);
          }
        }
      }
    }

    // ---- final: normalise column blocks b0 .. b0 + PDB - 1
    __syncthreads();  // every wave is past its last P.V: the rescale records are free
    __syncthreads();  // the score waves have published the row sums
    const LaneIds Lf = lane_ids();
#pragma unroll
    for (int hb = 0; hb < C::HB; ++hb) {
      const uint32_t head = (uint32_t)(h0 + 16 * hb + Lf.col);
      const float inv = 1.0f / l_x[16 * hb + Lf.col];
#pragma unroll
      for (int i = 0; i < C::PDB; ++i) {
        const int d = 16 * (b0 + i) + 4 * Lf.quad;
        const f32x4 v = op[i][hb] * inv;
        uint16_t *dst = split ? a.ws_o + ((uint64_t)rq.ws_orow + (uint64_t)slot * gm.hq + head) * C::DV + d
                              : a.out + rq.o_off + head * C::DV + d;
        *reinterpret_cast<uint2 *>(dst) = bf16x4_bits(v[0], v[1], v[2], v[3]);
      }
    }
  }
  __syncthreads();  // LDS is reused by the next unit
}

}  // namespace cp
