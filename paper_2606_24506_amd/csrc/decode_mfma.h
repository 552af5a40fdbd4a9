// Pieces shared by the matrix-core decode kernels (decode_narrow.h,
// decode_wide.h): operand vector types, direct HBM -> LDS loads with the
// non-temporal policy, vmcnt waits, and constants of the online softmax.
#pragma once

#include <hip/hip_runtime.h>

#include "device_common.h"
#include "kargs.h"

namespace cp {

typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

constexpr float kLazy = 8.0f;  // log2 headroom before the softmax reference moves

// Instruction classes of __builtin_amdgcn_sched_group_barrier.
constexpr int kSgValu = 0x2, kSgMfma = 0x8, kSgDsRead = 0x100, kSgDsWrite = 0x200, kSgTrans = 0x400;

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
// Two floats rounded to bf16 (nearest even), packed low | high << 16.
CP_DEV uint32_t pack_bf16x2(float lo, float hi) {
  const bf16x2 v = {(__bf16)lo, (__bf16)hi};
  return __builtin_bit_cast(uint32_t, v);
}

// Direct HBM -> LDS loads are issued through inline asm, so the compiler
// does not put a full vmcnt wait before every LDS read; completion is
// awaited with wait_vm<N>() below. KV is streamed once per call, so the
// loads carry the non-temporal policy (nt): on MI355X that lifts
// page-scattered reads from about 4.7 to about 6.8 TB/s. M0 is written
// inside the same asm statement as the loads that use it; nothing else in
// these kernels uses M0.
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
// Direct loads of N consecutive 1 KiB LDS chunks with a single M0 write:
// load j lands at lds_base + 1024 j + 16 lane and reads global address
// sbase + voff[j] + 1024 j (the instruction offset applies to both sides).
// Writing M0 makes a wave wait until its previous direct load has left the
// issue queue, so grouping four loads per M0 write removes most of that
// stall. Callers pass sbase lowered by kDmaBias and add kDmaBias to every
// offset, which keeps the unsigned per-lane offsets non-negative.
constexpr uint32_t kDmaBias = 4096;
template <int N>
CP_DEV void dma_group(uint64_t sbase, const uint32_t (&voff)[4], uint32_t lds_base) {
  static_assert(N >= 1 && N <= 4, "one to four loads per M0 write");
  lds_base = __builtin_amdgcn_readfirstlane(lds_base);
  if constexpr (N == 1) {
    asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, %2 nt" ::"v"(voff[0]), "s"(lds_base), "s"(sbase)
                 : "memory", "m0");
  } else if constexpr (N == 2) {
    asm volatile(
        "s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %3 nt\n\tglobal_load_lds_dwordx4 %1, %3 offset:1024 nt" ::"v"(
            voff[0]),
        "v"(voff[1]), "s"(lds_base), "s"(sbase)
        : "memory", "m0");
  } else if constexpr (N == 3) {
    asm volatile(
        "s_mov_b32 m0, %3\n\tglobal_load_lds_dwordx4 %0, %4 nt\n\tglobal_load_lds_dwordx4 %1, %4 offset:1024 nt\n\t"
        "global_load_lds_dwordx4 %2, %4 offset:2048 nt" ::"v"(voff[0]),
        "v"(voff[1]), "v"(voff[2]), "s"(lds_base), "s"(sbase)
        : "memory", "m0");
  } else {
    asm volatile(
        "s_mov_b32 m0, %4\n\tglobal_load_lds_dwordx4 %0, %5 nt\n\tglobal_load_lds_dwordx4 %1, %5 offset:1024 nt\n\t"
        "global_load_lds_dwordx4 %2, %5 offset:2048 nt\n\tglobal_load_lds_dwordx4 %3, %5 offset:3072 nt" ::"v"(voff[0]),
        "v"(voff[1]), "v"(voff[2]), "v"(voff[3]), "s"(lds_base), "s"(sbase)
        : "memory", "m0");
  }
}

// A pointer known to be the same in every lane, moved to scalar registers.
CP_DEV uint64_t uniform_ptr(const void *p) {
  const uint64_t v = (uint64_t)(uintptr_t)p;
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(v >> 32));
  return ((uint64_t)hi << 32) | lo;
}
#pragma clang diagnostic pop

// s_waitcnt immediate of vmcnt(0) with the other counters unconstrained.
constexpr int kWaitVmcnt0 = 0x0F70;

template <int N>
CP_DEV void wait_vm() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

CP_DEV uint32_t lds_addr(const void *p) { return (uint32_t)(uintptr_t)p; }

// Row pitch of K and V tiles in LDS: a row of R bytes (a multiple of 128)
// plus 32 bytes. With rows 2 mod 8 16-byte chunks apart, both the K operand
// reads (16 rows x 16 bytes per lane group) and the V transpose reads of
// these kernels are free of bank conflicts on gfx950; a 16-byte pad (1 mod
// 8) halves their rate, an unpadded row quarters it.
constexpr int lds_pitch(int row_bytes) { return row_bytes + 32; }

// Reductions over lanes l, l^16, l^32, l^48 (the four lane groups that hold
// one column of an mfma 16x16 result), by the gfx950 half-row and half-wave
// swaps: a swap of x with itself leaves lane l's partner value in one of the
// two results and its own in the other, so the pair reduces to both.
CP_DEV float xor_max_16_32(float x) {
  auto p = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  const float a = __uint_as_float(p[0]), b = __uint_as_float(p[1]);
  const float y = a > b ? a : b;
  auto q = __builtin_amdgcn_permlane16_swap(__float_as_uint(y), __float_as_uint(y), false, false);
  const float c = __uint_as_float(q[0]), d = __uint_as_float(q[1]);
  return c > d ? c : d;
}
CP_DEV float xor_sum_16_32(float x) {
  auto p = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  const float y = __uint_as_float(p[0]) + __uint_as_float(p[1]);
  auto q = __builtin_amdgcn_permlane16_swap(__float_as_uint(y), __float_as_uint(y), false, false);
  return __uint_as_float(q[0]) + __uint_as_float(q[1]);
}

}  // namespace cp
