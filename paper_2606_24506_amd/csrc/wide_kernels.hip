// gfx950 decode kernels of the wide matrix path (64 or 128 query heads per
// KV head): the pipelined 128-head MLA kernel (decode_mla.h) and one
// instantiation of the generic wide kernel (decode_wide.h) per head_dim-128
// geometry.
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include "decode_mla.h"
#include "decode_wide.h"
#include "kargs.h"
#include "schedule.h"

namespace cp {

template <int V> struct WideVar;
template <> struct WideVar<kM_D128_G64> { static constexpr int G = 64, DK = 128, DV = 128, QL = 0, NW = 4; static constexpr bool MLA = false; };
template <> struct WideVar<kM_D128_G128> { static constexpr int G = 128, DK = 128, DV = 128, QL = 0, NW = 4; static constexpr bool MLA = false; };

// 128-head MLA: one workgroup of eight waves per CU.
__global__ __launch_bounds__(64 * MlaCfg::NW, 1) void decode_mla_kernel(const DecodeArgs a) {
  __shared__ __attribute__((aligned(16))) char lds[MlaCfg::LDS];
  __shared__ uint32_t next;
  decode_loop(a, &next, [&](const DecReq &rq, const Seg &sg) { mla_unit(a, a.geom[sg.model], rq, sg, lds); });
}

// One workgroup of four waves per CU; every request of the launch uses
// variant V.
template <int V>
__global__ __launch_bounds__(64 * WideVar<V>::NW, 1) void decode_wide_kernel(const DecodeArgs a) {
  using W = WideVar<V>;
  using C = WideCfg<W::G, W::DK, W::DV, W::MLA, W::QL, W::NW>;
  __shared__ __attribute__((aligned(16))) char lds[C::LDS];
  __shared__ uint32_t next;
  decode_loop(a, &next, [&](const DecReq &rq, const Seg &sg) {
    wide_unit<W::G, W::DK, W::DV, W::MLA, W::QL, W::NW>(a, a.geom[sg.model], rq, sg, lds);
  });
}

// ev0 / ev1 (may be null) take the start and end time of the launch.
hipError_t launch_decode_wide(const DecodeArgs &a, int grid, int variant, hipStream_t stream, hipEvent_t ev0,
                              hipEvent_t ev1) {
  const dim3 g(grid);
  switch (variant) {
    case kM_MLA_G128:
      hipExtLaunchKernelGGL(decode_mla_kernel, g, dim3(64 * MlaCfg::NW), 0, stream, ev0, ev1, 0, a);
      return hipGetLastError();
    case kM_D128_G64:
      hipExtLaunchKernelGGL((decode_wide_kernel<kM_D128_G64>), g, dim3(64 * WideVar<kM_D128_G64>::NW), 0, stream, ev0, ev1, 0, a);
      return hipGetLastError();
    case kM_D128_G128:
      hipExtLaunchKernelGGL((decode_wide_kernel<kM_D128_G128>), g, dim3(64 * WideVar<kM_D128_G128>::NW), 0, stream, ev0, ev1, 0, a);
      return hipGetLastError();
    default:
      return hipErrorInvalidValue;
  }
}

}  // namespace cp
