// Shared device helpers of the HIP path (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/janus.h"

#define JANUS_HIP_TRY(expr)                                   \
  do {                                                        \
    hipError_t _e = (expr);                                   \
    if (_e != hipSuccess) return janus_set_hip_error(_e);     \
  } while (0)

int janus_set_hip_error(hipError_t e);

namespace janus {

constexpr int kWave = 64;

// SiLU(a) = a * s, SiLU'(a) = s + a s (1 - s), SiLU''(a) = s (1 - s) (2 + a (1 - 2 s)),
// s = 1 / (1 + exp(-a)), with the hardware exponential (v_exp_f32 on a * log2 e)
// and reciprocal (v_rcp_f32): relative error of s about 1e-6 at |a| = 20 and a few
// 1e-7 for |a| < 5, against the 1e-5 energy and 1e-3 gradient tolerances of the
// float64 comparison.  The GEMMs that apply these per element (SiLU of stored
// pre-activations, the SiLU' / SiLU'' epilogues) run 10-20 % faster than with the
// correctly rounded exp and division.  exp(-a) overflows to inf for a < -88 and
// rcp(inf) = 0, so s saturates cleanly at both ends.
__device__ __forceinline__ float sig(float a) { return __builtin_amdgcn_rcpf(1.0f + __expf(-a)); }
__device__ __forceinline__ float silu(float a) { return a * sig(a); }
__device__ __forceinline__ float silu_d1(float a) {
  float s = sig(a);
  return s + a * s * (1.0f - s);
}
__device__ __forceinline__ float silu_d2(float a) {
  float s = sig(a);
  return s * (1.0f - s) * (2.0f + a * (1.0f - 2.0f * s));
}

// Sum over the 64 lanes, returned (wave-uniform) in every lane: DPP steps
// inside each row of 16 lanes (quad_perm 1032, quad_perm 2301, half-row
// mirror, row mirror), then the four row sums read from lanes 0, 16, 32, 48
// and added in that order.
template <int CTRL>
__device__ __forceinline__ float dpp_step(float v) {
  return v + __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, true));
}
__device__ __forceinline__ float wave_sum(float v) {
  v = dpp_step<0xB1>(v);    // quad_perm(1, 0, 3, 2)
  v = dpp_step<0x4E>(v);    // quad_perm(2, 3, 0, 1)
  v = dpp_step<0x141>(v);   // row_half_mirror
  v = dpp_step<0x140>(v);   // row_mirror
  const int b = __float_as_int(v);
  return ((__int_as_float(__builtin_amdgcn_readlane(b, 0)) + __int_as_float(__builtin_amdgcn_readlane(b, 16))) +
          __int_as_float(__builtin_amdgcn_readlane(b, 32))) +
         __int_as_float(__builtin_amdgcn_readlane(b, 48));
}

__device__ __forceinline__ double wave_sum_d(double v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

__device__ __forceinline__ int lane_id() { return threadIdx.x & 63; }

inline unsigned cdiv(long long a, long long b) { return (unsigned)((a + b - 1) / b); }

}  // namespace janus
