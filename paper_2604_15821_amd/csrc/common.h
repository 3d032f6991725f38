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

__device__ __forceinline__ float sigmoidf_(float a) { return 1.0f / (1.0f + __expf(-a)); }

// SiLU(a) = a * s, SiLU'(a) = s + a s (1 - s), SiLU''(a) = s (1 - s) (2 + a (1 - 2 s)),
// s = 1 / (1 + exp(-a)).  Evaluated with the accurate expf: the training step
// is checked against a float64 reference.
__device__ __forceinline__ float sig(float a) { return 1.0f / (1.0f + expf(-a)); }
__device__ __forceinline__ float silu(float a) { return a * sig(a); }
__device__ __forceinline__ float silu_d1(float a) {
  float s = sig(a);
  return s + a * s * (1.0f - s);
}
__device__ __forceinline__ float silu_d2(float a) {
  float s = sig(a);
  return s * (1.0f - s) * (2.0f + a * (1.0f - 2.0f * s));
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

__device__ __forceinline__ double wave_sum_d(double v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

__device__ __forceinline__ int lane_id() { return threadIdx.x & 63; }

inline unsigned cdiv(long long a, long long b) { return (unsigned)((a + b - 1) / b); }

}  // namespace janus
