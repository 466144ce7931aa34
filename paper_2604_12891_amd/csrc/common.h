// Device helpers shared by the gfx950 kernels of libtcl.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace tcl {

constexpr float kLog2e = 1.4426950408889634f;

typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef float floatx16 __attribute__((ext_vector_type(16)));

// SiLU(x) = x * sigmoid(x).
__device__ __forceinline__ float silu(float x) { return x / (1.0f + expf(-x)); }

// softplus(x) = log(1 + e^x). log1pf keeps full relative precision for the
// small step sizes (dt ~ 1e-3) that the dt bias initialisation produces.
__device__ __forceinline__ float softplus(float x) {
  return x > 20.0f ? x : log1pf(expf(x));
}

// Sum over the 64 lanes of a wavefront; every lane receives the total.
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// bf16 <-> fp32. bf16 is the high half of an fp32; rounding is to nearest,
// ties to even (NaN inputs are not produced by the model's arithmetic).
__device__ __forceinline__ float bf16_to_f32(uint16_t h) {
  return __uint_as_float(((uint32_t)h) << 16);
}
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

}  // namespace tcl
