// Device helpers shared by the gfx950 kernels of libtcl.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace tcl {

constexpr float kLog2e = 1.4426950408889634f;

typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef float floatx16 __attribute__((ext_vector_type(16)));

constexpr float kLn2 = 0.6931471805599453f;

// exp(x) and 1/x on the transcendental unit (v_exp_f32 / v_rcp_f32, ~1 ulp).
// exp(x) is exp2(x * log2 e); the rounding of the product costs a relative
// error of |x| * 2^-24 * ln 2, i.e. < 1e-6 for |x| < 20.
__device__ __forceinline__ float exp_fast(float x) { return __builtin_amdgcn_exp2f(x * kLog2e); }
__device__ __forceinline__ float rcp_fast(float x) { return __builtin_amdgcn_rcpf(x); }

// SiLU(x) = x * sigmoid(x) = x / (1 + e^-x). For x < -88, e^-x = inf and the
// result is -0; relative error < 4e-6 elsewhere.
__device__ __forceinline__ float silu(float x) { return x * rcp_fast(1.0f + exp_fast(-x)); }

// log(1 + w) for w in [0, 1]: log2(u) with u = fl(1 + w), rescaled by
// w / (u - 1), which cancels the rounding of u exactly (u - 1 is exact) --
// D. Goldberg, "What every computer scientist should know about
// floating-point arithmetic", 1991, Theorem 4. The hardware log2 keeps its
// relative accuracy next to 1 (measured on gfx950: < 2 ulp of log2(u) for u
// in (1, 2), < 3e-7 relative for the result); w below 2^-24 (u = 1) is its
// own log1p.
__device__ __forceinline__ float log1p_unit(float w) {
  const float u = 1.0f + w;
  const float r = __builtin_amdgcn_logf(u) * kLn2 * (w * rcp_fast(u - 1.0f));
  return u == 1.0f ? w : r;
}

// softplus(x) = log(1 + e^x) = max(x, 0) + log1p(e^-|x|); relative error
// < 2e-6 over the whole range, including the dt ~ 1e-3 regime (x ~ -7)
// where log(1 + e^x) computed directly would lose most digits.
__device__ __forceinline__ float softplus(float x) {
  return fmaxf(x, 0.0f) + log1p_unit(exp_fast(-fabsf(x)));
}

// Raw buffer resource over `bytes` bytes at `base` (32-bit words, no
// stride): loads beyond `bytes` return 0 and stores beyond it are dropped.
// Its offsets are a per-lane VGPR part plus a wave-uniform SGPR part.
constexpr uint32_t kRawBufferFlags = 0x00020000;
__device__ __forceinline__ __amdgpu_buffer_rsrc_t raw_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, bytes, kRawBufferFlags);
}

// Sum over the 64 lanes of a wavefront; every lane receives the total.
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// bf16 <-> fp32. bf16 is the high half of an fp32. Narrowing uses gfx950's
// v_cvt_pk_bf16_f32 (round to nearest, ties to even).
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float floatx2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ float bf16_to_f32(uint16_t h) {
  return __uint_as_float(((uint32_t)h) << 16);
}
// two values -> one 32-bit word, a in the low half
__device__ __forceinline__ uint32_t f32x2_to_bf16x2(float a, float b) {
  const bf16x2_t h = __builtin_convertvector(floatx2_t{a, b}, bf16x2_t);
  return __builtin_bit_cast(uint32_t, h);
}
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  return (uint16_t)(f32x2_to_bf16x2(f, 0.0f) & 0xFFFFu);
}

// Exact three-way split of fp32 values into bf16 parts, x = x1 + x2 + x3:
// x1 = bf16(x), x2 = bf16(x - x1), x3 = x - x1 - x2. Both differences are
// exact in fp32, |x2| <= 2^-8 |x|, |x3| <= 2^-16 |x|, and x3 has at most 8
// significant bits, so bf16 holds it exactly (values below ~2^-110, whose
// parts would be denormal, aside). Two values at a time; each output word
// holds a's part in its low half and b's in its high half.
__device__ __forceinline__ void split3_pair(float a, float b, uint32_t& h, uint32_t& m, uint32_t& l) {
  h = f32x2_to_bf16x2(a, b);
  const float ra = a - __uint_as_float(h << 16), rb = b - __uint_as_float(h & 0xFFFF0000u);
  m = f32x2_to_bf16x2(ra, rb);
  l = f32x2_to_bf16x2(ra - __uint_as_float(m << 16), rb - __uint_as_float(m & 0xFFFF0000u));
}

// Two-part fp16 form of fp32 values (the fp16 split GEMMs): x = h + 2^-11 l
// + r, h = fp16(x), l = fp16(2^11 (x - h)), |r| <= 2^-22 |x| while x is in
// fp16's normal range. Weights are scaled by 2^kF16WeightExp first.
constexpr int kF16WeightExp = 10;
constexpr float kF16LowScale = 2048.0f;  // 2^11
__device__ __forceinline__ void split2_f16_scaled(float v, uint16_t& h, uint16_t& l) {
  const float x = v * (float)(1 << kF16WeightExp);
  const _Float16 hh = (_Float16)x;
  const _Float16 ll = (_Float16)((x - (float)hh) * kF16LowScale);
  h = __builtin_bit_cast(uint16_t, hh);
  l = __builtin_bit_cast(uint16_t, ll);
}
// The same with the low part unscaled, l = fp16(x - h), for kernels that sum
// all part products into one accumulator; |r| <= 2^-22 |x| while x - h is
// in fp16's normal range (|x| >= 2^-3 after the 2^10 scale).
__device__ __forceinline__ void split2_f16_flat(float v, uint16_t& h, uint16_t& l) {
  const float x = v * (float)(1 << kF16WeightExp);
  const _Float16 hh = (_Float16)x;
  const _Float16 ll = (_Float16)(x - (float)hh);
  h = __builtin_bit_cast(uint16_t, hh);
  l = __builtin_bit_cast(uint16_t, ll);
}

}  // namespace tcl
