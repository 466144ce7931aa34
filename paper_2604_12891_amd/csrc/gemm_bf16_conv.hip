// x_proj of a bf16 model with the causal depthwise conv + SiLU in front
// (section 5.2's Mamba block: conv, SiLU, then the projection to
// [dt_r | B | C]), on the bf16 matrix cores.
//
// A workgroup owns 128 packed rows (32 per wavefront) and all N <= 64
// columns, walking the channels in chunks of 128. Per chunk each wavefront
// computes the conv + SiLU of its 32 rows (lane = two channels, so the 35
// input rows -- three of them before the wavefront's first row -- are
// 256-byte coalesced loads, held in registers one chunk ahead), rounds to
// bf16, parks the chunk in LDS, stores u from there in 16-byte rows (the
// scan reads it) and reads its MFMA fragments back in the fragment layout.
// Taps that reach before a program's first token read zero; the taps are
// summed in the order of the stand-alone conv kernel and rounded the same
// way, so u is the same bits either way.
#include "common.h"
#include "kernels.h"

namespace tcl {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int kWaves = 4;
constexpr uint32_t kBufferFlags = 0x00020000;  // 32-bit data format, raw (stride 0)
constexpr uint32_t kOutOfRange = 0x80000000u;  // beyond every resource used here

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, bytes, kBufferFlags);
}
// copies the compiler cannot see through (values derived from them are
// rebuilt per chunk instead of being kept live across all chunks)
__device__ __forceinline__ uint32_t opaque_s(uint32_t v) {
  asm volatile("" : "+s"(v));
  return v;
}
__device__ __forceinline__ uint32_t opaque_v(uint32_t v) {
  asm volatile("" : "+v"(v));
  return v;
}

template <int KCH>
__global__ __launch_bounds__(kWaves * 64, 2) void gemm_bf16conv_kernel(ConvArgsBF16 p) {
  constexpr int CW = 128;        // channels per chunk
  constexpr int NS = CW / 16;    // MFMA k-steps per chunk
  constexpr int PA = CW + 8;     // bf16 pitch of a parked row (conflict-free 16-byte reads)
  constexpr int WPB = CW + 8;    // bf16 pitch of a staged W row
  constexpr int XR = 32 + 3;     // conv input rows per wavefront
  constexpr int BM = kWaves * 32;
  __shared__ __attribute__((aligned(16))) uint16_t sW[2 * 32 * WPB];
  __shared__ __attribute__((aligned(16))) uint16_t sA[BM * PA];

  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63;
  const int li = lane & 31, lg = lane >> 5;
  const int M = *p.Mdev;
  const int row0 = blockIdx.x * BM;
  if (row0 >= M) return;
  const int E = p.E;

  // W [N][ldw] bf16: a block is 32 rows x 128 k, two 16-byte units per thread
  const __amdgpu_buffer_rsrc_t wres =
      make_rsrc(p.W, (uint32_t)__builtin_amdgcn_readfirstlane(p.N * p.ldw * 2));
  u32x4 wr[2];
  auto wload = [&](int nb, int c) {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int u = tid + i * 256;
      const int n = nb * 32 + (u >> 4), k = c * CW + 8 * (u & 15);
      const bool ok = n < p.N && k < E;
      const uint32_t off = (uint32_t)((n * p.ldw + k) * 2) | ((uint32_t)!ok << 31);
      wr[i] = __builtin_amdgcn_raw_buffer_load_b128(wres, off, 0, 0);
    }
  };
  auto wstage = [&](int buf) {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int u = tid + i * 256;
      *reinterpret_cast<u32x4*>(&sW[buf * 32 * WPB + (u >> 4) * WPB + 8 * (u & 15)]) = wr[i];
    }
  };
  wload(0, 0);

  // rows wb .. wb + 31; p0 = position of row wb in its program (clamped to
  // 3); bit r of `starts` (r >= 1): row wb + r is a program's first row
  const int wb = row0 + wave * 32;
  int tp = 3;
  if (lane < 32 && wb + lane < M) tp = min((int)p.tpos[wb + lane], 3);
  const uint32_t p0 = (uint32_t)__builtin_amdgcn_readfirstlane(tp);
  const uint32_t starts = (uint32_t)__builtin_amdgcn_ballot_w64(lane >= 1 && lane < 32 && tp == 0);
  const int xr0 = max(row0 - 3, 0);
  const int xrows = min(M, row0 + BM) - xr0;
  const __amdgpu_buffer_rsrc_t xres = make_rsrc(p.x + (int64_t)xr0 * p.ldx, (uint32_t)(xrows * p.ldx * 2));
  const __amdgpu_buffer_rsrc_t ures = make_rsrc(p.u + (int64_t)row0 * E, (uint32_t)(min(BM, M - row0) * E * 2));
  const __amdgpu_buffer_rsrc_t cwres = make_rsrc(p.w, (uint32_t)(E * 4 * 4));
  const __amdgpu_buffer_rsrc_t cbres = make_rsrc(p.b, (uint32_t)(E * 4));

  const uint32_t ldx2 = (uint32_t)(p.ldx * 2);
  uint32_t xw[XR];
  u32x4 cw0, cw1;
  u32x2 cb;
  auto load_chunk = [&](int c) {
    const uint32_t e = c * CW + 2 * lane;
    const uint32_t ve = opaque_v(e * 2), ld = opaque_s(ldx2);
#pragma unroll
    for (int i = 0; i < XR; ++i) {
      const int row = wb - 3 + i;
      const uint32_t off = row >= 0 ? (uint32_t)(row - xr0) * ld + ve : kOutOfRange;
      xw[i] = __builtin_amdgcn_raw_buffer_load_b32(xres, off, 0, 0);
    }
    cw0 = __builtin_amdgcn_raw_buffer_load_b128(cwres, ve * 8, 0, 0);
    cw1 = __builtin_amdgcn_raw_buffer_load_b128(cwres, ve * 8 + 16, 0, 0);
    cb = __builtin_amdgcn_raw_buffer_load_b64(cbres, ve * 2, 0, 0);
  };
  load_chunk(0);

  floatx16 acc[2];
#pragma unroll
  for (int nb = 0; nb < 2; ++nb)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[nb][r] = 0.f;
  wstage(0);

  uint16_t* myA = &sA[wave * 32 * PA];
#pragma unroll
  for (int c = 0; c < KCH; ++c) {
    __builtin_amdgcn_sched_barrier(0);
    {
      const float w[2][4] = {{__uint_as_float(cw0.x), __uint_as_float(cw0.y), __uint_as_float(cw0.z),
                              __uint_as_float(cw0.w)},
                             {__uint_as_float(cw1.x), __uint_as_float(cw1.y), __uint_as_float(cw1.z),
                              __uint_as_float(cw1.w)}};
      const float bias[2] = {__uint_as_float(cb.x), __uint_as_float(cb.y)};
      const uint32_t pc = opaque_s(p0), sc = opaque_s(starts);
      if (pc < 3) xw[0] = 0u;
      if (pc < 2) xw[1] = 0u;
      if (pc < 1) xw[2] = 0u;
#pragma unroll
      for (int r = 0; r < 32; ++r) {
        // row wb + r starts a program: the three rows before it are no
        // longer anyone's taps
        if (r > 0 && ((sc >> r) & 1u)) xw[r] = xw[r + 1] = xw[r + 2] = 0u;
        float o[2];
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          auto xv = [&](int i) { return __uint_as_float(j ? (xw[i] & 0xFFFF0000u) : (xw[i] << 16)); };
          float a = bias[j];
          a = fmaf(w[j][0], xv(r), a);
          a = fmaf(w[j][1], xv(r + 1), a);
          a = fmaf(w[j][2], xv(r + 2), a);
          a = fmaf(w[j][3], xv(r + 3), a);
          o[j] = silu(a);
        }
        *reinterpret_cast<uint32_t*>(&myA[r * PA + 2 * lane]) = f32x2_to_bf16x2(o[0], o[1]);
      }
    }
    if (c + 1 < KCH) load_chunk(c + 1);
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    // u: the parked rows stored 16 bytes per lane (four rows per instruction)
    {
      const uint32_t uo = opaque_v((uint32_t)((wave * 32 + (lane >> 4)) * E + c * CW + 8 * (lane & 15)) * 2);
      const uint32_t ur = opaque_s((uint32_t)E * 8);
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const u32x4 v = *reinterpret_cast<const u32x4*>(&myA[(4 * i + (lane >> 4)) * PA + 8 * (lane & 15)]);
        __builtin_amdgcn_raw_buffer_store_b128(v, ures, uo + i * ur, 0, 0);
      }
    }
    bf16x8 a[NS];
#pragma unroll
    for (int s2 = 0; s2 < NS; ++s2)
      a[s2] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(&myA[li * PA + 16 * s2 + 8 * lg]));
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
    for (int nb = 0; nb < 2; ++nb) {
      const int buf = (c * 2 + nb) & 1;
      __syncthreads();  // this block visible; the other buffer is free for the next
      const bool more = nb == 0 || c + 1 < KCH;
      if (nb == 0) wload(1, c);
      else if (c + 1 < KCH) wload(0, c + 1);
      const uint16_t* wbp = &sW[buf * 32 * WPB + li * WPB + 8 * lg];
#pragma unroll
      for (int ks = 0; ks < NS; ++ks) {
        const bf16x8 wf = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(wbp + 16 * ks));
        acc[nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[ks], wf, acc[nb], 0, 0, 0);
      }
      if (more) wstage(buf ^ 1);
    }
  }

  // epilogue: lane l holds column nb*32 + l % 32 and rows 8*(r/4) + 4*(l/32) + (r%4)
  const __amdgpu_buffer_rsrc_t cres =
      make_rsrc(p.C + (int64_t)row0 * p.ldc, (uint32_t)(min(BM, M - row0) * p.ldc * 4));
#pragma unroll
  for (int nb = 0; nb < 2; ++nb) {
    const int col = nb * 32 + li;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int rl = 8 * (r >> 2) + 4 * lg + (r & 3);
      const uint32_t off = (uint32_t)(((wave * 32 + rl) * p.ldc + col) * 4) | ((uint32_t)(col >= p.N) << 31);
      __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(acc[nb][r]), cres, off, 0, 0);
    }
  }
}

}  // namespace

bool gemm_bf16_conv_supports(const ConvArgsBF16& a, int d_conv) {
  const auto a16 = [](const void* q) { return reinterpret_cast<uintptr_t>(q) % 16 == 0; };
  return d_conv == 4 && a.E % 128 == 0 && a.E >= 128 && a.E <= 512 && a.N >= 1 && a.N <= 64 && a.x && a.w &&
         a.b && a.tpos && a.u && a.W && a.C && a.Mdev && a16(a.x) && a16(a.w) && a16(a.u) && a16(a.W) &&
         a.ldx % 8 == 0 && a.ldx >= a.E && a.ldw % 8 == 0 && a.ldw >= a.E &&
         (int64_t)(kWaves * 32 + 3) * a.ldx * 2 < (1ll << 31) && (int64_t)kWaves * 32 * a.ldc * 4 < (1ll << 31);
}

hipError_t launch_gemm_bf16_conv(const ConvArgsBF16& a, hipStream_t s) {
  if (!gemm_bf16_conv_supports(a, 4)) return hipErrorInvalidValue;
  const int grid = (a.Mmax + kWaves * 32 - 1) / (kWaves * 32);
  if (grid <= 0) return hipSuccess;
  switch (a.E / 128) {
    case 1: hipLaunchKernelGGL((gemm_bf16conv_kernel<1>), dim3(grid), dim3(kWaves * 64), 0, s, a); break;
    case 2: hipLaunchKernelGGL((gemm_bf16conv_kernel<2>), dim3(grid), dim3(kWaves * 64), 0, s, a); break;
    case 3: hipLaunchKernelGGL((gemm_bf16conv_kernel<3>), dim3(grid), dim3(kWaves * 64), 0, s, a); break;
    case 4: hipLaunchKernelGGL((gemm_bf16conv_kernel<4>), dim3(grid), dim3(kWaves * 64), 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace tcl
