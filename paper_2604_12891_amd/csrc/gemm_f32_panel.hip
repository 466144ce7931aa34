// Row-panel fp32 GEMMs: C[M, N] = rowscale * (A W^T) + bias on
// v_mfma_f32_32x32x2_f32 for K <= 256, and C (+)= A W^T (+ bias) on
// v_mfma_f32_16x16x4f32 for K <= 512.
//
// The tiled fp32 GEMM stages A and W through LDS every 32 or 64 k, with two
// barriers per chunk for 32-64 MFMAs per wavefront. Here a workgroup of 4
// wavefronts owns 128 rows and all N columns:
//
//  * prologue: each wavefront loads its 32 rows of A once (gathered rows for
//    the input Linear) and keeps them as fp32 MFMA fragments in registers
//    (K / 2 VGPRs); the RMSNorm row statistics come from the same registers;
//  * main loop: 32 columns of W at a time go through a double-buffered LDS
//    stage (one barrier per step, next step's W loaded into registers while
//    the MFMAs run); one step is K / 2 MFMAs per wavefront, so the barrier,
//    the staging and the epilogue are amortised over ~8K MFMA cycles;
//  * epilogue per step: row scale and bias, buffer stores straight from the
//    accumulators (32 lanes write one row's 32 consecutive floats).
//
// Fragment k-order (A and W alike): within each group of 8 k, lane half g
// supplies k = 8i + 4g + j in MFMA step 4i + j, so each lane reads its
// operands as 16-byte vectors.
#include "common.h"
#include "kernels.h"

namespace tcl {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kWaves = 4;
constexpr int BM = kWaves * 32;  // rows per workgroup
constexpr uint32_t kBufferFlags = 0x00020000;  // 32-bit data format, raw (stride 0)
constexpr uint32_t kOutOfRange = 0x80000000u;  // beyond every resource used here

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, bytes, kBufferFlags);
}

// G groups of 8 k (K <= 8 G)
template <int G, int FL>
__global__ __launch_bounds__(kWaves * 64, 2) void gemm_f32_panel_kernel(GemmArgs p) {
  constexpr int KP = 8 * G;          // padded K
  constexpr int WP = KP + 4;         // floats per staged W row (conflict-free 16-byte reads)
  constexpr int WU = KP / 4;         // 16-byte units per staged W row
  constexpr int NWU = 32 * WU;                  // W units per step
  constexpr int NW = (NWU + kWaves * 64 - 1) / (kWaves * 64);  // per thread (the last may be idle)
  constexpr bool kNorm = (FL & kRowNorm) != 0;

  __shared__ __attribute__((aligned(16))) float sW[2][32 * WP];
  __shared__ float sR[kWaves][32];
  __shared__ int sSrc[BM];

  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63;
  const int li = lane & 31, lg = lane >> 5;
  const int M = p.Mdev ? *p.Mdev : p.Mmax;
  const int row0 = blockIdx.x * BM;
  if (row0 >= M) return;

  // source row of each panel row (packed-token gather, or the row itself)
  for (int r = tid; r < BM; r += kWaves * 64) {
    const int grow = row0 + r;
    int src = grow < M ? grow : -1;
    if constexpr ((FL & kGather) != 0) {
      if (src >= 0) {
        int lo = 0, hi = p.B;
        while (hi - lo > 1) {
          const int mid = (lo + hi) >> 1;
          if (p.offs[mid] <= grow) lo = mid; else hi = mid;
        }
        src = lo * p.L + (grow - p.offs[lo]);
      }
    }
    sSrc[r] = src;
  }

  // W stage: unit i of this thread is row u / WU, k = 4 (u % WU); rows past
  // N read zero through the resource, units past K are zeroed when staged
  const __amdgpu_buffer_rsrc_t wres = make_rsrc(p.W, (uint32_t)(p.N * p.ldw * 4));
  const int nsteps = (p.N + 31) / 32;
  u32x4 rw[NW];
  auto gload_w = [&](int n0) {
#pragma unroll
    for (int i = 0; i < NW; ++i) {
      const int u = tid + i * kWaves * 64;
      const int n = n0 + u / WU, k = 4 * (u % WU);
      const uint32_t off = u < NWU ? (uint32_t)((n * p.ldw + k) * 4) : kOutOfRange;
      rw[i] = __builtin_amdgcn_raw_buffer_load_b128(wres, off, 0, 0);
    }
  };
  auto stage_w = [&](int buf) {
#pragma unroll
    for (int i = 0; i < NW; ++i) {
      const int u = tid + i * kWaves * 64;
      const int k = 4 * (u % WU);
      if (NWU % (kWaves * 64) == 0 || u < NWU)
        *reinterpret_cast<u32x4*>(&sW[buf][(u / WU) * WP + k]) = k < p.K ? rw[i] : u32x4{0u, 0u, 0u, 0u};
    }
  };
  gload_w(0);  // in flight during the prologue
  __syncthreads();  // sSrc

  // ---- prologue: row li of this wavefront's 32, lane half lg's k of every group
  float af[4 * G];
  {
    const int src = sSrc[wave * 32 + li];
    const float* arow = p.A + (src >= 0 ? (int64_t)src * p.lda : 0);
    float ss = 0.f;
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const int k = 8 * g + 4 * lg;
      const bool ok = src >= 0 && k < p.K;  // K % 4 == 0: a unit is all in or all out
      floatx4 v = *reinterpret_cast<const floatx4*>(arow + (ok ? k : 0));
      if (!ok) v = floatx4{0.f, 0.f, 0.f, 0.f};
      if constexpr (kNorm) ss += v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
      af[4 * g + 0] = v.x;
      af[4 * g + 1] = v.y;
      af[4 * g + 2] = v.z;
      af[4 * g + 3] = v.w;
    }
    if constexpr (kNorm) {
      ss += __shfl_xor(ss, 32, 64);  // the other half of the row
      if (lg == 0) sR[wave][li] = 1.0f / sqrtf(ss / (float)p.K + p.eps);
    }
  }

  // this panel's rows of C
  const uint32_t panel_bytes = (uint32_t)(min(BM, M - row0) * p.ldc * 4);
  const __amdgpu_buffer_rsrc_t cres = make_rsrc(p.C + (int64_t)row0 * p.ldc, panel_bytes);

  for (int s = 0; s < nsteps; ++s) {
    const int buf = s & 1, n0 = s * 32;
    stage_w(buf);
    __syncthreads();  // W step s (and the row scales) visible; step s-1's reads of this buffer's pair done
    if (s + 1 < nsteps) gload_w(n0 + 32);

    floatx16 acc;
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[r] = 0.f;
    const float* wsrc = &sW[buf][li * WP + 4 * lg];
    // W fragments two groups ahead of their MFMAs
    floatx4 bq[3];
    bq[0] = *reinterpret_cast<const floatx4*>(wsrc);
    if (G > 1) bq[1] = *reinterpret_cast<const floatx4*>(wsrc + 8);
    __builtin_amdgcn_sched_group_barrier(0x0100, G > 1 ? 2 : 1, 0);
#pragma unroll
    for (int g = 0; g < G; ++g) {
      if (g + 2 < G) bq[(g + 2) % 3] = *reinterpret_cast<const floatx4*>(wsrc + 8 * (g + 2));
      const floatx4 b = bq[g % 3];
#pragma unroll
      for (int j = 0; j < 4; ++j) acc = __builtin_amdgcn_mfma_f32_32x32x2f32(af[4 * g + j], b[j], acc, 0, 0, 0);
      if (g + 2 < G) __builtin_amdgcn_sched_group_barrier(0x0100, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x0008, 4, 0);
    }

    // epilogue: lane l holds column l % 32 and rows 8*(r/4) + 4*(l/32) + (r%4)
    const int col = n0 + li;
    const bool cok = col < p.N;
    const float bias = ((FL & kBias) != 0) ? p.bias[cok ? col : 0] : 0.f;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int rl = 8 * (r >> 2) + 4 * lg + (r & 3);
      float v = acc[r];
      if constexpr (kNorm) v *= sR[wave][rl];
      v += bias;
      if (p.relu) v = fmaxf(v, 0.f);
      // rows past M fall outside cres
      const uint32_t off = cok ? (uint32_t)(((wave * 32 + rl) * p.ldc + col) * 4) : kOutOfRange;
      __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, v), cres, off, 0, 0);
    }
  }
}

// The same with 16-row MFMA blocks (v_mfma_f32_16x16x4f32) for K up to 512
// (out_proj): a wavefront holds 16 rows x K of A (K / 4 VGPRs), a workgroup
// 64 rows; W goes through LDS 16 columns at a time; the residual epilogue
// reads C (or R) and adds. Fragment k-order: within each group of 16 k, lane
// quarter q supplies k = 16i + 4q + j in MFMA step 4i + j.
template <int G16, int FL>
__global__ __launch_bounds__(kWaves * 64, 2) void gemm_f32_panel16_kernel(GemmArgs p) {
  constexpr int KP = 16 * G16;       // padded K
  constexpr int WP = KP + 4;         // floats per staged W row
  constexpr int WU = KP / 4;         // 16-byte units per staged W row
  constexpr int NWU = 16 * WU;       // W units per step
  constexpr int NW = (NWU + kWaves * 64 - 1) / (kWaves * 64);
  constexpr int BM16 = kWaves * 16;  // rows per workgroup
  static_assert((FL & (kRowNorm | kGather)) == 0, "16-row panels serve plain, bias and residual GEMMs");

  __shared__ __attribute__((aligned(16))) float sW[2][16 * WP];

  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63;
  const int lr = lane & 15, lq = lane >> 4;
  const int M = p.Mdev ? *p.Mdev : p.Mmax;
  const int row0 = blockIdx.x * BM16;
  if (row0 >= M) return;

  const __amdgpu_buffer_rsrc_t wres = make_rsrc(p.W, (uint32_t)(p.N * p.ldw * 4));
  const int nsteps = (p.N + 15) / 16;
  u32x4 rw[NW];
  auto gload_w = [&](int n0) {
#pragma unroll
    for (int i = 0; i < NW; ++i) {
      const int u = tid + i * kWaves * 64;
      const int n = n0 + u / WU, k = 4 * (u % WU);
      const uint32_t off = u < NWU ? (uint32_t)((n * p.ldw + k) * 4) : kOutOfRange;
      rw[i] = __builtin_amdgcn_raw_buffer_load_b128(wres, off, 0, 0);
    }
  };
  auto stage_w = [&](int buf) {
#pragma unroll
    for (int i = 0; i < NW; ++i) {
      const int u = tid + i * kWaves * 64;
      const int k = 4 * (u % WU);
      if (NWU % (kWaves * 64) == 0 || u < NWU)
        *reinterpret_cast<u32x4*>(&sW[buf][(u / WU) * WP + k]) = k < p.K ? rw[i] : u32x4{0u, 0u, 0u, 0u};
    }
  };
  gload_w(0);

  // prologue: row lr of this wavefront's 16, lane quarter lq's k of every group
  float af[4 * G16];
  {
    const int grow = row0 + wave * 16 + lr;
    const bool rok = grow < M;
    const float* arow = p.A + (rok ? (int64_t)grow * p.lda : 0);
#pragma unroll
    for (int i = 0; i < G16; ++i) {
      const int k = 16 * i + 4 * lq;
      const bool ok = rok && k < p.K;  // K % 4 == 0: a unit is all in or all out
      floatx4 v = *reinterpret_cast<const floatx4*>(arow + (ok ? k : 0));
      if (!ok) v = floatx4{0.f, 0.f, 0.f, 0.f};
      af[4 * i + 0] = v.x;
      af[4 * i + 1] = v.y;
      af[4 * i + 2] = v.z;
      af[4 * i + 3] = v.w;
    }
  }

  // this panel's rows of C and of the residual source
  const uint32_t panel_bytes = (uint32_t)(min(BM16, M - row0) * p.ldc * 4);
  const __amdgpu_buffer_rsrc_t cres = make_rsrc(p.C + (int64_t)row0 * p.ldc, panel_bytes);
  const __amdgpu_buffer_rsrc_t rres =
      make_rsrc((p.R ? p.R : p.C) + (int64_t)row0 * p.ldc, (FL & kResid) != 0 ? panel_bytes : 0);

  for (int s = 0; s < nsteps; ++s) {
    const int buf = s & 1, n0 = s * 16;
    stage_w(buf);
    __syncthreads();  // W step s visible; step s-1's reads of this buffer's pair done
    if (s + 1 < nsteps) gload_w(n0 + 16);

    // the residual of this step's outputs, loaded while the MFMAs run
    const int col = n0 + lr;
    const bool cok = col < p.N;
    float res[4] = {0.f, 0.f, 0.f, 0.f};
    if constexpr ((FL & kResid) != 0) {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const uint32_t off = cok ? (uint32_t)(((wave * 16 + 4 * lq + r) * p.ldc + col) * 4) : kOutOfRange;
        res[r] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rres, off, 0, 0));
      }
    }

    floatx4 acc = floatx4{0.f, 0.f, 0.f, 0.f};
    const float* wsrc = &sW[buf][lr * WP + 4 * lq];
    floatx4 bq[3];
    bq[0] = *reinterpret_cast<const floatx4*>(wsrc);
    if (G16 > 1) bq[1] = *reinterpret_cast<const floatx4*>(wsrc + 16);
    __builtin_amdgcn_sched_group_barrier(0x0100, G16 > 1 ? 2 : 1, 0);
#pragma unroll
    for (int i = 0; i < G16; ++i) {
      if (i + 2 < G16) bq[(i + 2) % 3] = *reinterpret_cast<const floatx4*>(wsrc + 16 * (i + 2));
      const floatx4 b = bq[i % 3];
#pragma unroll
      for (int j = 0; j < 4; ++j) acc = __builtin_amdgcn_mfma_f32_16x16x4f32(af[4 * i + j], b[j], acc, 0, 0, 0);
      if (i + 2 < G16) __builtin_amdgcn_sched_group_barrier(0x0100, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x0008, 4, 0);
    }

    // epilogue: lane l holds column l % 16 and rows 4*(l/16) + r
    const float bias = ((FL & kBias) != 0) ? p.bias[cok ? col : 0] : 0.f;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      float v = acc[r] + bias + res[r];
      if (p.relu) v = fmaxf(v, 0.f);
      const uint32_t off = cok ? (uint32_t)(((wave * 16 + 4 * lq + r) * p.ldc + col) * 4) : kOutOfRange;
      __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, v), cres, off, 0, 0);
    }
  }
}

template <int FL>
hipError_t launch_g16(const GemmArgs& a, hipStream_t s) {
  const int grid = (a.Mmax + kWaves * 16 - 1) / (kWaves * 16);
  if (grid <= 0) return hipSuccess;
  switch ((a.K + 15) / 16) {
    case 16: hipLaunchKernelGGL((gemm_f32_panel16_kernel<16, FL>), dim3(grid), dim3(kWaves * 64), 0, s, a); break;
    case 24: hipLaunchKernelGGL((gemm_f32_panel16_kernel<24, FL>), dim3(grid), dim3(kWaves * 64), 0, s, a); break;
    case 32: hipLaunchKernelGGL((gemm_f32_panel16_kernel<32, FL>), dim3(grid), dim3(kWaves * 64), 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <int FL>
hipError_t launch_g(const GemmArgs& a, hipStream_t s) {
  const int grid = (a.Mmax + BM - 1) / BM;
  if (grid <= 0) return hipSuccess;
  const int g = (a.K + 7) / 8;
#define TCL_PANEL32(GG)                                                                                \
  hipLaunchKernelGGL((gemm_f32_panel_kernel<GG, FL>), dim3(grid), dim3(kWaves * 64), 0, s, a); break
  switch (g) {
    case 8: TCL_PANEL32(8);
    case 16: TCL_PANEL32(16);
    case 21: TCL_PANEL32(21);
    case 24: TCL_PANEL32(24);
    case 32: TCL_PANEL32(32);
    default: return hipErrorInvalidValue;
  }
#undef TCL_PANEL32
  return hipGetLastError();
}

}  // namespace

bool gemm_f32_panel_fits(const GemmArgs& a, int flags) {
  const int g = (a.K + 7) / 8;
  const bool gsup = g == 8 || g == 16 || g == 21 || g == 24 || g == 32;
  return gsup && a.K % 4 == 0 && a.lda % 4 == 0 && reinterpret_cast<uintptr_t>(a.A) % 16 == 0 &&
         (flags & kResid) == 0 && a.R == nullptr &&
         // byte offsets of the buffer resources stay below 2^31
         (int64_t)BM * a.ldc * 4 < (1ll << 31) && (int64_t)(a.N + 32) * a.ldw * 4 < (1ll << 31);
}

bool gemm_f32_panel16_fits(const GemmArgs& a, int flags) {
  const int g = (a.K + 15) / 16;
  return (g == 16 || g == 24 || g == 32) && a.K % 4 == 0 && a.lda % 4 == 0 &&
         reinterpret_cast<uintptr_t>(a.A) % 16 == 0 && (flags & (kRowNorm | kGather)) == 0 &&
         (int64_t)kWaves * 16 * a.ldc * 4 < (1ll << 31) && (int64_t)(a.N + 16) * a.ldw * 4 < (1ll << 31);
}

hipError_t launch_gemm_f32_panel16(const GemmArgs& a, int flags, hipStream_t s) {
  switch (flags) {
    case 0: return launch_g16<0>(a, s);
    case kBias: return launch_g16<kBias>(a, s);
    case kResid: return launch_g16<kResid>(a, s);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_gemm_f32_panel(const GemmArgs& a, int flags, hipStream_t s) {
  switch (flags) {
    case 0: return launch_g<0>(a, s);
    case kBias: return launch_g<kBias>(a, s);
    case kRowNorm: return launch_g<kRowNorm>(a, s);
    case kBias | kGather: return launch_g<kBias | kGather>(a, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace tcl
