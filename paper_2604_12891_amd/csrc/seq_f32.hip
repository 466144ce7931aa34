// Per-program kernels of the fp32 forward: token packing, causal conv +
// SiLU, the selective scan, and the pool + score head.
//
// Tokens are packed program by program: program b owns rows
// offs[b] .. offs[b+1]-1 of every activation. Each kernel here maps one
// thread to one channel of one program and walks that program's tokens in
// order, so the loads of a token row are coalesced across channels and the
// recurrence over t stays in registers.
#include "common.h"
#include "kernels.h"

namespace tcl {
namespace {

// ---------------------------------------------------------------- offsets
// One workgroup of 1024 threads: each thread sums a contiguous slice of the
// lengths, a block-wide exclusive scan gives the slice's start, and the
// slice is written out.
__global__ __launch_bounds__(1024) void offsets_kernel(const int* __restrict__ lengths, int B, int L,
                                                       int* __restrict__ offs) {
  __shared__ int wsum[16];
  const int tid = threadIdx.x;
  const int per = (B + 1023) / 1024;
  const int s = min(tid * per, B), e = min(s + per, B);
  int sum = 0;
  for (int i = s; i < e; ++i) {
    const int len = lengths[i];
    sum += (len >= 1 && len <= L) ? len : 0;
  }
  // inclusive scan within the wavefront
  const int lane = tid & 63, wave = tid >> 6;
  int inc = sum;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int v = __shfl_up(inc, o, 64);
    if (lane >= o) inc += v;
  }
  if (lane == 63) wsum[wave] = inc;
  __syncthreads();
  int before = 0;
  for (int w = 0; w < wave; ++w) before += wsum[w];
  int run = before + inc - sum;
  for (int i = s; i < e; ++i) {
    offs[i] = run;
    const int len = lengths[i];
    run += (len >= 1 && len <= L) ? len : 0;
  }
  if (tid == 1023) offs[B] = before + inc;
}

// ---------------------------------------------------------------- conv + SiLU
// x_{t-K+1..t} of one channel live in a K-register window.
template <int K>
__global__ __launch_bounds__(256) void conv_silu_kernel(const int* __restrict__ offs, int E,
                                                        const float* __restrict__ x, int ldx,
                                                        const float* __restrict__ w,
                                                        const float* __restrict__ bias,
                                                        float* __restrict__ u) {
  const int b = blockIdx.x;
  const int e = blockIdx.y * blockDim.x + threadIdx.x;
  if (e >= E) return;
  const int base = offs[b], len = offs[b + 1] - base;
  float wk[K], win[K];
#pragma unroll
  for (int k = 0; k < K; ++k) {
    wk[k] = w[e * K + k];
    win[k] = 0.f;
  }
  const float be = bias[e];
  for (int t = 0; t < len; ++t) {
    const int64_t row = base + t;
#pragma unroll
    for (int k = 0; k < K - 1; ++k) win[k] = win[k + 1];
    win[K - 1] = x[row * ldx + e];
    float acc = be;
#pragma unroll
    for (int k = 0; k < K; ++k) acc = fmaf(wk[k], win[k], acc);
    u[row * E + e] = silu(acc);
  }
}

// ---------------------------------------------------------------- selective scan
// One thread per (program, channel e). The N states of the channel, its
// N decay rates A*log2(e), and its row of W_dt stay in registers. The
// [dt_r | B | C] rows of the program are staged through LDS TC tokens at
// a time and read as wavefront-wide broadcasts. exp(dt*A) is formed on the
// fly as exp2(dt * A*log2 e); nothing of size [tokens, E, N] is stored.
constexpr int kScanThreads = 128;
constexpr int kScanTC = 32;

template <int N, int R>
__global__ __launch_bounds__(kScanThreads) void scan_kernel(
    const int* __restrict__ offs, int E, const float* u, const float* __restrict__ xdbl,
    const float* __restrict__ z, int ldz, const float* __restrict__ W_dt,
    const float* __restrict__ b_dt, const float* __restrict__ A_log,
    const float* __restrict__ Dp, float* out) {
  constexpr int XW = R + 2 * N;
  __shared__ __attribute__((aligned(16))) float sX[kScanTC * XW];
  const int b = blockIdx.x;
  const int e = blockIdx.y * kScanThreads + threadIdx.x;
  const bool active = e < E;
  const int ec = active ? e : 0;
  const int base = offs[b], len = offs[b + 1] - base;

  float a2[N], s[N], wdt[R];
#pragma unroll
  for (int n = 0; n < N; ++n) {
    a2[n] = -expf(A_log[ec * N + n]) * kLog2e;
    s[n] = 0.f;
  }
#pragma unroll
  for (int r = 0; r < R; ++r) wdt[r] = W_dt[ec * R + r];
  const float bdt = b_dt[ec], Dv = Dp[ec];

  for (int t0 = 0; t0 < len; t0 += kScanTC) {
    const int nt = min(kScanTC, len - t0);
    __syncthreads();
    const float* src = xdbl + (int64_t)(base + t0) * XW;
    for (int i = threadIdx.x; i < nt * XW; i += kScanThreads) sX[i] = src[i];
    __syncthreads();
    if (!active) continue;
    for (int tt = 0; tt < nt; ++tt) {
      const int64_t row = base + t0 + tt;
      const float* xr = &sX[tt * XW];
      const float uv = u[row * E + e];
      const float zv = z[row * ldz + e];
      float v = bdt;
#pragma unroll
      for (int r = 0; r < R; ++r) v = fmaf(wdt[r], xr[r], v);
      const float dt = softplus(v);
      const float dtu = dt * uv;
      float y = 0.f;
#pragma unroll
      for (int n = 0; n < N; ++n) {
        const float a = __builtin_amdgcn_exp2f(dt * a2[n]);
        s[n] = fmaf(a, s[n], dtu * xr[R + n]);
        y = fmaf(s[n], xr[R + N + n], y);
      }
      y = fmaf(Dv, uv, y);
      out[row * E + e] = y * silu(zv);
    }
  }
}

// ---------------------------------------------------------------- tail
// PB programs per workgroup. Phase 1: each wavefront pools whole programs
// (per token: RMSNorm statistics by a wavefront reduction, then accumulate
// the normalised row). Phase 2: thread j computes hidden unit j of the head
// for all PB programs (W1 is read once per workgroup, transposed so the
// reads are coalesced), then the ReLU'd units are dotted with W2 by a
// block reduction.
constexpr int kTailPB = 16;

template <int DM>
__global__ __launch_bounds__(256) void tail_kernel(int B, int L, int h, const int* __restrict__ offs,
                                                   const int* __restrict__ lengths,
                                                   const float* __restrict__ H,
                                                   const float* __restrict__ g_f, int final_norm,
                                                   float eps, const float* __restrict__ W1T,
                                                   const float* __restrict__ b1,
                                                   const float* __restrict__ W2,
                                                   const float* __restrict__ b2,
                                                   float* __restrict__ scores) {
  constexpr int PL = DM / 64;  // values per lane
  __shared__ float sP[DM][kTailPB];
  __shared__ float sRed[4][kTailPB];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int b0 = blockIdx.x * kTailPB;

  for (int p = wave; p < kTailPB; p += 4) {
    const int b = b0 + p;
    float acc[PL];
#pragma unroll
    for (int i = 0; i < PL; ++i) acc[i] = 0.f;
    int len = 0;
    if (b < B) {
      const int base = offs[b];
      len = offs[b + 1] - base;
      for (int t = 0; t < len; ++t) {
        const float* hr = H + (int64_t)(base + t) * DM + lane * PL;
        float v[PL];
#pragma unroll
        for (int i = 0; i < PL; ++i) v[i] = hr[i];
        float rs = 1.f;
        if (final_norm) {
          float ss = 0.f;
#pragma unroll
          for (int i = 0; i < PL; ++i) ss = fmaf(v[i], v[i], ss);
          ss = wave_sum(ss);
          rs = 1.0f / sqrtf(ss / (float)DM + eps);
        }
#pragma unroll
        for (int i = 0; i < PL; ++i) acc[i] = fmaf(v[i], rs, acc[i]);
      }
    }
    const float inv = len > 0 ? 1.0f / (float)len : 0.f;
#pragma unroll
    for (int i = 0; i < PL; ++i) {
      const int k = lane * PL + i;
      const float g = final_norm ? g_f[k] : 1.f;
      sP[k][p] = acc[i] * g * inv;
    }
  }
  __syncthreads();

  float part[kTailPB];
#pragma unroll
  for (int p = 0; p < kTailPB; ++p) part[p] = 0.f;
  if (tid < h) {
    float a[kTailPB];
    const float bj = b1[tid];
#pragma unroll
    for (int p = 0; p < kTailPB; ++p) a[p] = bj;
    for (int k = 0; k < DM; ++k) {
      const float wv = W1T[k * h + tid];
#pragma unroll
      for (int p = 0; p < kTailPB; ++p) a[p] = fmaf(wv, sP[k][p], a[p]);
    }
    const float w2 = W2[tid];
#pragma unroll
    for (int p = 0; p < kTailPB; ++p) part[p] = w2 * fmaxf(a[p], 0.f);
  }
#pragma unroll
  for (int p = 0; p < kTailPB; ++p) {
    const float v = wave_sum(part[p]);
    if (lane == 0) sRed[wave][p] = v;
  }
  __syncthreads();
  if (tid < kTailPB) {
    const int b = b0 + tid;
    if (b < B) {
      const float sc = sRed[0][tid] + sRed[1][tid] + sRed[2][tid] + sRed[3][tid] + b2[0];
      const int len = lengths[b];
      scores[b] = (len >= 1 && len <= L) ? sc : __builtin_nanf("");
    }
  }
}

}  // namespace

hipError_t launch_offsets(const int* lengths, int B, int L, int* offs, hipStream_t s) {
  hipLaunchKernelGGL(offsets_kernel, dim3(1), dim3(1024), 0, s, lengths, B, L, offs);
  return hipGetLastError();
}

hipError_t launch_conv_silu_f32(int B, int E, int K, const int* offs, const float* x, int ldx,
                                const float* w, const float* b, float* u, hipStream_t s) {
  if (B <= 0) return hipSuccess;
  dim3 grid(B, (E + 255) / 256);
  switch (K) {
    case 1: hipLaunchKernelGGL(conv_silu_kernel<1>, grid, dim3(256), 0, s, offs, E, x, ldx, w, b, u); break;
    case 2: hipLaunchKernelGGL(conv_silu_kernel<2>, grid, dim3(256), 0, s, offs, E, x, ldx, w, b, u); break;
    case 3: hipLaunchKernelGGL(conv_silu_kernel<3>, grid, dim3(256), 0, s, offs, E, x, ldx, w, b, u); break;
    case 4: hipLaunchKernelGGL(conv_silu_kernel<4>, grid, dim3(256), 0, s, offs, E, x, ldx, w, b, u); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_scan_f32(int B, int E, int N, int R, const int* offs, const float* u,
                           const float* xdbl, const float* z, int ldz, const float* W_dt,
                           const float* b_dt, const float* A_log, const float* D, float* out,
                           hipStream_t s) {
  if (B <= 0) return hipSuccess;
  if (N != 16) return hipErrorInvalidValue;
  dim3 grid(B, (E + kScanThreads - 1) / kScanThreads);
#define TCL_SCAN(RR)                                                                              \
  hipLaunchKernelGGL((scan_kernel<16, RR>), grid, dim3(kScanThreads), 0, s, offs, E, u, xdbl, z, \
                     ldz, W_dt, b_dt, A_log, D, out)
  switch (R) {
    case 4: TCL_SCAN(4); break;
    case 8: TCL_SCAN(8); break;
    case 12: TCL_SCAN(12); break;
    case 16: TCL_SCAN(16); break;
    case 20: TCL_SCAN(20); break;
    case 24: TCL_SCAN(24); break;
    case 28: TCL_SCAN(28); break;
    case 32: TCL_SCAN(32); break;
    default: return hipErrorInvalidValue;
  }
#undef TCL_SCAN
  return hipGetLastError();
}

hipError_t launch_tail_f32(int B, int L, int d, int h, const int* offs, const int* lengths,
                           const float* H, const float* g_f, int final_norm, float eps,
                           const float* W1T, const float* b1, const float* W2, const float* b2,
                           float* scores, hipStream_t s) {
  if (B <= 0) return hipSuccess;
  if (h > 256) return hipErrorInvalidValue;
  dim3 grid((B + kTailPB - 1) / kTailPB);
#define TCL_TAIL(DD)                                                                          \
  hipLaunchKernelGGL((tail_kernel<DD>), grid, dim3(256), 0, s, B, L, h, offs, lengths, H, g_f, \
                     final_norm, eps, W1T, b1, W2, b2, scores)
  switch (d) {
    case 64: TCL_TAIL(64); break;
    case 128: TCL_TAIL(128); break;
    case 256: TCL_TAIL(256); break;
    default: return hipErrorInvalidValue;
  }
#undef TCL_TAIL
  return hipGetLastError();
}

}  // namespace tcl
