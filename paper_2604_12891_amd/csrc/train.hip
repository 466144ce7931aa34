// Kernels of the teacher -> student distillation step (forward with saved
// activations, backward, Adam, weight refresh). Reverse-mode derivatives of
// the model that the scoring kernels compute; tokens are packed program by
// program as everywhere else, and every reduction over tokens or programs
// goes through per-block partials summed in a fixed order (deterministic).
#include "common.h"
#include "kernels.h"

namespace tcl {
namespace {

__device__ __forceinline__ float sigmoid_fast(float x) { return rcp_fast(1.0f + exp_fast(-x)); }

// d/dx SiLU(x) = s (1 + x (1 - s)), s = sigmoid(x)
__device__ __forceinline__ float silu_grad(float x) {
  const float s = sigmoid_fast(x);
  return s * (1.0f + x * (1.0f - s));
}

__device__ __forceinline__ float ld_act(const float* p) { return *p; }
__device__ __forceinline__ float ld_act(const uint16_t* p) { return bf16_to_f32(*p); }
// an activation held as loaded (bf16 in the low half of a 32-bit register)
// and widened to fp32 at use
template <typename T> using act_raw_t = std::conditional_t<sizeof(T) == 2, uint32_t, float>;
__device__ __forceinline__ float act_f32(float v) { return v; }
__device__ __forceinline__ float act_f32(uint32_t v) { return __uint_as_float(v << 16); }
__device__ __forceinline__ float to_f32(float v) { return v; }
__device__ __forceinline__ float to_f32(uint16_t v) { return bf16_to_f32(v); }

// ---------------------------------------------------------------- RMSNorm forward
// One wavefront per token row: n = bf16(h * r * g), r = (mean h^2 + eps)^-1/2.
template <int DM>
__global__ __launch_bounds__(256) void rmsnorm_fwd_kernel(const int* __restrict__ Mdev,
                                                          const float* __restrict__ H,
                                                          const float* __restrict__ g, float eps,
                                                          uint16_t* __restrict__ n,
                                                          float* __restrict__ rstd) {
  constexpr int PL = DM / 64;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= *Mdev) return;
  const float* hr = H + (int64_t)row * DM + lane * PL;
  float v[PL], ss = 0.f;
#pragma unroll
  for (int i = 0; i < PL; ++i) {
    v[i] = hr[i];
    ss = fmaf(v[i], v[i], ss);
  }
  ss = wave_sum(ss);
  const float r = 1.0f / sqrtf(ss / (float)DM + eps);
#pragma unroll
  for (int i = 0; i < PL; ++i) n[(int64_t)row * DM + lane * PL + i] = f32_to_bf16(v[i] * r * g[lane * PL + i]);
  if (lane == 0) rstd[row] = r;
}

// ---------------------------------------------------------------- RMSNorm backward
// dH[row] += r (g dN) - (r^3 / d) h sum(g dN h); per-block partial of
// dg = sum over rows of dN h r. kRnWaves wavefronts per block, each taking
// every kRnWaves-th row of the block's range.
constexpr int kRnWaves = 16;
template <int DM>
__global__ __launch_bounds__(64 * kRnWaves) void rmsnorm_bwd_kernel(const int* __restrict__ Mdev,
                                                          const float* __restrict__ dN,
                                                          const float* __restrict__ H,
                                                          const float* __restrict__ rstd,
                                                          const float* __restrict__ g,
                                                          float* __restrict__ dH,
                                                          float* __restrict__ dg_part,
                                                          int rows_per_block) {
  constexpr int PL = DM / 64;
  __shared__ float sdg[kRnWaves][DM];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int M = *Mdev;
  float dg[PL];
#pragma unroll
  for (int i = 0; i < PL; ++i) dg[i] = 0.f;
  const int r0 = blockIdx.x * rows_per_block;
  const int r1 = min(r0 + rows_per_block, M);
  // rows of this wavefront in groups of U: the group's loads are issued
  // together (one memory latency per group instead of one per row); a row
  // past the block's range re-reads row r0 and is skipped at use
  constexpr int U = 4;
  float gl[PL];
#pragma unroll
  for (int i = 0; i < PL; ++i) gl[i] = g[lane * PL + i];
  for (int rw = r0 + wave; rw < r1; rw += kRnWaves * U) {
    float h[U][PL], dn[U][PL], dh[U][PL], r[U];
#pragma unroll
    for (int j = 0; j < U; ++j) {
      const int row = rw + kRnWaves * j < r1 ? rw + kRnWaves * j : r0;
      const int64_t o = (int64_t)row * DM + lane * PL;
      r[j] = rstd[row];
#pragma unroll
      for (int i = 0; i < PL; ++i) {
        h[j][i] = H[o + i];
        dn[j][i] = dN[o + i];
        dh[j][i] = dH[o + i];
      }
    }
    // every row of the group is computed (so the loads above stay where
    // they are: a per-row branch would let the compiler sink each row's
    // loads to its use); rows past the range are neither stored nor summed
#pragma unroll
    for (int j = 0; j < U; ++j) {
      const int row = rw + kRnWaves * j;
      const bool ok = row < r1;  // wave-uniform
      const int64_t o = (int64_t)row * DM + lane * PL;
      float gd[PL], dot = 0.f;
#pragma unroll
      for (int i = 0; i < PL; ++i) {
        gd[i] = dn[j][i] * gl[i];
        dot = fmaf(gd[i], h[j][i], dot);
        const float dgi = fmaf(dn[j][i], h[j][i] * r[j], dg[i]);
        dg[i] = ok ? dgi : dg[i];
      }
      dot = wave_sum(dot);
      const float c = r[j] * r[j] * r[j] / (float)DM * dot;
      if (ok) {
#pragma unroll
        for (int i = 0; i < PL; ++i) dH[o + i] = dh[j][i] + (r[j] * gd[i] - c * h[j][i]);
      }
    }
  }
#pragma unroll
  for (int i = 0; i < PL; ++i) sdg[wave][lane * PL + i] = dg[i];
  __syncthreads();
  for (int k = threadIdx.x; k < DM; k += 64 * kRnWaves) {
    float t = 0.f;
#pragma unroll
    for (int w = 0; w < kRnWaves; ++w) t += sdg[w][k];
    dg_part[(int64_t)blockIdx.x * DM + k] = t;
  }
}

// ---------------------------------------------------------------- loss + head backward
// 16 programs per block. For program b: ds = (2/B)(2 s - t - y),
// da1 = ds W2 (a1 > 0), dpooled = da1 W1. Per-block partials of
// [dW2 (h) | db1 (h) | db2 | sum (s-t)^2 | sum (s-y)^2].
constexpr int kHB = 16;
__global__ __launch_bounds__(256) void loss_head_bwd_kernel(
    int B, int d, int h, const float* __restrict__ s, const float* __restrict__ t,
    const float* __restrict__ y, const float* __restrict__ a1, const float* __restrict__ W1,
    const float* __restrict__ W2, float* __restrict__ da1, float* __restrict__ dpooled,
    float* __restrict__ part, const float* __restrict__ ds_in, const float* __restrict__ loss_in) {
  __shared__ float sda[kHB][256];
  __shared__ float sds[kHB];
  const int tid = threadIdx.x;
  const int b0 = blockIdx.x * kHB;
  const float inv = 2.0f / (float)B;
  if (tid < kHB) {
    const int b = b0 + tid;
    sds[tid] = b >= B ? 0.f : ds_in ? ds_in[b] : inv * (2.0f * s[b] - t[b] - y[b]);
  }
  __syncthreads();
  float pw2 = 0.f, pb1 = 0.f;
  if (tid < h) {
    const float w2 = W2[tid];
    float av[kHB];  // every program's activation loaded up front (one latency)
#pragma unroll
    for (int p = 0; p < kHB; ++p) av[p] = b0 + p < B ? a1[(int64_t)(b0 + p) * h + tid] : 0.f;
#pragma unroll
    for (int p = 0; p < kHB; ++p) {
      const int b = b0 + p;
      float g = 0.f;
      if (b < B) {
        const float a = av[p];
        g = a > 0.f ? sds[p] * w2 : 0.f;
        pw2 = fmaf(sds[p], fmaxf(a, 0.f), pw2);
        da1[(int64_t)b * h + tid] = g;
      }
      sda[p][tid] = g;
      pb1 += g;
    }
  }
  __syncthreads();
  if (tid < d) {
    float acc[kHB];
#pragma unroll
    for (int p = 0; p < kHB; ++p) acc[p] = 0.f;
    // 32 rows of W1 loaded together per batch (h is a multiple of 64): one
    // memory latency per batch
    for (int j0 = 0; j0 < h; j0 += 32) {
      float w[32];
#pragma unroll
      for (int jj = 0; jj < 32; ++jj) w[jj] = W1[(int64_t)(j0 + jj) * d + tid];
      __builtin_amdgcn_sched_barrier(0);  // every load of the batch before its first use
#pragma unroll
      for (int jj = 0; jj < 32; ++jj)
#pragma unroll
        for (int p = 0; p < kHB; ++p) acc[p] = fmaf(sda[p][j0 + jj], w[jj], acc[p]);
    }
#pragma unroll
    for (int p = 0; p < kHB; ++p)
      if (b0 + p < B) dpooled[(int64_t)(b0 + p) * d + tid] = acc[p];
  }
  const int W = 2 * h + 4;
  float* out = part + (int64_t)blockIdx.x * W;
  if (tid < h) {
    out[tid] = pw2;
    out[h + tid] = pb1;
  }
  if (tid == 0) {
    float db2 = 0.f, lt = 0.f, ly = 0.f;
    for (int p = 0; p < kHB; ++p) {
      const int b = b0 + p;
      if (b >= B) break;
      db2 += sds[p];
      lt += (s[b] - t[b]) * (s[b] - t[b]);
      ly += (s[b] - y[b]) * (s[b] - y[b]);
    }
    const float invB = 1.0f / (float)B;
    out[2 * h] = db2;
    if (ds_in) {
      // the loss was computed with the gradient: block 0 carries it, the
      // others add zero, so the reduction reproduces it exactly
      const bool first = blockIdx.x == 0;
      out[2 * h + 1] = first ? loss_in[1] : 0.f;
      out[2 * h + 2] = first ? loss_in[2] : 0.f;
      out[2 * h + 3] = first ? loss_in[0] : 0.f;
    } else {
      out[2 * h + 1] = lt * invB;
      out[2 * h + 2] = ly * invB;
      out[2 * h + 3] = (lt + ly) * invB;
    }
  }
}

// ---------------------------------------------------------------- final norm + pool backward
// Block per program; wavefronts take its tokens. dhf = dpooled[b] / len for
// every valid token; dH = RMSNorm_f backward of dhf (or dhf itself without
// the final norm). Per-program partial of dg_f.
template <int DM>
__global__ __launch_bounds__(256) void normf_pool_bwd_kernel(const int* __restrict__ offs,
                                                             const float* __restrict__ H,
                                                             const float* __restrict__ g_f,
                                                             int final_norm, float eps,
                                                             const float* __restrict__ dpooled,
                                                             float* __restrict__ dH,
                                                             float* __restrict__ dg_part) {
  constexpr int PL = DM / 64;
  __shared__ float sdg[4][DM];
  const int b = blockIdx.x;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int base = offs[b], len = offs[b + 1] - base;
  const float inv = len > 0 ? 1.0f / (float)len : 0.f;
  float dhf[PL], gg[PL], dg[PL];
#pragma unroll
  for (int i = 0; i < PL; ++i) {
    dhf[i] = dpooled[(int64_t)b * DM + lane * PL + i] * inv;
    gg[i] = final_norm ? g_f[lane * PL + i] : 1.f;
    dg[i] = 0.f;
  }
  if (!final_norm) {
    for (int t = wave; t < len; t += 4) {
      const int64_t o = (int64_t)(base + t) * DM + lane * PL;
#pragma unroll
      for (int i = 0; i < PL; ++i) dH[o + i] = dhf[i];
    }
  } else {
    // this wavefront's tokens in groups of U whose rows are loaded together
    // (a token past the end re-reads the first row and is skipped)
    constexpr int U = 4;
    for (int t0 = wave; t0 < len; t0 += 4 * U) {
      float hv[U][PL];
#pragma unroll
      for (int j = 0; j < U; ++j) {
        const int t = t0 + 4 * j < len ? t0 + 4 * j : 0;
        const int64_t o = (int64_t)(base + t) * DM + lane * PL;
#pragma unroll
        for (int i = 0; i < PL; ++i) hv[j][i] = H[o + i];
      }
      // every token of the group is computed (a per-token branch would let
      // the compiler sink each token's loads to its use); tokens past the
      // end are neither stored nor summed
#pragma unroll
      for (int j = 0; j < U; ++j) {
        const int t = t0 + 4 * j;
        const bool ok = t < len;  // wave-uniform
        const int64_t o = (int64_t)(base + t) * DM + lane * PL;
        float ss = 0.f, dot = 0.f;
#pragma unroll
        for (int i = 0; i < PL; ++i) {
          ss = fmaf(hv[j][i], hv[j][i], ss);
          dot = fmaf(gg[i] * dhf[i], hv[j][i], dot);
        }
        ss = wave_sum(ss);
        dot = wave_sum(dot);
        const float r = 1.0f / sqrtf(ss / (float)DM + eps);
        const float c = r * r * r / (float)DM * dot;
#pragma unroll
        for (int i = 0; i < PL; ++i) {
          if (ok) dH[o + i] = r * gg[i] * dhf[i] - c * hv[j][i];
          const float dgi = fmaf(dhf[i], hv[j][i] * r, dg[i]);
          dg[i] = ok ? dgi : dg[i];
        }
      }
    }
  }
#pragma unroll
  for (int i = 0; i < PL; ++i) sdg[wave][lane * PL + i] = dg[i];
  __syncthreads();
  for (int k = threadIdx.x; k < DM; k += 256)
    dg_part[(int64_t)b * DM + k] = sdg[0][k] + sdg[1][k] + sdg[2][k] + sdg[3][k];
}

// ---------------------------------------------------------------- selective-scan backward
// Block per program, two lanes per channel e: lane 2e+h owns states
// n = 8h .. 8h+7 (sums over n are completed with one lane-pair shuffle).
// Per channel:
//   the state every TC tokens comes from the forward scan, which stored it
//   (launch_scan's checkpoints, one [N] vector per chunk boundary; the
//   recurrence below is the forward kernel's, operation for operation, so
//   the recomputed states are the same bits);
//   reverse sweep chunk by chunk: the chunk's states are recomputed into
//   registers from its checkpoint, then tokens are walked backwards with the
//   state adjoint g_t = C_t dy_t + a_{t+1} g_{t+1}, a_t = exp(dt_t A).
// Per token it writes dz (gate), du (scan part), dv = ddt * softplus'(v);
// dB_t and dC_t are sums over channels, formed by a butterfly reduce-scatter
// over the same-parity lanes of each wavefront, parked in LDS per token and
// summed across wavefronts once at the end (no barrier inside the sweep).
// dA_log and dD are accumulated per lane and written as per-program partials.
constexpr int kTC = kScanCkptTokens;
constexpr int kHalfN = 8;

// Reduce 16 values across the 32 same-parity lanes of a wavefront: lane l
// ends with the total (over lanes of parity l & 1) of value ((l >> 2) & 15).
// A reduce-scatter over lane bits 5, 4, 3, 2, then a plain sum over bit 1.
// The bit-5 and bit-4 steps use gfx950's half-wave / row swaps, which route
// both values of a pair at once (no per-lane select); bit 3 is a DPP row
// rotate by 8 (= xor 8 inside a row of 16), bit 2 a swizzle (xor 4), bit 1 a
// DPP quad permutation. Every lane of the wavefront must be active.
__device__ __forceinline__ float dpp_xor1(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0xB1, 0xF, 0xF, false));  // quad_perm [1,0,3,2]
}
__device__ __forceinline__ float butterfly16(float* v, int lane) {
  float w[8], x[4];
#pragma unroll
  for (int i = 0; i < 8; ++i) {  // lanes 0-31 keep v[i], 32-63 keep v[8 + i]
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v[i]), __float_as_uint(v[8 + i]), false, false);
    w[i] = __uint_as_float(r[0]) + __uint_as_float(r[1]);
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {  // rows 0, 2 keep w[i], rows 1, 3 keep w[4 + i]
    const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(w[i]), __float_as_uint(w[4 + i]), false, false);
    x[i] = __uint_as_float(r[0]) + __uint_as_float(r[1]);
  }
  const bool b3 = (lane & 8) != 0, b2 = (lane & 4) != 0;
  float y[2];
#pragma unroll
  for (int i = 0; i < 2; ++i) {  // bit 3: row_ror:8
    const float mine = b3 ? x[2 + i] : x[i], other = b3 ? x[i] : x[2 + i];
    y[i] = mine + __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(other), 0x128, 0xF, 0xF, false));
  }
  const float mine = b2 ? y[1] : y[0], other = b2 ? y[0] : y[1];
  const float z = mine + __int_as_float(__builtin_amdgcn_ds_swizzle(__float_as_int(other), 0x101F));  // xor 4
  return z + __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(z), 0x4E, 0xF, 0xF, false));  // xor 2
}

template <int N, int R, typename T>
__global__ __launch_bounds__(512, 2) void scan_bwd_kernel(
    const int* __restrict__ offs, int E, int L, const T* __restrict__ u,
    const float* __restrict__ xdbl, const T* __restrict__ xz, const T* __restrict__ ysave,
    const float* __restrict__ dyg, const float* __restrict__ W_dt,
    const float* __restrict__ b_dt, const float* __restrict__ A_log, const float* __restrict__ Dp,
    const float* __restrict__ ckpt, float* __restrict__ dv_out, float* __restrict__ du_out,
    float* __restrict__ dxz, float* __restrict__ dxdbl, float* __restrict__ dA_part,
    float* __restrict__ dD_part, float* __restrict__ dbc_part, int Mmax, int TW, const int* __restrict__ ord) {
  static_assert(N == 2 * kHalfN, "two lanes per channel, eight states each");
  constexpr int XW = R + 2 * N;
  constexpr int NH = kHalfN;
  extern __shared__ float smem[];
  // a window of TW tokens (a multiple of the checkpoint interval) at a time
  float* sX = smem;                       // [TW][XW] the window's rows
  float* sRed = smem + TW * XW;           // [TW][8 waves][2N] per-wavefront dB_t | dC_t
  const int b = ord ? ord[blockIdx.x] : (int)blockIdx.x;  // longest programs first when ordered
  const int tid = threadIdx.x;            // blockDim == 2E / gridDim.y: the program's channels in groups
  const int e = blockIdx.y * (blockDim.x >> 1) + (tid >> 1), hf = tid & 1, n0 = hf * NH;
  const int wave = tid >> 6, lane = tid & 63;
  const int base = offs[b], len = offs[b + 1] - base;
  const int nck = (len + kTC - 1) / kTC;
  const int ldz = 2 * E;

  int wbase = 0, wend = 0;  // the staged window [wbase, wend)
  auto stage_window = [&](int w0) {
    wbase = w0;
    wend = min(w0 + TW, len);
    __syncthreads();  // every wavefront is done with the previous window's rows
    for (int i = tid; i < (wend - wbase) * XW; i += blockDim.x) sX[i] = xdbl[(int64_t)(base + wbase) * XW + i];
    __syncthreads();
  };
  const int nw = blockDim.x >> 6;
  // dB_t, dC_t of the window's tokens = sums over the block's wavefronts
  auto flush_window = [&]() {
    __syncthreads();
    for (int i = tid; i < (wend - wbase) * 2 * N; i += blockDim.x) {
      const int tl = i / (2 * N), j = i % (2 * N), t = wbase + tl;
      float acc = 0.f;
      for (int w = 0; w < nw; ++w) acc += sRed[(tl * 8 + w) * 2 * N + j];
      if (gridDim.y == 1) dxdbl[(int64_t)(base + t) * XW + R + j] = acc;
      else dbc_part[((int64_t)blockIdx.y * Mmax + base + t) * 2 * N + j] = acc;
    }
  };

  float a2[NH], wdt[R];  // a2 = A log2(e); A itself is a2 ln(2) where needed
#pragma unroll
  for (int n = 0; n < NH; ++n) a2[n] = -__builtin_amdgcn_exp2f(A_log[e * N + n0 + n] * kLog2e) * kLog2e;
#pragma unroll
  for (int r = 0; r < R; ++r) wdt[r] = W_dt[e * R + r];
  const float bdt = b_dt[e], Dv = Dp[e];
  const float* ck = ckpt + ((int64_t)b * E + e) * (int64_t)((L + kTC - 1) / kTC) * N + n0;

  auto dt_of = [&](int t, float& sig) {
    const float* xr = &sX[(t - wbase) * XW];
    float v = bdt;
#pragma unroll
    for (int r = 0; r < R; ++r) v = fmaf(wdt[r], xr[r], v);
    sig = sigmoid_fast(v);
    return softplus(v);
  };

  float g[NH], anext[NH], dA[NH];
#pragma unroll
  for (int n = 0; n < NH; ++n) {
    g[n] = 0.f;
    anext[n] = 0.f;
    dA[n] = 0.f;
  }
  float dD = 0.f;

  // a chunk's per-token inputs and starting state are loaded (raw) one chunk
  // ahead, while the previous chunk is computed
  T ur[kTC], zr[kTC], yr[kTC];
  float gr[kTC], spr[NH];
  auto load_chunk = [&](int c) {
#pragma unroll
    for (int tt = 0; tt < kTC; ++tt) {
      const int t = min(c * kTC + tt, len - 1);
      const int64_t row = base + t;
      ur[tt] = u[row * E + e];
      zr[tt] = xz[row * ldz + E + e];
      yr[tt] = ysave[row * E + e];
      gr[tt] = dyg[row * E + e];
    }
#pragma unroll
    for (int n = 0; n < NH; ++n) spr[n] = c > 0 ? ck[(c - 1) * N + n] : 0.f;
  };
  if (nck > 0) load_chunk(nck - 1);
  for (int c = nck - 1; c >= 0; --c) {
    const int t0 = c * kTC;
    // windows begin at multiples of TW (a multiple of kTC): a chunk never
    // straddles two; entering a new window flushes the one after it
    if (c == nck - 1 || t0 < wbase) {
      if (c != nck - 1) flush_window();
      stage_window(t0 / TW * TW);
    }
    float sp[NH];  // state before the chunk
    float uc[kTC], zc[kTC], yc[kTC], gc[kTC];
#pragma unroll
    for (int n = 0; n < NH; ++n) sp[n] = spr[n];
#pragma unroll
    for (int tt = 0; tt < kTC; ++tt) {
      uc[tt] = to_f32(ur[tt]);
      zc[tt] = to_f32(zr[tt]);
      yc[tt] = to_f32(yr[tt]);
      gc[tt] = gr[tt];
    }
    if (c > 0) load_chunk(c - 1);
    float hist[kTC][NH];
    {
      float s[NH];
#pragma unroll
      for (int n = 0; n < NH; ++n) s[n] = sp[n];
#pragma unroll
      for (int tt = 0; tt < kTC; ++tt) {
        const int t = t0 + tt;
        if (t < len) {
          float sig;
          const float dt = dt_of(t, sig);
          const float dtu = dt * uc[tt];
          const float* xr = &sX[(t - wbase) * XW] + R + n0;
#pragma unroll
          for (int n = 0; n < NH; ++n) s[n] = fmaf(__builtin_amdgcn_exp2f(dt * a2[n]), s[n], dtu * xr[n]);
        }
#pragma unroll
        for (int n = 0; n < NH; ++n) hist[tt][n] = s[n];
      }
    }
#pragma unroll
    for (int tt = kTC - 1; tt >= 0; --tt) {
      const int t = t0 + tt;
      if (t < len) {  // uniform across the block: len is per program
        const int64_t row = base + t;
        const float* xB = &sX[(t - wbase) * XW] + R + n0;
        const float* xC = &sX[(t - wbase) * XW] + R + N + n0;
        float sig;
        const float dt = dt_of(t, sig);
        const float uv = uc[tt], zv = zc[tt];
        const float dy = gc[tt] * silu(zv);
        float red[2 * NH];
        float gB = 0.f, ddt_a = 0.f;
#pragma unroll
        for (int n = 0; n < NH; ++n) {
          const float a = __builtin_amdgcn_exp2f(dt * a2[n]);
          g[n] = fmaf(xC[n], dy, anext[n] * g[n]);
          anext[n] = a;
          const float sprev = tt > 0 ? hist[tt - 1][n] : sp[n];
          const float gsa = g[n] * sprev * a;
          gB = fmaf(g[n], xB[n], gB);
          ddt_a = fmaf(gsa, a2[n], ddt_a);  // scaled by ln 2 below
          dA[n] = fmaf(gsa, dt, dA[n]);
          red[n] = g[n] * dt * uv;          // dB_t[n0 + n] contribution
          red[NH + n] = dy * hist[tt][n];   // dC_t[n0 + n] contribution
        }
        gB += dpp_xor1(gB);
        ddt_a += dpp_xor1(ddt_a);
        if (hf == 0) {
          dD = fmaf(dy, uv, dD);
          dxz[row * ldz + E + e] = gc[tt] * yc[tt] * silu_grad(zv);
          du_out[row * E + e] = fmaf(Dv, dy, dt * gB);
          dv_out[row * E + e] = fmaf(ddt_a, kLn2, uv * gB) * sig;
        }
        const float tot = butterfly16(red, lane);
        if ((lane & 2) == 0) {
          const int k = (lane >> 2) & 15;
          const int j = k < NH ? n0 + k : N + n0 + (k - NH);
          sRed[((t - wbase) * 8 + wave) * 2 * N + j] = tot;
        }
      }
    }
  }
  if (nck > 0) flush_window();
#pragma unroll
  for (int n = 0; n < NH; ++n)
    dA_part[((int64_t)b * E + e) * N + n0 + n] = dA[n] * (a2[n] * kLn2);  // d/dA_log
  if (hf == 0) dD_part[(int64_t)b * E + e] = dD;
}

// ---------------------------------------------------------------- conv + SiLU backward
// Thread per (program, channel), tokens walked backwards. xc is recomputed
// from the x window; dx_t = sum_k w_k dxc_{t+K-1-k} uses a window of future
// dxc. Per-program partials of dw (K values) and db.
template <int K, typename T>
__global__ __launch_bounds__(256) void conv_bwd_kernel(const int* __restrict__ offs, int E,
                                                       const T* __restrict__ x, int ldx,
                                                       const float* __restrict__ w,
                                                       const float* __restrict__ bias,
                                                       const float* __restrict__ du,
                                                       float* __restrict__ dx, int lddx,
                                                       float* __restrict__ part) {
  const int b = blockIdx.x;
  const int e = blockIdx.y * blockDim.x + threadIdx.x;
  if (e >= E) return;
  const int base = offs[b], len = offs[b + 1] - base;
  float wk[K], xw[K], fut[K], dw[K];
#pragma unroll
  for (int k = 0; k < K; ++k) {
    wk[k] = w[e * K + k];
    fut[k] = 0.f;
    dw[k] = 0.f;
  }
  // xw[k] = x_{t-K+1+k} for the current t (zero before the program start)
  act_raw_t<T> xr[K];  // (an empty program reads row 0 and uses none of it)
#pragma unroll
  for (int k = 0; k < K; ++k) xr[k] = x[(int64_t)(len > 0 ? base + max(len - K + k, 0) : 0) * ldx + e];
#pragma unroll
  for (int k = 0; k < K; ++k) xw[k] = len - K + k >= 0 ? act_f32(xr[k]) : 0.f;
  const float be = bias[e];
  float db = 0.f;
  // tokens in groups of U, walked backwards; the next group's du and x
  // values are loaded while the current group is processed (ping-pong
  // between two register sets), so a group costs one memory latency
  constexpr int U = 4;
  // Loads are unconditional, from clamped rows (the program has a token
  // when a group is loaded), and kept raw: values outside the program are
  // zeroed, and bf16 widened, only at use, so nothing waits between loads.
  using Raw = act_raw_t<T>;
  auto load_group = [&](int t0, float* dv, Raw* xv) {  // tokens t0, t0 - 1, ..., t0 - U + 1
#pragma unroll
    for (int j = 0; j < U; ++j) {
      const int tt = t0 - j, tn = tt - K;
      dv[j] = du[(int64_t)(base + max(tt, 0)) * E + e];
      xv[j] = x[(int64_t)(base + max(tn, 0)) * ldx + e];
    }
  };
  auto run_group = [&](int t0, const float* dv, const Raw* xv) {
#pragma unroll
    for (int j = 0; j < U; ++j) {
      const int t = t0 - j;
      if (t < 0) break;  // block-uniform
      float xc = be;
#pragma unroll
      for (int k = 0; k < K; ++k) xc = fmaf(wk[k], xw[k], xc);
      const float dxc = dv[j] * silu_grad(xc);  // t >= 0 here: dv[j] is token t's
      // future window: fut[i] = dxc_{t+i}
#pragma unroll
      for (int i = K - 1; i > 0; --i) fut[i] = fut[i - 1];
      fut[0] = dxc;
      float dxv = 0.f;
#pragma unroll
      for (int k = 0; k < K; ++k) dxv = fmaf(wk[k], fut[K - 1 - k], dxv);
      dx[(int64_t)(base + t) * lddx + e] = dxv;
#pragma unroll
      for (int k = 0; k < K; ++k) dw[k] = fmaf(dxc, xw[k], dw[k]);
      db += dxc;
      // slide the x window one token back: xw[0] = x_{t-K}
#pragma unroll
      for (int k = K - 1; k > 0; --k) xw[k] = xw[k - 1];
      xw[0] = t - K >= 0 ? act_f32(xv[j]) : 0.f;
    }
  };
  // (the next group is loaded even when the program has none left: its rows
  // clamp to the program's first token, so no load is conditional)
  float da[U], dbv[U];
  Raw xa[U], xb[U];
  int t = len - 1;
  if (t >= 0) load_group(t, da, xa);
  for (;;) {
    if (t < 0) break;  // da, xa hold the group at t
    load_group(t - U, dbv, xb);
    run_group(t, da, xa);
    t -= U;
    if (t < 0) break;  // dbv, xb hold the group at t
    load_group(t - U, da, xa);
    run_group(t, dbv, xb);
    t -= U;
  }
  float* o = part + (int64_t)b * (K + 1) * E + e;
#pragma unroll
  for (int k = 0; k < K; ++k) o[(int64_t)k * E] = dw[k];
  o[(int64_t)K * E] = db;
}

// ---------------------------------------------------------------- column sums
// part[s][c] = sum over rows of split s of A[m, c]  (rows < *Mdev).
__global__ __launch_bounds__(256) void colsum_kernel(const int* __restrict__ Mdev, int Mmax,
                                                     const float* __restrict__ A, int64_t lda, int C,
                                                     int rows_per_split, float* __restrict__ part) {
  const int c = blockIdx.x * 256 + threadIdx.x;
  if (c >= C) return;
  const int M = Mdev ? *Mdev : Mmax;
  const int r0 = blockIdx.y * rows_per_split;
  const int r1 = min(r0 + rows_per_split, M);
  float acc = 0.f;
  // unrolled so that several rows' loads are in flight (the sum stays sequential)
#pragma unroll 8
  for (int m = r0; m < r1; ++m) acc += A[(int64_t)m * lda + c];
  part[(int64_t)blockIdx.y * C + c] = acc;
}

// ---------------------------------------------------------------- reductions
// One launch covers several jobs; each job has its own range of blocks
// (about one per 64 outputs), so no block is launched without work. A block
// finds its job from the ranges (staged in LDS), takes 64 consecutive
// outputs; its 16 wavefronts each sum a contiguous sixteenth of the splits
// with eight independent partial sums (eight loads in flight per lane), then
// the partial sums and the sixteenths are added in a fixed order
// (deterministic for a given split count).
constexpr int kRedGroups = 16;
__global__ __launch_bounds__(64 * kRedGroups) void reduce_kernel(const ReduceJob* __restrict__ jobs, int njobs,
                                                                const float* __restrict__ ws,
                                                                float* __restrict__ grad,
                                                                float* __restrict__ loss) {
  __shared__ float sq[kRedGroups][64];
  __shared__ int sb[kMaxReduceJobs];
  __shared__ int sj;
  for (int k = threadIdx.x; k < njobs; k += 64 * kRedGroups) sb[k] = jobs[k].block0;
  __syncthreads();
  if (threadIdx.x == 0) {
    int lo = 0, hi = njobs;  // the last job whose range starts at or before this block
    while (hi - lo > 1) {
      const int mid = (lo + hi) >> 1;
      if (sb[mid] <= (int)blockIdx.x) lo = mid; else hi = mid;
    }
    sj = lo;
  }
  __syncthreads();
  const ReduceJob J = jobs[sj];
  float* dst = (J.dst_buf == 0 ? grad : loss) + J.dst;
  const float* src = ws + J.src;
  const int lane = threadIdx.x & 63, q = threadIdx.x >> 6;
  const int per = (J.nsplit + kRedGroups - 1) / kRedGroups;
  const int s0 = q * per, s1 = min(s0 + per, J.nsplit);
  for (int64_t i0 = (int64_t)((int)blockIdx.x - J.block0) * 64; i0 < J.n; i0 += (int64_t)J.nblocks * 64) {
    const int64_t i = i0 + lane;
    float a[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    if (i < J.n) {
      const float* p = src + i * J.src_stride;
      int s = s0;
      for (; s + 7 < s1; s += 8) {
#pragma unroll
        for (int k = 0; k < 8; ++k) a[k] += p[(int64_t)(s + k) * J.split_stride];
      }
      for (; s < s1; ++s) a[0] += p[(int64_t)s * J.split_stride];
    }
    sq[q][lane] = ((a[0] + a[1]) + (a[2] + a[3])) + ((a[4] + a[5]) + (a[6] + a[7]));
    __syncthreads();
    if (q == 0 && i < J.n) {
      float t = 0.f;
#pragma unroll
      for (int g = 0; g < kRedGroups; ++g) t += sq[g][lane];
      dst[i * J.dst_stride] = t;
    }
    __syncthreads();
  }
}

// ---------------------------------------------------------------- Adam
// Bias correction from the step count on the device (the steps already
// taken, before this one), so that a captured step replays with the right
// correction: bc_k = 1 - beta_k^t for t = *d_step + 1.
__global__ __launch_bounds__(256) void adam_kernel(int64_t n, float* __restrict__ p,
                                                   float* __restrict__ m, float* __restrict__ v,
                                                   const float* __restrict__ g, float lr, float b1,
                                                   float b2, float eps, const int64_t* __restrict__ d_step) {
  const double t = (double)(*d_step + 1);
  const float bc1 = 1.0f - (float)pow((double)b1, t);
  const float bc2 = 1.0f - (float)pow((double)b2, t);
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256) {
    const float gi = g[i];
    const float mi = fmaf(b1, m[i], (1.0f - b1) * gi);
    const float vi = fmaf(b2, v[i], (1.0f - b2) * gi * gi);
    m[i] = mi;
    v[i] = vi;
    p[i] -= lr * (mi / bc1) / (sqrtf(vi / bc2) + eps);
  }
}

// ---------------------------------------------------------------- weight derivation
// Every device-side weight layout is derived from the fp32 master blob by a
// table of jobs (copy, bf16 conversion, transpose, gain fold), in one launch.
__device__ __forceinline__ float round_to_bf16(float f) { return bf16_to_f32(f32_to_bf16(f)); }

__global__ __launch_bounds__(256) void derive_kernel(const float* __restrict__ master,
                                                     const DeriveJob* __restrict__ jobs, int njobs,
                                                     int64_t total, uint8_t* __restrict__ base,
                                                     int round_bf16, int64_t* __restrict__ step_bump) {
  // after a training step's Adam (the previous kernel on the stream, done
  // reading the count): advance the step count
  if (step_bump && blockIdx.x == 0 && threadIdx.x == 0) *step_bump += 1;
  for (int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x; idx < total;
       idx += (int64_t)gridDim.x * 256) {
    int lo = 0, hi = njobs;
    while (hi - lo > 1) {
      const int mid = (lo + hi) >> 1;
      if (jobs[mid].start <= idx) lo = mid; else hi = mid;
    }
    const DeriveJob J = jobs[lo];
    const int64_t k = idx - J.start;
    const int r = (int)(k / J.cols), c = (int)(k % J.cols);
    float v = master[J.src + k];
    if (round_bf16) v = round_to_bf16(v);
    if (J.kind == kDeriveFold || J.kind == kDeriveFoldSplit || J.kind == kDeriveFoldSplitF16) {
      float gv = master[J.src2 + c];
      if (round_bf16) gv = round_to_bf16(gv);
      v = v * gv;
    }
    const int64_t o = J.transpose ? (int64_t)c * J.ld + r : (int64_t)r * J.ld + c;
    if (J.kind == kDeriveSplit || J.kind == kDeriveFoldSplit) {
      uint32_t h, m, l;
      split3_pair(v, 0.f, h, m, l);
      uint16_t* d = reinterpret_cast<uint16_t*>(base + J.dst);
      const int64_t part = (int64_t)(J.transpose ? J.cols : J.rows) * J.ld;
      d[o] = (uint16_t)h;
      d[part + o] = (uint16_t)m;
      d[2 * part + o] = (uint16_t)l;
    } else if (J.kind == kDeriveSplitF16 || J.kind == kDeriveFoldSplitF16 || J.kind == kDeriveSplitF16Flat) {
      uint16_t h, l;
      if (J.kind == kDeriveSplitF16Flat)
        split2_f16_flat(v, h, l);
      else
        split2_f16_scaled(v, h, l);
      uint16_t* d = reinterpret_cast<uint16_t*>(base + J.dst);
      const int64_t part = (int64_t)(J.transpose ? J.cols : J.rows) * J.ld;
      d[o] = h;
      d[part + o] = l;
    } else if (J.kind == kDeriveBF16) {
      reinterpret_cast<uint16_t*>(base + J.dst)[o] = f32_to_bf16(v);
    } else {
      reinterpret_cast<float*>(base + J.dst)[o] = v;
    }
  }
}

}  // namespace

// ---------------------------------------------------------------- launchers

hipError_t launch_rmsnorm_fwd(int d, int Mmax, const int* Mdev, const float* H, const float* g,
                              float eps, uint16_t* n, float* rstd, hipStream_t s) {
  dim3 grid((Mmax + 3) / 4);
  switch (d) {
    case 64: hipLaunchKernelGGL(rmsnorm_fwd_kernel<64>, grid, dim3(256), 0, s, Mdev, H, g, eps, n, rstd); break;
    case 128: hipLaunchKernelGGL(rmsnorm_fwd_kernel<128>, grid, dim3(256), 0, s, Mdev, H, g, eps, n, rstd); break;
    case 256: hipLaunchKernelGGL(rmsnorm_fwd_kernel<256>, grid, dim3(256), 0, s, Mdev, H, g, eps, n, rstd); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

int rmsnorm_bwd_blocks(int Mmax) { return (Mmax + 63) / 64; }

hipError_t launch_rmsnorm_bwd(int d, int Mmax, const int* Mdev, const float* dN, const float* H,
                              const float* rstd, const float* g, float* dH, float* dg_part,
                              hipStream_t s) {
  dim3 grid(rmsnorm_bwd_blocks(Mmax));
  switch (d) {
    case 64: hipLaunchKernelGGL(rmsnorm_bwd_kernel<64>, grid, dim3(64 * kRnWaves), 0, s, Mdev, dN, H, rstd, g, dH, dg_part, 64); break;
    case 128: hipLaunchKernelGGL(rmsnorm_bwd_kernel<128>, grid, dim3(64 * kRnWaves), 0, s, Mdev, dN, H, rstd, g, dH, dg_part, 64); break;
    case 256: hipLaunchKernelGGL(rmsnorm_bwd_kernel<256>, grid, dim3(64 * kRnWaves), 0, s, Mdev, dN, H, rstd, g, dH, dg_part, 64); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

int loss_head_blocks(int B) { return (B + kHB - 1) / kHB; }

hipError_t launch_loss_head_bwd(int B, int d, int h, const float* s, const float* t, const float* y,
                                const float* a1, const float* W1, const float* W2, float* da1,
                                float* dpooled, float* part, hipStream_t st, const float* ds_in,
                                const float* loss_in) {
  if (h > 256 || d > 256 || (ds_in != nullptr) != (loss_in != nullptr)) return hipErrorInvalidValue;
  hipLaunchKernelGGL(loss_head_bwd_kernel, dim3(loss_head_blocks(B)), dim3(256), 0, st, B, d, h, s, t, y,
                     a1, W1, W2, da1, dpooled, part, ds_in, loss_in);
  return hipGetLastError();
}

hipError_t launch_normf_pool_bwd(int B, int d, const int* offs, const float* H, const float* g_f,
                                 int final_norm, float eps, const float* dpooled, float* dH,
                                 float* dg_part, hipStream_t s) {
  switch (d) {
    case 64: hipLaunchKernelGGL(normf_pool_bwd_kernel<64>, dim3(B), dim3(256), 0, s, offs, H, g_f, final_norm, eps, dpooled, dH, dg_part); break;
    case 128: hipLaunchKernelGGL(normf_pool_bwd_kernel<128>, dim3(B), dim3(256), 0, s, offs, H, g_f, final_norm, eps, dpooled, dH, dg_part); break;
    case 256: hipLaunchKernelGGL(normf_pool_bwd_kernel<256>, dim3(B), dim3(256), 0, s, offs, H, g_f, final_norm, eps, dpooled, dH, dg_part); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

size_t scan_bwd_ckpt_floats(int B, int E, int L, int N) {
  return (size_t)B * E * ((L + kTC - 1) / kTC) * N;
}

namespace {
// dB_t | dC_t of every token = the two channel groups' partial sums, in that order.
__global__ __launch_bounds__(256) void sum_dbc_kernel(const int* __restrict__ Mdev, int Mmax, int XW, int R,
                                                      int N2, const float* __restrict__ part,
                                                      float* __restrict__ dxdbl) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t row = i / N2;
  if (row >= *Mdev) return;
  dxdbl[row * XW + R + i % N2] = part[i] + part[(int64_t)Mmax * N2 + i];
}
}  // namespace

size_t scan_bwd_part_floats(int B, int L, int N) { return (size_t)2 * B * L * 2 * N; }

hipError_t launch_scan_bwd(int B, int E, int L, int N, int R, const int* offs, const uint16_t* u,
                           const float* xdbl, const uint16_t* xz, const uint16_t* ysave,
                           const float* dyg, const float* W_dt, const float* b_dt,
                           const float* A_log, const float* D, const float* ckpt, float* dv, float* du,
                           float* dxz, float* dxdbl, float* dA_part, float* dD_part, float* dbc_part,
                           hipStream_t s, const int* ord) {
  if (N != 16 || E % 32 || E > 256 || B <= 0 || L <= 0) return hipErrorInvalidValue;
  // the program's tokens are staged in windows of TW (a multiple of the
  // checkpoint interval) within 64 KiB of LDS: a window's [dt_r | B | C]
  // rows and its per-wavefront dB | dC partial sums
  const size_t per_token = ((size_t)(R + 2 * N) + (size_t)8 * 2 * N) * sizeof(float);
  const int fit = (int)((64 * 1024) / per_token) / kScanCkptTokens * kScanCkptTokens;
  const int TW = std::min((L + kScanCkptTokens - 1) / kScanCkptTokens * kScanCkptTokens, fit);
  const size_t shm = (size_t)TW * per_token;
  // the channels of a program in two blocks of E threads where E allows
  // (three such blocks fit a CU at this kernel's register count, against one
  // block of 2E threads); their dB/dC partial sums are added afterwards
  const int groups = (E % 64 == 0 && dbc_part) ? 2 : 1;
  const int Mmax = B * L;
#define TCL_SB(RR)                                                                                       \
  hipLaunchKernelGGL((scan_bwd_kernel<16, RR, uint16_t>), dim3(B, groups), dim3(2 * E / groups), shm, s, \
                     offs, E, L, u, xdbl, xz, ysave, dyg, W_dt, b_dt, A_log, D, ckpt, dv, du, dxz, dxdbl,   \
                     dA_part, dD_part, dbc_part, Mmax, TW, ord)
  switch (R) {
    case 4: TCL_SB(4); break;
    case 8: TCL_SB(8); break;
    case 16: TCL_SB(16); break;
    default: return hipErrorInvalidValue;
  }
#undef TCL_SB
  if (groups == 2) {
    const int64_t n = (int64_t)Mmax * 2 * N;
    hipLaunchKernelGGL(sum_dbc_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, offs + B, Mmax,
                       R + 2 * N, R, 2 * N, dbc_part, dxdbl);
  }
  return hipGetLastError();
}

hipError_t launch_conv_bwd(int B, int E, int K, const int* offs, const uint16_t* x, int ldx,
                           const float* w, const float* b, const float* du, float* dx, int lddx,
                           float* part, hipStream_t s) {
  dim3 grid(B, (E + 255) / 256);
  switch (K) {
    case 1: hipLaunchKernelGGL((conv_bwd_kernel<1, uint16_t>), grid, dim3(256), 0, s, offs, E, x, ldx, w, b, du, dx, lddx, part); break;
    case 2: hipLaunchKernelGGL((conv_bwd_kernel<2, uint16_t>), grid, dim3(256), 0, s, offs, E, x, ldx, w, b, du, dx, lddx, part); break;
    case 3: hipLaunchKernelGGL((conv_bwd_kernel<3, uint16_t>), grid, dim3(256), 0, s, offs, E, x, ldx, w, b, du, dx, lddx, part); break;
    case 4: hipLaunchKernelGGL((conv_bwd_kernel<4, uint16_t>), grid, dim3(256), 0, s, offs, E, x, ldx, w, b, du, dx, lddx, part); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

int colsum_splits(int Mmax) { return min(1024, max(1, (Mmax + 31) / 32)); }

hipError_t launch_colsum(const int* Mdev, int Mmax, const float* A, int64_t lda, int C, int splits,
                         float* part, hipStream_t s) {
  const int rps = (Mmax + splits - 1) / splits;
  hipLaunchKernelGGL(colsum_kernel, dim3((C + 255) / 256, splits), dim3(256), 0, s, Mdev, Mmax, A, lda,
                     C, rps, part);
  return hipGetLastError();
}

int reduce_blocks(ReduceJob* jobs, int njobs) {
  int total = 0;
  for (int j = 0; j < njobs; ++j) {
    jobs[j].block0 = total;
    jobs[j].nblocks = (int)std::min<int64_t>(std::max<int64_t>((jobs[j].n + 63) / 64, 1), 512);
    total += jobs[j].nblocks;
  }
  return total;
}

hipError_t launch_reduce(const ReduceJob* d_jobs, int njobs, int nblocks, const float* ws, float* grad,
                         float* loss, hipStream_t s) {
  if (njobs <= 0 || nblocks <= 0) return hipSuccess;
  if (njobs > kMaxReduceJobs) return hipErrorInvalidValue;
  hipLaunchKernelGGL(reduce_kernel, dim3(nblocks), dim3(64 * kRedGroups), 0, s, d_jobs, njobs, ws, grad, loss);
  return hipGetLastError();
}

hipError_t launch_adam(int64_t n, float* p, float* m, float* v, const float* g, float lr, float b1,
                       float b2, float eps, const int64_t* d_step, hipStream_t s) {
  const int grid = (int)std::min<int64_t>((n + 255) / 256, 2048);
  hipLaunchKernelGGL(adam_kernel, dim3(grid), dim3(256), 0, s, n, p, m, v, g, lr, b1, b2, eps, d_step);
  return hipGetLastError();
}

hipError_t launch_derive(const float* master, const DeriveJob* d_jobs, int njobs, int64_t total,
                         void* base, int round_bf16, hipStream_t s, int64_t* step_bump) {
  if (total <= 0) return hipSuccess;
  const int grid = (int)std::min<int64_t>((total + 255) / 256, 4096);
  hipLaunchKernelGGL(derive_kernel, dim3(grid), dim3(256), 0, s, master, d_jobs, njobs, total,
                     static_cast<uint8_t*>(base), round_bf16, step_bump);
  return hipGetLastError();
}

}  // namespace tcl
