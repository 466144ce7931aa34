// Per-program kernels of the forward pass: token packing, causal conv +
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
// slice is written out. With `ord`, the programs are also listed longest
// first (a counting sort over the lengths in LDS; the order of programs of
// equal length is unspecified), for kernels that walk each program's tokens
// in sequence: handing out the long programs first shortens the last round.
__device__ __forceinline__ int block_exclusive_scan(int v, int* wsum) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  int inc = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int u = __shfl_up(inc, o, 64);
    if (lane >= o) inc += u;
  }
  __syncthreads();  // wsum is free
  if (lane == 63) wsum[wave] = inc;
  __syncthreads();
  int before = 0;
  for (int w = 0; w < wave; ++w) before += wsum[w];
  return before + inc - v;
}
__global__ __launch_bounds__(1024) void offsets_kernel(const int* __restrict__ lengths, int B, int L,
                                                       int* __restrict__ offs, int* __restrict__ ord) {
  __shared__ int wsum[16];
  __shared__ int cnt[kOrderMaxL + 1];
  const int tid = threadIdx.x;
  // each thread owns a contiguous segment of a multiple of 4 programs, read
  // and written 16 bytes at a time when the arrays allow it
  const int per = (((B + 1023) / 1024) + 3) & ~3;
  const int s = min(tid * per, B), e = min(s + per, B);
  const bool vec = reinterpret_cast<uintptr_t>(lengths) % 16 == 0 && reinterpret_cast<uintptr_t>(offs) % 16 == 0;
  auto valid = [&](int len) { return (len >= 1 && len <= L) ? len : 0; };
  int sum = 0;
  int i = s;
  if (vec) {
#pragma unroll 4
    for (; i + 4 <= e; i += 4) {
      const int4 v = *reinterpret_cast<const int4*>(lengths + i);
      sum += valid(v.x) + valid(v.y) + valid(v.z) + valid(v.w);
    }
  }
  for (; i < e; ++i) sum += valid(lengths[i]);
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
  i = s;
  if (vec) {
#pragma unroll 4
    for (; i + 4 <= e; i += 4) {
      const int4 v = *reinterpret_cast<const int4*>(lengths + i);
      int4 o;
      o.x = run; run += valid(v.x);
      o.y = run; run += valid(v.y);
      o.z = run; run += valid(v.z);
      o.w = run; run += valid(v.w);
      *reinterpret_cast<int4*>(offs + i) = o;
    }
  }
  for (; i < e; ++i) {
    offs[i] = run;
    run += valid(lengths[i]);
  }
  if (tid == 1023) offs[B] = before + inc;
  if (ord == nullptr || L > kOrderMaxL) return;  // block-uniform

  // counting sort, longest first: bucket L - len
  const int nb = L + 1;
  for (int k = tid; k < nb; k += 1024) cnt[k] = 0;
  __syncthreads();
  for (int k = tid; k < B; k += 1024) atomicAdd(&cnt[L - valid(lengths[k])], 1);
  __syncthreads();
  const int pb = (nb + 1023) / 1024;
  const int b0 = min(tid * pb, nb), b1 = min(b0 + pb, nb);
  int csum = 0;
  for (int k = b0; k < b1; ++k) csum += cnt[k];
  int at = block_exclusive_scan(csum, wsum);
  for (int k = b0; k < b1; ++k) {
    const int c = cnt[k];
    cnt[k] = at;
    at += c;
  }
  __syncthreads();
  for (int k = tid; k < B; k += 1024) ord[atomicAdd(&cnt[L - valid(lengths[k])], 1)] = k;
}

// ---------------------------------------------------------------- element access
// Activations are fp32 or bf16 in memory; every kernel computes in fp32.
__device__ __forceinline__ float ld1(const float* p) { return *p; }
__device__ __forceinline__ float ld1(const uint16_t* p) { return bf16_to_f32(*p); }
__device__ __forceinline__ float to_f32(float v) { return v; }
__device__ __forceinline__ float to_f32(uint16_t v) { return bf16_to_f32(v); }
__device__ __forceinline__ void st1(float* p, float v) { *p = v; }
__device__ __forceinline__ void st1(uint16_t* p, float v) { *p = f32_to_bf16(v); }

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// One element per lane of row `row` of a buffer of rows: the lane's byte
// offset is fixed, the row's is wave-uniform (scalar), so a sequential
// kernel walking rows spends no vector instruction on addresses.
__device__ __forceinline__ float buf_ld(__amdgpu_buffer_rsrc_t r, uint32_t lane_bytes, uint32_t row_bytes,
                                        const float*) {
  return __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(r, lane_bytes, row_bytes, 0));
}
__device__ __forceinline__ uint16_t buf_ld(__amdgpu_buffer_rsrc_t r, uint32_t lane_bytes, uint32_t row_bytes,
                                           const uint16_t*) {
  return __builtin_amdgcn_raw_buffer_load_b16(r, lane_bytes, row_bytes, 0);
}
__device__ __forceinline__ void buf_st(float v, __amdgpu_buffer_rsrc_t r, uint32_t lane_bytes,
                                       uint32_t row_bytes, float*) {
  __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(v), r, lane_bytes, row_bytes, 0);
}
__device__ __forceinline__ void buf_st(float v, __amdgpu_buffer_rsrc_t r, uint32_t lane_bytes,
                                       uint32_t row_bytes, uint16_t*) {
  __builtin_amdgcn_raw_buffer_store_b16(f32_to_bf16(v), r, lane_bytes, row_bytes, 0);
}

// CH adjacent channels per thread: one 16-byte access (4 fp32 or 8 bf16).
template <typename T> struct Vec;
template <> struct Vec<float> {
  static constexpr int CH = 4;
  static __device__ __forceinline__ void load(const float* p, float* v) {
    const floatx4 x = *reinterpret_cast<const floatx4*>(p);
    v[0] = x.x; v[1] = x.y; v[2] = x.z; v[3] = x.w;
  }
  static __device__ __forceinline__ void cvt(u32x4 x, float* v) {
    v[0] = __uint_as_float(x[0]); v[1] = __uint_as_float(x[1]);
    v[2] = __uint_as_float(x[2]); v[3] = __uint_as_float(x[3]);
  }
  static __device__ __forceinline__ void store(float* p, const float* v) {
    *reinterpret_cast<floatx4*>(p) = floatx4{v[0], v[1], v[2], v[3]};
  }
};
template <> struct Vec<uint16_t> {
  static constexpr int CH = 8;
  static __device__ __forceinline__ void load(const uint16_t* p, float* v) {
    const u32x4 x = *reinterpret_cast<const u32x4*>(p);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      v[2 * i] = __uint_as_float(x[i] << 16);
      v[2 * i + 1] = __uint_as_float(x[i] & 0xFFFF0000u);
    }
  }
  static __device__ __forceinline__ void cvt(u32x4 x, float* v) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      v[2 * i] = __uint_as_float(x[i] << 16);
      v[2 * i + 1] = __uint_as_float(x[i] & 0xFFFF0000u);
    }
  }
  static __device__ __forceinline__ void store(uint16_t* p, const float* v) {
    u32x4 x;
#pragma unroll
    for (int i = 0; i < 4; ++i) x[i] = f32x2_to_bf16x2(v[2 * i], v[2 * i + 1]);
    *reinterpret_cast<u32x4*>(p) = x;
  }
};

// ---------------------------------------------------------------- conv + SiLU
// One thread per (program, CH adjacent channels): 16-byte loads and stores,
// x_{t-K+1..t} of its channels in a K-deep register window. Tokens go in
// groups of 4 whose loads are issued one group ahead of the arithmetic.
template <typename T, int K>
__global__ __launch_bounds__(256) void conv_silu_kernel(const int* __restrict__ offs, int E,
                                                        const T* __restrict__ x, int ldx,
                                                        const float* __restrict__ w,
                                                        const float* __restrict__ bias,
                                                        T* __restrict__ u) {
  constexpr int CH = Vec<T>::CH;
  const int b = blockIdx.x;
  const int e0 = (blockIdx.y * blockDim.x + threadIdx.x) * CH;
  if (e0 >= E) return;
  const int base = offs[b], len = offs[b + 1] - base;
  float wk[K][CH], win[K][CH], be[CH];
#pragma unroll
  for (int c = 0; c < CH; ++c) {
    be[c] = bias[e0 + c];
#pragma unroll
    for (int k = 0; k < K; ++k) {
      wk[k][c] = w[(e0 + c) * K + k];
      win[k][c] = 0.f;
    }
  }
  const T* xp = x + (int64_t)base * ldx + e0;
  T* up = u + (int64_t)base * E + e0;
  auto step = [&](const float* xin, T* dst) {
#pragma unroll
    for (int k = 0; k < K - 1; ++k)
#pragma unroll
      for (int c = 0; c < CH; ++c) win[k][c] = win[k + 1][c];
    float acc[CH];
#pragma unroll
    for (int c = 0; c < CH; ++c) {
      win[K - 1][c] = xin[c];
      acc[c] = be[c];
#pragma unroll
      for (int k = 0; k < K; ++k) acc[c] = fmaf(wk[k][c], win[k][c], acc[c]);
      acc[c] = silu(acc[c]);
    }
    Vec<T>::store(dst, acc);
  };
  // groups of U tokens, ping-ponged between two raw register sets: group
  // t + U is loaded while group t is converted and computed
  constexpr int U = 4;
  auto load_group = [&](int t0, u32x4* g) {
#pragma unroll
    for (int j = 0; j < U; ++j) g[j] = *reinterpret_cast<const u32x4*>(xp + (int64_t)(t0 + j) * ldx);
  };
  auto run_group = [&](int t0, const u32x4* g) {
#pragma unroll
    for (int j = 0; j < U; ++j) {
      float xin[CH];
      Vec<T>::cvt(g[j], xin);
      step(xin, up + (int64_t)(t0 + j) * E);
    }
  };
  u32x4 ga[U], gb[U];
  int t = 0;
  if (U <= len) load_group(0, ga);
  for (;;) {
    if (t + U > len) break;  // ga holds group t
    if (t + 2 * U <= len) load_group(t + U, gb);
    run_group(t, ga);
    t += U;
    if (t + U > len) break;  // gb holds group t
    if (t + 2 * U <= len) load_group(t + U, ga);
    run_group(t, gb);
    t += U;
  }
  for (; t < len; ++t) {
    float xin[CH];
    Vec<T>::load(xp + (int64_t)t * ldx, xin);
    step(xin, up + (int64_t)t * E);
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

template <typename T, int N, int R>
__global__ __launch_bounds__(kScanThreads) void scan_kernel(
    int B, const int* __restrict__ offs, int E, const T* u, const float* __restrict__ xdbl,
    const T* __restrict__ z, int ldz, const float* __restrict__ W_dt,
    const float* __restrict__ b_dt, const float* __restrict__ A_log,
    const float* __restrict__ Dp, T* out, T* __restrict__ ysave, float* __restrict__ ckpt, int nck,
    const int* __restrict__ ord) {
  constexpr int XW = R + 2 * N;
  __shared__ __attribute__((aligned(16))) float sX[kScanTC * XW];
  // workgroups are handed to the 8 XCDs round-robin: the CG channel groups
  // of a program take consecutive slots on one XCD, so its xdbl rows are
  // read from HBM once and then hit that XCD's L2; slots go to programs in
  // the order `ord` gives (longest first) when there is one
  const int CG = (E + kScanThreads - 1) / kScanThreads;
  const int xcd = blockIdx.x & 7, j = blockIdx.x >> 3;
  const int slot = (j / CG) * 8 + xcd;
  if (slot >= B) return;
  const int b = ord ? ord[slot] : slot;
  const int e = (j % CG) * kScanThreads + threadIdx.x;
  const bool active = e < E;
  const int ec = active ? e : 0;
  const int base = offs[b], len = offs[b + 1] - base;

  float a2[N], s[N], wdt[R];
#pragma unroll
  for (int n = 0; n < N; ++n) {
    a2[n] = -__builtin_amdgcn_exp2f(A_log[ec * N + n] * kLog2e) * kLog2e;
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
    // this chunk's rows of u, z, out and ysave as buffers: row offsets stay
    // scalar (each resource spans at most kScanTC rows, so 32 bits suffice)
    const int64_t r0 = base + t0;
    const __amdgpu_buffer_rsrc_t ub = raw_rsrc(u + r0 * E, (uint32_t)(nt * E * sizeof(T)));
    const __amdgpu_buffer_rsrc_t zb = raw_rsrc(z + r0 * ldz, (uint32_t)(nt * ldz * sizeof(T)));
    const __amdgpu_buffer_rsrc_t ob = raw_rsrc(out + r0 * E, (uint32_t)(nt * E * sizeof(T)));
    const __amdgpu_buffer_rsrc_t yb = raw_rsrc(ysave ? ysave + r0 * E : out, ysave ? (uint32_t)(nt * E * sizeof(T)) : 0u);
    const uint32_t lane = (uint32_t)(e * sizeof(T)), urow = (uint32_t)(E * sizeof(T)),
                   zrow = (uint32_t)(ldz * sizeof(T));
    auto token = [&](int tt, T ut, T zt) {
      const float* xr = &sX[tt * XW];
      const float uv = to_f32(ut), zv = to_f32(zt);
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
      if (ysave) buf_st(y, yb, lane, tt * urow, ysave);
      buf_st(y * silu(zv), ob, lane, tt * urow, out);
      const int t = t0 + tt;
      if (ckpt && t % kScanCkptTokens == kScanCkptTokens - 1 && t + 1 < len) {
        floatx4* dst = reinterpret_cast<floatx4*>(ckpt + (((int64_t)b * E + e) * nck + t / kScanCkptTokens) * N);
#pragma unroll
        for (int n = 0; n < N; n += 4) dst[n / 4] = floatx4{s[n], s[n + 1], s[n + 2], s[n + 3]};
      }
    };
    // Two tokens per trip (the state then alternates between two register
    // sets instead of being copied back after every token). u and z are
    // loaded a pair ahead of their use; rows past the chunk read as 0 from
    // the buffer, so the loads need no guard. They stay in their storage
    // type until used, so that converting them does not wait for the load.
    T u0 = buf_ld(ub, lane, 0, u), z0 = buf_ld(zb, lane, 0, z);
    T u1 = buf_ld(ub, lane, urow, u), z1 = buf_ld(zb, lane, zrow, z);
    int tt = 0;
    for (; tt + 1 < nt; tt += 2) {
      const T ua = u0, za = z0, ub1 = u1, zb1 = z1;
      u0 = buf_ld(ub, lane, (tt + 2) * urow, u);
      z0 = buf_ld(zb, lane, (tt + 2) * zrow, z);
      u1 = buf_ld(ub, lane, (tt + 3) * urow, u);
      z1 = buf_ld(zb, lane, (tt + 3) * zrow, z);
      token(tt, ua, za);
      token(tt + 1, ub1, zb1);
    }
    if (tt < nt) token(tt, u0, z0);
  }
}

// Lane i of each row of 16 lanes takes lane i - D's value (DPP row_shr:D);
// the first D lanes of a row receive 0.
template <int D>
__device__ __forceinline__ float row_shr(float v) {
  static_assert(D >= 1 && D <= 15, "row_shr:1..15");
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x110 + D, 0xF, 0xF, false));
}

// ---------------------------------------------------------------- chunked two-level scan
// For batches too small to fill the GPU with one thread per (program,
// channel): the sequence is split into W chunks that run concurrently, one
// wavefront each, for 64 channels of one program (lane = channel, so every
// load stays coalesced). The recurrence s_t = a_t s_{t-1} + b_t is affine, so
// a chunk acts on its incoming state as s -> P s + s_loc with
// P = prod_t a_t = exp(A sum_t dt_t) and s_loc the chunk's end state from a
// zero start. Level 1: every wavefront scans its chunk from zero and parks
// (P, s_loc) in LDS. Carry: the chunks' maps are composed in order by a
// prefix scan across lanes (DPP row shifts, eight lanes per channel and
// state), which leaves every chunk's incoming state in LDS. Level 2: each
// wavefront re-runs its chunk from there, writing the outputs. This spends twice the exponentials
// of the sequential scan; it pays only when the extra concurrency is needed.
template <typename T, int N, int R>
__global__ __launch_bounds__(512) void scan_chunked_kernel(
    const int* __restrict__ offs, int E, const T* u, const float* __restrict__ xdbl,
    const T* __restrict__ z, int ldz, const float* __restrict__ W_dt,
    const float* __restrict__ b_dt, const float* __restrict__ A_log,
    const float* __restrict__ Dp, T* out) {
  constexpr int XW = R + 2 * N;
  extern __shared__ float sSum[];  // [W chunks][64 lanes][2N]: P | s_loc
  const int b = blockIdx.x;
  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int nw = blockDim.x >> 6;
  const int e = blockIdx.y * 64 + lane;
  const bool active = e < E;
  const int ec = active ? e : 0;
  const int base = offs[b], len = offs[b + 1] - base;
  const int tpc = (len + nw - 1) / nw;  // tokens per chunk
  const int t_begin = min(w * tpc, len), t_end = min(t_begin + tpc, len);

  float a2[N], wdt[R];
#pragma unroll
  for (int n = 0; n < N; ++n) a2[n] = -__builtin_amdgcn_exp2f(A_log[ec * N + n] * kLog2e) * kLog2e;
#pragma unroll
  for (int r = 0; r < R; ++r) wdt[r] = W_dt[ec * R + r];
  const float bdt = b_dt[ec], Dv = Dp[ec];

  auto dt_at = [&](const float* xr) {
    float v = bdt;
#pragma unroll
    for (int r = 0; r < R; ++r) v = fmaf(wdt[r], xr[r], v);
    return softplus(v);
  };

  // level 1: the chunk's summary from a zero incoming state
  float s[N];
  float sumdt = 0.f;
#pragma unroll
  for (int n = 0; n < N; ++n) s[n] = 0.f;
  // u (and z) of the next token are loaded while this token is computed
  T un = t_begin < t_end ? u[(int64_t)(base + t_begin) * E + ec] : T(0);
  for (int t = t_begin; t < t_end; ++t) {
    const float* xr = xdbl + (int64_t)(base + t) * XW;  // wavefront-uniform row
    const float uv = to_f32(un);
    if (t + 1 < t_end) un = u[(int64_t)(base + t + 1) * E + ec];
    const float dt = dt_at(xr);
    sumdt += dt;
    const float dtu = dt * uv;
#pragma unroll
    for (int n = 0; n < N; ++n) s[n] = fmaf(__builtin_amdgcn_exp2f(dt * a2[n]), s[n], dtu * xr[R + n]);
  }
  float* mine = sSum + ((int64_t)w * 64 + lane) * 2 * N;
#pragma unroll
  for (int n = 0; n < N; ++n) {
    mine[n] = __builtin_amdgcn_exp2f(a2[n] * sumdt);
    mine[N + n] = s[n];
  }
  __syncthreads();

  // carry: for every (channel, state) the chunks' maps s -> P s + S are
  // composed in chunk order by a scan across lanes. Eight lanes take one
  // (channel, state), lane j of the eight holding chunk j (chunks past nw
  // hold the identity); three DPP row shifts (by 1, 2, 4 lanes, masked at
  // the group's start) form the inclusive scan, one more shift the
  // exclusive one: chunk j's incoming state is the composed S of chunks
  // 0..j-1 applied to a zero state. It replaces P in the summary slot.
  {
    const int j = lane & 7;
    for (int task0 = 0; task0 < N * 64; task0 += 8 * nw) {
      const int task = task0 + w * 8 + (lane >> 3);
      const int c = task & 63, n = task >> 6;
      const bool ok = task < N * 64 && j < nw;
      float* slot = sSum + ((int64_t)j * 64 + c) * 2 * N + n;
      float P = ok ? slot[0] : 1.f, S = ok ? slot[N] : 0.f;
      float Pp = row_shr<1>(P), Sp = row_shr<1>(S);
      if (j >= 1) { S = fmaf(P, Sp, S); P *= Pp; }
      Pp = row_shr<2>(P); Sp = row_shr<2>(S);
      if (j >= 2) { S = fmaf(P, Sp, S); P *= Pp; }
      Pp = row_shr<4>(P); Sp = row_shr<4>(S);
      if (j >= 4) { S = fmaf(P, Sp, S); P *= Pp; }
      Sp = row_shr<1>(S);
      if (ok) slot[0] = j >= 1 ? Sp : 0.f;
    }
  }
  __syncthreads();

  // level 2: each chunk re-run from its incoming state
#pragma unroll
  for (int n = 0; n < N; ++n) s[n] = mine[n];
  if (!active) return;
  un = t_begin < t_end ? u[(int64_t)(base + t_begin) * E + e] : T(0);
  T zn = t_begin < t_end ? z[(int64_t)(base + t_begin) * ldz + e] : T(0);
  for (int t = t_begin; t < t_end; ++t) {
    const int64_t row = base + t;
    const float* xr = xdbl + row * XW;
    const float uv = to_f32(un), zv = to_f32(zn);
    if (t + 1 < t_end) {
      un = u[(row + 1) * E + e];
      zn = z[(row + 1) * ldz + e];
    }
    const float dt = dt_at(xr);
    const float dtu = dt * uv;
    float y = 0.f;
#pragma unroll
    for (int n = 0; n < N; ++n) {
      s[n] = fmaf(__builtin_amdgcn_exp2f(dt * a2[n]), s[n], dtu * xr[R + n]);
      y = fmaf(s[n], xr[R + N + n], y);
    }
    y = fmaf(Dv, uv, y);
    st1(out + row * E + e, y * silu(zv));
  }
}

// ---------------------------------------------------------------- tail
// PB programs per workgroup. Phase 1: each wavefront pools whole programs
// (per token: RMSNorm statistics by a wavefront reduction, then accumulate
// the normalised row). Phase 2: thread j computes hidden unit j of the head
// for all PB programs (W1 is read once per workgroup, transposed so the
// reads are coalesced), then the ReLU'd units are dotted with W2 by a
// block reduction. With DEC3 (a three-layer decoder) the ReLU'd units go
// through LDS to a second hidden layer of h2 units, thread j computing unit
// j, and those are dotted with W3 (b2 is then the second layer's bias
// vector, b3 the output bias).
template <int DM, int kTailPB, bool DEC3>
__global__ __launch_bounds__(256) void tail_kernel(int B, int L, int h, const int* __restrict__ offs,
                                                   const int* __restrict__ lengths,
                                                   const float* __restrict__ H,
                                                   const float* __restrict__ g_f, int final_norm,
                                                   float eps, const float* __restrict__ W1T,
                                                   const float* __restrict__ b1,
                                                   const float* __restrict__ W2,
                                                   const float* __restrict__ b2,
                                                   float* __restrict__ scores,
                                                   float* __restrict__ pooled_out,
                                                   float* __restrict__ a1_out, int h2,
                                                   const float* __restrict__ W3,
                                                   const float* __restrict__ b3) {
  constexpr int PL = DM / 64;  // values per lane
  __shared__ float sP[DM][kTailPB];
  __shared__ float sRed[4][kTailPB];
  __shared__ float sH1[DEC3 ? 256 : 1][kTailPB];
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
      // tokens in groups of U rows, ping-ponged between two register sets:
      // group t + U is loaded while group t is reduced and accumulated
      // (loads clamp to the last row; rows past the end are masked at use)
      constexpr int U = 4;
      auto load_group = [&](int t0, float (*g)[PL]) {
#pragma unroll
        for (int j = 0; j < U; ++j) {
          const float* hr = H + (int64_t)(base + min(t0 + j, len - 1)) * DM + lane * PL;
#pragma unroll
          for (int i = 0; i < PL; ++i) g[j][i] = hr[i];
        }
      };
      auto run_group = [&](int t0, float (*g)[PL]) {
        float rs[U];
#pragma unroll
        for (int j = 0; j < U; ++j) {
          rs[j] = t0 + j < len ? 1.f : 0.f;
          if (final_norm) {
            float ss = 0.f;
#pragma unroll
            for (int i = 0; i < PL; ++i) ss = fmaf(g[j][i], g[j][i], ss);
            ss = wave_sum(ss);
            rs[j] *= 1.0f / sqrtf(ss / (float)DM + eps);
          }
        }
#pragma unroll
        for (int j = 0; j < U; ++j)
#pragma unroll
          for (int i = 0; i < PL; ++i) acc[i] = fmaf(g[j][i], rs[j], acc[i]);
      };
      float ga[U][PL], gb[U][PL];
      if (len > 0) load_group(0, ga);
      for (int t = 0;;) {
        if (t >= len) break;  // ga holds group t
        if (t + U < len) load_group(t + U, gb);
        run_group(t, ga);
        t += U;
        if (t >= len) break;  // gb holds group t
        if (t + U < len) load_group(t + U, ga);
        run_group(t, gb);
        t += U;
      }
    }
    const float inv = len > 0 ? 1.0f / (float)len : 0.f;
#pragma unroll
    for (int i = 0; i < PL; ++i) {
      const int k = lane * PL + i;
      const float g = final_norm ? g_f[k] : 1.f;
      sP[k][p] = acc[i] * g * inv;
      if (pooled_out && b < B) pooled_out[(int64_t)b * DM + k] = acc[i] * g * inv;
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
    // W1 in batches of KB rows, the next batch loaded while the current one
    // is used (L2 latency, not the FMAs, bounds this loop); fully unrolled,
    // so the batches are fixed registers and no load is conditional
    constexpr int KB = kTailPB > 4 ? 8 : 16;  // (more programs: more FMAs per row, fewer rows needed in flight)
    static_assert(DM % (2 * KB) == 0, "whole pairs of W1 batches");
    float wa[KB], wb[KB];
    auto load_w = [&](int k0, float* w) {
#pragma unroll
      for (int j = 0; j < KB; ++j) w[j] = W1T[(k0 + j) * h + tid];
    };
    auto use_w = [&](int k0, const float* w) {
#pragma unroll
      for (int j = 0; j < KB; ++j)
#pragma unroll
        for (int p = 0; p < kTailPB; ++p) a[p] = fmaf(w[j], sP[k0 + j][p], a[p]);
    };
    load_w(0, wa);
#pragma unroll
    for (int k0 = 0; k0 < DM; k0 += 2 * KB) {
      load_w(k0 + KB, wb);
      use_w(k0, wa);
      if (k0 + 2 * KB < DM) load_w(k0 + 2 * KB, wa);
      use_w(k0 + KB, wb);
    }
    if constexpr (DEC3) {
#pragma unroll
      for (int p = 0; p < kTailPB; ++p) sH1[tid][p] = fmaxf(a[p], 0.f);
    } else {
      const float w2 = W2[tid];
#pragma unroll
      for (int p = 0; p < kTailPB; ++p) part[p] = w2 * fmaxf(a[p], 0.f);
    }
    if (a1_out) {
#pragma unroll
      for (int p = 0; p < kTailPB; ++p)
        if (b0 + p < B) a1_out[(int64_t)(b0 + p) * h + tid] = a[p];
    }
  }
  if constexpr (DEC3) {
    // second hidden layer: W2 is passed transposed, [h][h2]
    __syncthreads();
    if (tid < h2) {
      float a[kTailPB];
      const float bj = b2[tid];
#pragma unroll
      for (int p = 0; p < kTailPB; ++p) a[p] = bj;
#pragma unroll 32
      for (int k = 0; k < h; ++k) {
        const float wv = W2[k * h2 + tid];
#pragma unroll
        for (int p = 0; p < kTailPB; ++p) a[p] = fmaf(wv, sH1[k][p], a[p]);
      }
      const float w3 = W3[tid];
#pragma unroll
      for (int p = 0; p < kTailPB; ++p) part[p] = w3 * fmaxf(a[p], 0.f);
    }
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
      const float sc = sRed[0][tid] + sRed[1][tid] + sRed[2][tid] + sRed[3][tid] + (DEC3 ? b3[0] : b2[0]);
      const int len = lengths[b];
      scores[b] = (len >= 1 && len <= L) ? sc : __builtin_nanf("");
    }
  }
}

}  // namespace

namespace {

__global__ __launch_bounds__(256) void pad_rows_kernel(int64_t n, int F, int ld, const float* __restrict__ src,
                                                       float* __restrict__ dst) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256) {
    const int64_t r = i / ld;
    const int c = (int)(i - r * ld);
    dst[i] = c < F ? src[r * F + c] : 0.f;
  }
}

__global__ __launch_bounds__(256) void mask_scores_kernel(int B, int L, const int* __restrict__ lengths,
                                                          float* __restrict__ scores) {
  const int b = blockIdx.x * 256 + threadIdx.x;
  if (b < B) {
    const int len = lengths[b];
    if (len < 1 || len > L) scores[b] = __builtin_nanf("");
  }
}

}  // namespace

hipError_t launch_mask_scores(int B, int L, const int* lengths, float* scores, hipStream_t s) {
  if (B <= 0) return hipSuccess;
  hipLaunchKernelGGL(mask_scores_kernel, dim3((B + 255) / 256), dim3(256), 0, s, B, L, lengths, scores);
  return hipGetLastError();
}

hipError_t launch_pad_rows(const float* src, int64_t rows, int F, int ld, float* dst, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  if (F <= 0 || ld < F) return hipErrorInvalidValue;
  const int64_t n = rows * ld;
  const int grid = (int)std::min<int64_t>((n + 255) / 256, 8192);
  hipLaunchKernelGGL(pad_rows_kernel, dim3(grid), dim3(256), 0, s, n, F, ld, src, dst);
  return hipGetLastError();
}

hipError_t launch_offsets(const int* lengths, int B, int L, int* offs, hipStream_t s, int* ord) {
  hipLaunchKernelGGL(offsets_kernel, dim3(1), dim3(1024), 0, s, lengths, B, L, offs, ord);
  return hipGetLastError();
}

namespace {
// One thread per program writes the positions of its tokens.
__global__ __launch_bounds__(256) void token_pos_kernel(const int* __restrict__ offs, int B,
                                                        uint8_t* __restrict__ tpos) {
  const int b = blockIdx.x * 256 + threadIdx.x;
  if (b >= B) return;
  const int base = offs[b], len = offs[b + 1] - base;
  for (int t = 0; t < len; ++t) tpos[base + t] = (uint8_t)min(t, 255);
}
}  // namespace

hipError_t launch_token_pos(const int* offs, int B, uint8_t* tpos, hipStream_t s) {
  if (B <= 0) return hipSuccess;
  hipLaunchKernelGGL(token_pos_kernel, dim3((B + 255) / 256), dim3(256), 0, s, offs, B, tpos);
  return hipGetLastError();
}

template <typename T>
hipError_t launch_conv_silu(int B, int E, int K, const int* offs, const T* x, int ldx,
                            const float* w, const float* b, T* u, hipStream_t s) {
  constexpr int CH = Vec<T>::CH;
  if (B <= 0) return hipSuccess;
  if (E % CH || ldx % CH) return hipErrorInvalidValue;
  dim3 grid(B, (E / CH + 255) / 256);
  switch (K) {
    case 1: hipLaunchKernelGGL((conv_silu_kernel<T, 1>), grid, dim3(256), 0, s, offs, E, x, ldx, w, b, u); break;
    case 2: hipLaunchKernelGGL((conv_silu_kernel<T, 2>), grid, dim3(256), 0, s, offs, E, x, ldx, w, b, u); break;
    case 3: hipLaunchKernelGGL((conv_silu_kernel<T, 3>), grid, dim3(256), 0, s, offs, E, x, ldx, w, b, u); break;
    case 4: hipLaunchKernelGGL((conv_silu_kernel<T, 4>), grid, dim3(256), 0, s, offs, E, x, ldx, w, b, u); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <typename T>
hipError_t launch_scan_chunked(int B, int E, int N, int R, int chunks, const int* offs, const T* u,
                               const float* xdbl, const T* z, int ldz, const float* W_dt,
                               const float* b_dt, const float* A_log, const float* D, T* out,
                               hipStream_t s) {
  if (B <= 0) return hipSuccess;
  if ((N != 16 && N != 8) || chunks < 1 || chunks > 8) return hipErrorInvalidValue;
  dim3 grid(B, (E + 63) / 64);
  const size_t shm = (size_t)chunks * 64 * 2 * N * sizeof(float);
#define TCL_SCANC(NN, RR)                                                                      \
  hipLaunchKernelGGL((scan_chunked_kernel<T, NN, RR>), grid, dim3(64 * chunks), shm, s, offs, E, u, \
                     xdbl, z, ldz, W_dt, b_dt, A_log, D, out)
  switch (N * 100 + R) {
    case 1604: TCL_SCANC(16, 4); break;
    case 1608: TCL_SCANC(16, 8); break;
    case 1612: TCL_SCANC(16, 12); break;
    case 1616: TCL_SCANC(16, 16); break;
    case 1620: TCL_SCANC(16, 20); break;
    case 1624: TCL_SCANC(16, 24); break;
    case 1628: TCL_SCANC(16, 28); break;
    case 1632: TCL_SCANC(16, 32); break;
    case 804: TCL_SCANC(8, 4); break;
    case 808: TCL_SCANC(8, 8); break;
    case 816: TCL_SCANC(8, 16); break;
    default: return hipErrorInvalidValue;
  }
#undef TCL_SCANC
  return hipGetLastError();
}

int scan_chunks_for(int B, int E, int L) {
  // One thread per (program, channel) gives B*E/64 wavefronts. Measured on
  // MI355X at L = 256, E = 512: the sequential scan wins from 2048 wavefronts
  // up (B >= 256), the chunked scan from 512 down (1.7x at B = 64 with 4
  // chunks, 2.3x at B = 16 with 4-8). Aim for >= 2048 wavefronts in total.
  const int64_t waves = (int64_t)B * ((E + 63) / 64);
  if (L < 64 || waves >= 1024) return 0;
  int c = 2;
  while (c < 8 && waves * c < 2048 && L / (2 * c) >= 8) c *= 2;
  return c;
}

template <typename T>
hipError_t launch_scan(int B, int E, int N, int R, const int* offs, const T* u, const float* xdbl,
                       const T* z, int ldz, const float* W_dt, const float* b_dt, const float* A_log,
                       const float* D, T* out, hipStream_t s, T* ysave, float* ckpt, int L, const int* ord) {
  if (B <= 0) return hipSuccess;
  if (N != 16 && N != 8) return hipErrorInvalidValue;
  if (ckpt && (L <= 0 || reinterpret_cast<uintptr_t>(ckpt) % 16)) return hipErrorInvalidValue;
  const int nck = (L + kScanCkptTokens - 1) / kScanCkptTokens;
  const int cgroups = (E + kScanThreads - 1) / kScanThreads;
  const int grid = 8 * cgroups * ((B + 7) / 8);
#define TCL_SCAN(NN, RR)                                                                                \
  hipLaunchKernelGGL((scan_kernel<T, NN, RR>), dim3(grid), dim3(kScanThreads), 0, s, B, offs, E, u, xdbl, \
                     z, ldz, W_dt, b_dt, A_log, D, out, ysave, ckpt, nck, ord)
  switch (N * 100 + R) {
    case 1604: TCL_SCAN(16, 4); break;
    case 1608: TCL_SCAN(16, 8); break;
    case 1612: TCL_SCAN(16, 12); break;
    case 1616: TCL_SCAN(16, 16); break;
    case 1620: TCL_SCAN(16, 20); break;
    case 1624: TCL_SCAN(16, 24); break;
    case 1628: TCL_SCAN(16, 28); break;
    case 1632: TCL_SCAN(16, 32); break;
    case 804: TCL_SCAN(8, 4); break;
    case 808: TCL_SCAN(8, 8); break;
    case 816: TCL_SCAN(8, 16); break;
    default: return hipErrorInvalidValue;
  }
#undef TCL_SCAN
  return hipGetLastError();
}

template hipError_t launch_conv_silu<float>(int, int, int, const int*, const float*, int, const float*,
                                            const float*, float*, hipStream_t);
template hipError_t launch_conv_silu<uint16_t>(int, int, int, const int*, const uint16_t*, int,
                                               const float*, const float*, uint16_t*, hipStream_t);
template hipError_t launch_scan_chunked<float>(int, int, int, int, int, const int*, const float*,
                                               const float*, const float*, int, const float*,
                                               const float*, const float*, const float*, float*,
                                               hipStream_t);
template hipError_t launch_scan_chunked<uint16_t>(int, int, int, int, int, const int*,
                                                  const uint16_t*, const float*, const uint16_t*, int,
                                                  const float*, const float*, const float*,
                                                  const float*, uint16_t*, hipStream_t);
template hipError_t launch_scan<float>(int, int, int, int, const int*, const float*, const float*,
                                       const float*, int, const float*, const float*, const float*,
                                       const float*, float*, hipStream_t, float*, float*, int, const int*);
template hipError_t launch_scan<uint16_t>(int, int, int, int, const int*, const uint16_t*,
                                          const float*, const uint16_t*, int, const float*,
                                          const float*, const float*, const float*, uint16_t*,
                                          hipStream_t, uint16_t*, float*, int, const int*);

namespace {

hipError_t tail_any(int B, int L, int d, int h, const int* offs, const int* lengths, const float* H,
                    const float* g_f, int final_norm, float eps, const float* W1T, const float* b1,
                    const float* W2, const float* b2, float* scores, hipStream_t s, float* pooled_out,
                    float* a1_out, int h2, const float* W3, const float* b3) {
  if (B <= 0) return hipSuccess;
  if (h <= 0 || h > 256 || h2 < 0 || h2 > 256) return hipErrorInvalidValue;
  // 16 programs per workgroup share each W1 read; small batches use 4 so
  // that there are enough workgroups to spread over the CUs
  const int pb = B >= 8192 ? 16 : 4;
  dim3 grid((B + pb - 1) / pb);
  const bool d3 = h2 > 0;
#define TCL_TAIL(DD, PB)                                                                                  \
  if (d3)                                                                                                 \
    hipLaunchKernelGGL((tail_kernel<DD, PB, true>), grid, dim3(256), 0, s, B, L, h, offs, lengths, H, g_f, \
                       final_norm, eps, W1T, b1, W2, b2, scores, pooled_out, a1_out, h2, W3, b3);         \
  else                                                                                                    \
    hipLaunchKernelGGL((tail_kernel<DD, PB, false>), grid, dim3(256), 0, s, B, L, h, offs, lengths, H,    \
                       g_f, final_norm, eps, W1T, b1, W2, b2, scores, pooled_out, a1_out, 0, nullptr,     \
                       nullptr)
  switch (d * 100 + pb) {
    case 6416: TCL_TAIL(64, 16); break;
    case 12816: TCL_TAIL(128, 16); break;
    case 25616: TCL_TAIL(256, 16); break;
    case 6404: TCL_TAIL(64, 4); break;
    case 12804: TCL_TAIL(128, 4); break;
    case 25604: TCL_TAIL(256, 4); break;
    default: return hipErrorInvalidValue;
  }
#undef TCL_TAIL
  return hipGetLastError();
}

}  // namespace

hipError_t launch_tail_f32(int B, int L, int d, int h, const int* offs, const int* lengths,
                           const float* H, const float* g_f, int final_norm, float eps,
                           const float* W1T, const float* b1, const float* W2, const float* b2,
                           float* scores, hipStream_t s, float* pooled_out, float* a1_out) {
  return tail_any(B, L, d, h, offs, lengths, H, g_f, final_norm, eps, W1T, b1, W2, b2, scores, s,
                  pooled_out, a1_out, 0, nullptr, nullptr);
}

hipError_t launch_tail3_f32(int B, int L, int d, int h, int h2, const int* offs, const int* lengths,
                            const float* H, const float* g_f, int final_norm, float eps,
                            const float* W1T, const float* b1, const float* W2T, const float* b2,
                            const float* W3, const float* b3, float* scores, hipStream_t s) {
  if (h2 <= 0) return hipErrorInvalidValue;
  return tail_any(B, L, d, h, offs, lengths, H, g_f, final_norm, eps, W1T, b1, W2T, b2, scores, s,
                  nullptr, nullptr, h2, W3, b3);
}

}  // namespace tcl
