// fp32 GEMMs on the bf16 matrix cores: C = rowscale * (A W^T) + bias (+ R),
// A and W fp32, with fp32 accuracy.
//
// Every fp32 value splits exactly into three bf16 values, x = x1 + x2 + x3
// (split3 in common.h). Of the nine products x_i y_j of two split values the
// six with i + j <= 4 are kept; the three dropped ones (x2 y3, x3 y2, x3 y3)
// are at most 2^-23 |x y| together, two units of fp32 rounding, while the
// fp32 sum of a K-term dot product is itself only bounded by K units. Each
// bf16 x bf16 product is exact in fp32 and the MFMA accumulates in fp32. On
// gfx950 a bf16 MFMA does 16x the work of an fp32 MFMA in the same time, so
// six of them reach 2.67x the fp32 matrix peak.
//
// Row panels, as in the fp32 and bf16 panel kernels: a workgroup of 4
// wavefronts owns a panel of rows and all N columns.
//  * prologue: each wavefront loads its rows of A once (gathered rows for
//    the input Linear), takes the RMSNorm row statistics from them, splits
//    them and keeps the three parts as MFMA fragments in registers;
//  * main loop: the three bf16 parts of W (split once when the model's
//    weights are derived) go through a double-buffered LDS stage a column
//    block at a time, one barrier per block; the next block's W is loaded
//    into registers at the start of a block and written to the other buffer
//    halfway through its MFMAs (with one wavefront per SIMD nothing else
//    would cover the staging); per k-step a wavefront reads three W
//    fragments and issues six MFMAs;
//  * epilogue per block: row scale, bias and residual on the accumulators,
//    buffer stores straight from them.
// Variants (what limits them is the LDS traffic of the streamed W
// fragments: one fragment read feeds two MFMAs on average, so a 16-row
// panel on 16x16 blocks needs twice the LDS bytes per flop of a 32-row one):
//  1. split32: v_mfma_f32_32x32x16_bf16, 32 rows per wavefront, K <= 256,
//     any N (in_proj, the input Linear);
//  2. split16: v_mfma_f32_16x16x32_bf16, 16 rows per wavefront, K <= 512,
//     any N;
//  3. split32acc: 32 rows per wavefront and N <= 256, K <= 512: the
//     accumulators of all N columns stay in registers while K is walked in
//     chunks (of 128 above K = 256; A's parts for one chunk at a time), so
//     a 32-row panel fits at K = 512 (out_proj).
//
// Fragment k-order (A and W alike, which is all the contraction needs):
// split32 k-step s, lane half g holds k = 16 s + 8 g .. +7; split16 k-step
// s, lane quarter q holds k = 32 s + 8 q .. +7.
#include <algorithm>
#include <type_traits>

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

// 8 consecutive fp32 values of a row -> their three bf16 parts, element j
// of each fragment holding value j
__device__ __forceinline__ void split8(const floatx4 a, const floatx4 b, bf16x8& p1, bf16x8& p2,
                                       bf16x8& p3) {
  const float x[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
  u32x4 w1, w2, w3;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    uint32_t h, m, l;
    split3_pair(x[2 * i], x[2 * i + 1], h, m, l);
    w1[i] = h;
    w2[i] = m;
    w3[i] = l;
  }
  p1 = __builtin_bit_cast(bf16x8, w1);
  p2 = __builtin_bit_cast(bf16x8, w2);
  p3 = __builtin_bit_cast(bf16x8, w3);
}

// Loads 8 fp32 of row `arow` at k (zero past K or for a missing row);
// K % 4 == 0, so each half is all in or all out.
__device__ __forceinline__ void load8(const float* arow, bool rok, int k, int K, floatx4& v0,
                                      floatx4& v1) {
  const bool ok0 = rok && k < K, ok1 = rok && k + 4 < K;
  v0 = *reinterpret_cast<const floatx4*>(arow + (ok0 ? k : 0));
  v1 = *reinterpret_cast<const floatx4*>(arow + (ok1 ? k + 4 : 0));
  if (!ok0) v0 = floatx4{0.f, 0.f, 0.f, 0.f};
  if (!ok1) v1 = floatx4{0.f, 0.f, 0.f, 0.f};
}

// The W stage of one column block: NR rows of each of the three parts, KC
// chunks of 64 k. Unit u of the block is part u / (NR WU), row (u / WU) % NR,
// k = 8 (u % WU); rows past N and k past the padded K read zero through the
// resource (the part stride is N ldw, so a row past N must not be read as
// the next part's).
template <int NR, int KC, int NT = kWaves * 64>
struct WStage {
  static constexpr int WP = KC * 64 + 8;  // bf16 pitch of a staged row (conflict-free 16-byte reads)
  static constexpr int WU = KC * 8;       // 16-byte units per row
  static constexpr int NWU = 3 * NR * WU; // units per block
  static constexpr int NW = (NWU + NT - 1) / NT;
  u32x4 r[NW];
  __device__ __forceinline__ void load(const __amdgpu_buffer_rsrc_t& res, int tid, int n0, int N,
                                       int ldw, int Kw, int k0 = 0) {
#pragma unroll
    for (int i = 0; i < NW; ++i) {
      const int u = tid + i * NT;
      const int part = u / (NR * WU), n = n0 + (u / WU) % NR, k = k0 + 8 * (u % WU);
      const bool ok = (NWU % NT == 0 || u < NWU) && n < N && k < Kw;
      // 32-bit offsets (the resource is below 2^31 bytes), moved out of range
      // by setting bit 31: arithmetic, not a branch around the load (which
      // makes the compiler wait for every outstanding memory operation
      // before the other side reuses the registers)
      const uint32_t off = (uint32_t)(((part * N + n) * ldw + k) * 2) | ((uint32_t)!ok << 31);
      r[i] = __builtin_amdgcn_raw_buffer_load_b128(res, off, 0, 0);
    }
  }
  __device__ __forceinline__ void stage(uint16_t* s, int tid) const {
#pragma unroll
    for (int i = 0; i < NW; ++i) {
      const int u = tid + i * NT;
      if (NWU % NT == 0 || u < NWU)
        *reinterpret_cast<u32x4*>(&s[(u / WU) * WP + 8 * (u % WU)]) = r[i];
    }
  }
};

// The same units loaded and staged in two halves through NW / 2 + 1
// registers: [0, H) then [H, NW).
template <int NR, int KC, int NT>
struct WStageHalves {
  using S = WStage<NR, KC, NT>;
  static constexpr int NW = S::NW, H = (NW + 1) / 2, WP = S::WP, WU = S::WU, NWU = S::NWU;
  u32x4 r[H];
  template <int I0, int I1>
  __device__ __forceinline__ void load(const __amdgpu_buffer_rsrc_t& res, int tid, int n0, int N, int ldw, int Kw) {
#pragma unroll
    for (int i = I0; i < I1; ++i) {
      const int u = tid + i * NT;
      const int part = u / (NR * WU), n = n0 + (u / WU) % NR, k = 8 * (u % WU);
      const bool ok = (NWU % NT == 0 || u < NWU) && n < N && k < Kw;
      const uint32_t off = (uint32_t)(((part * N + n) * ldw + k) * 2) | ((uint32_t)!ok << 31);
      r[i - I0] = __builtin_amdgcn_raw_buffer_load_b128(res, off, 0, 0);
    }
  }
  template <int I0, int I1>
  __device__ __forceinline__ void stage(uint16_t* s, int tid) const {
#pragma unroll
    for (int i = I0; i < I1; ++i) {
      const int u = tid + i * NT;
      if (NWU % NT == 0 || u < NWU)
        *reinterpret_cast<u32x4*>(&s[(u / WU) * WP + 8 * (u % WU)]) = r[i - I0];
    }
  }
};

// ---------------------------------------------------------------- 32-row panels
template <int KC, int FL>
__global__ __launch_bounds__(kWaves * 64, 1) void gemm_split32_kernel(GemmArgs p, const uint16_t* Ws,
                                                                      int ldws) {
  constexpr int NS = KC * 4;  // 16-k MFMA steps
  constexpr int BM = kWaves * 32;
  using Stage = WStage<32, KC>;
  constexpr int WP = Stage::WP;
  constexpr int PART = 32 * WP;  // one part of one buffer
  constexpr bool kNorm = (FL & kRowNorm) != 0;
  static_assert((FL & kResid) == 0, "32-row split panels have no residual epilogue");

  __shared__ __attribute__((aligned(16))) uint16_t sW[2 * 3 * PART];
  __shared__ float sR[kWaves][32];
  __shared__ int sSrc[BM];

  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63;
  const int li = lane & 31, lg = lane >> 5;
  const int M = p.Mdev ? *p.Mdev : p.Mmax;
  const int row0 = blockIdx.x * BM;
  if (row0 >= M) return;

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
        if (p.tpos) p.tpos[grow] = (uint8_t)min(grow - p.offs[lo], 255);
      }
    }
    sSrc[r] = src;
  }

  const int Kw = (p.K + 7) & ~7;
  const __amdgpu_buffer_rsrc_t wres = make_rsrc(Ws, (uint32_t)__builtin_amdgcn_readfirstlane(3 * p.N * ldws * 2));
  const int nsteps = (p.N + 31) / 32;
  Stage st;
  st.load(wres, tid, 0, p.N, ldws, Kw);  // in flight during the prologue
  __syncthreads();  // sSrc

  // prologue: row li of this wavefront's 32, lane half lg's 8 k of every step
  bf16x8 a1[NS], a2[NS], a3[NS];
  {
    const int src = sSrc[wave * 32 + li];
    const float* arow = p.A + (src >= 0 ? (int64_t)src * p.lda : 0);
    float ss = 0.f;
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      floatx4 v0, v1;
      load8(arow, src >= 0, 16 * s + 8 * lg, p.K, v0, v1);
      if constexpr (kNorm)
        ss += v0.x * v0.x + v0.y * v0.y + v0.z * v0.z + v0.w * v0.w + v1.x * v1.x + v1.y * v1.y +
              v1.z * v1.z + v1.w * v1.w;
      split8(v0, v1, a1[s], a2[s], a3[s]);
    }
    if constexpr (kNorm) {
      ss += __shfl_xor(ss, 32, 64);  // the other half of the row
      if (lg == 0) sR[wave][li] = 1.0f / sqrtf(ss / (float)p.K + p.eps);
    }
  }

  const uint32_t panel_bytes = (uint32_t)(min(BM, M - row0) * p.ldc * 4);
  const __amdgpu_buffer_rsrc_t cres = make_rsrc(p.C + (int64_t)row0 * p.ldc, panel_bytes);

  st.stage(&sW[0], tid);
  for (int s = 0; s < nsteps; ++s) {
    const int buf = s & 1, n0 = s * 32;
    // block s (staged during block s-1) visible; every wavefront is past
    // block s-1, so the other buffer is free for block s+1
    __syncthreads();
    const bool more = s + 1 < nsteps;
    if (more) st.load(wres, tid, n0 + 32, p.N, ldws, Kw);

    // two accumulation chains (the small part products, then the large),
    // so that consecutive MFMAs do not wait for each other's results
    floatx16 acc, acc2;
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[r] = acc2[r] = 0.f;
    const uint16_t* wb = &sW[buf * 3 * PART + li * WP + 8 * lg];
    auto wfrag = [&](int part, int ks) {
      return __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(wb + part * PART + 16 * ks));
    };
    // W fragments two k-steps ahead of their MFMAs, in a ring of three
    bf16x8 q[3][3];
#pragma unroll
    for (int ks = 0; ks < 2 && ks < NS; ++ks)
#pragma unroll
      for (int j = 0; j < 3; ++j) q[ks][j] = wfrag(j, ks);
    __builtin_amdgcn_sched_group_barrier(0x0100, NS > 1 ? 6 : 3, 0);
#pragma unroll
    for (int ks = 0; ks < NS; ++ks) {
      if (ks + 2 < NS) {
#pragma unroll
        for (int j = 0; j < 3; ++j) q[(ks + 2) % 3][j] = wfrag(j, ks + 2);
      }
      const bf16x8* w = q[ks % 3];
      acc2 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a3[ks], w[0], acc2, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a2[ks], w[0], acc, 0, 0, 0);
      acc2 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1[ks], w[2], acc2, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1[ks], w[1], acc, 0, 0, 0);
      acc2 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a2[ks], w[1], acc2, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1[ks], w[0], acc, 0, 0, 0);
      if (ks + 2 < NS) __builtin_amdgcn_sched_group_barrier(0x0100, 3, 0);
      __builtin_amdgcn_sched_group_barrier(0x0008, 6, 0);
      // block s+1 into the other buffer halfway through this block's MFMAs
      if (ks == NS / 2 && more) {
        st.stage(&sW[(buf ^ 1) * 3 * PART], tid);
        __builtin_amdgcn_sched_group_barrier(0x0200, Stage::NW, 0);
      }
    }

    // epilogue: lane l holds column l % 32 and rows 8*(r/4) + 4*(l/32) + (r%4)
    const int col = n0 + li;
    const bool cok = col < p.N;
    const float bias = ((FL & kBias) != 0) ? p.bias[cok ? col : 0] : 0.f;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int rl = 8 * (r >> 2) + 4 * lg + (r & 3);
      float v = acc[r] + acc2[r];
      if constexpr (kNorm) v *= sR[wave][rl];
      v += bias;
      if (p.relu) v = fmaxf(v, 0.f);
      // rows past M fall outside cres
      const uint32_t off = cok ? (uint32_t)(((wave * 32 + rl) * p.ldc + col) * 4) : kOutOfRange;
      __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, v), cres, off, 0, 0);
    }
  }
}

// ---------------------------------------------------------------- 32-row panels, K in two halves
// The 32-row panel with K split between two wavefronts per SIMD: eight
// wavefronts per workgroup, wavefront w owning rows 32 (w % 4) .. +31 and
// the K half w / 4 (KH chunks of 64 each). Each holds only its half of A's
// parts (half the registers of the one-wavefront panel), so two wavefronts
// share every SIMD and one issues while the other waits. Per column block
// the upper-half wavefronts park their partial sums in LDS at the end of the
// block, and the lower-half wavefronts add them and run the epilogue of that
// block while the next block's MFMAs go on (the W stage and the partials are
// both double-buffered, one barrier per block).
constexpr int kWavesH = 8;
template <int KH, int FL>
__global__ __launch_bounds__(kWavesH * 64, 1) void gemm_split32h_kernel(GemmArgs p, const uint16_t* Ws,
                                                                        int ldws) {
  constexpr int NSH = KH * 4;  // 16-k MFMA steps per half
  constexpr int KC = 2 * KH;
  constexpr int BM = 128;
  constexpr int NT = kWavesH * 64;
  using Stage = WStageHalves<32, KC, NT>;
  constexpr int WP = Stage::WP;
  constexpr int PART = 32 * WP;
  constexpr int NW = Stage::NW, HW = Stage::H;
  constexpr bool kNorm = (FL & kRowNorm) != 0;
  static_assert((FL & kResid) == 0, "no residual epilogue");

  __shared__ __attribute__((aligned(16))) uint16_t sW[2 * 3 * PART];
  // upper-half partial sums, [buffer][row group][quarter q][lane][4]: a
  // lane's four values of quarter q are one 16-byte unit and consecutive
  // lanes' units are consecutive (conflict-free 16-byte accesses)
  __shared__ __attribute__((aligned(16))) float sP[2][4][4][64][4];
  __shared__ float sSS[2][4][32];
  __shared__ float sR[4][32];
  __shared__ int sSrc[BM];

  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63;
  const int g = wave & 3, h = wave >> 2;
  const int li = lane & 31, lg = lane >> 5;
  const int M = p.Mdev ? *p.Mdev : p.Mmax;
  const int row0 = blockIdx.x * BM;
  if (row0 >= M) return;

  for (int r = tid; r < BM; r += NT) {
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
        if (p.tpos) p.tpos[grow] = (uint8_t)min(grow - p.offs[lo], 255);
      }
    }
    sSrc[r] = src;
  }

  const int Kw = (p.K + 7) & ~7;
  const __amdgpu_buffer_rsrc_t wres = make_rsrc(Ws, (uint32_t)__builtin_amdgcn_readfirstlane(3 * p.N * ldws * 2));
  // this workgroup's column blocks [sb, se): all of them, or one of
  // gridDim.y ranges when a small batch leaves too few panels for the GPU
  const int nblk = (p.N + 31) / 32;
  const int sb = (int)(blockIdx.y * nblk / gridDim.y), se = (int)((blockIdx.y + 1) * nblk / gridDim.y);
  Stage st;
  __syncthreads();  // sSrc

  // prologue: row li of this wavefront's 32, lane half lg's 8 k of every
  // step of this wavefront's K half
  const int kh = h * KH * 64;
  bf16x8 a1[NSH], a2[NSH], a3[NSH];
  {
    const int src = sSrc[g * 32 + li];
    const float* arow = p.A + (src >= 0 ? (int64_t)src * p.lda : 0);
    float ss = 0.f;
#pragma unroll
    for (int s = 0; s < NSH; ++s) {
      floatx4 v0, v1;
      load8(arow, src >= 0, kh + 16 * s + 8 * lg, p.K, v0, v1);
      if constexpr (kNorm)
        ss += v0.x * v0.x + v0.y * v0.y + v0.z * v0.z + v0.w * v0.w + v1.x * v1.x + v1.y * v1.y +
              v1.z * v1.z + v1.w * v1.w;
      split8(v0, v1, a1[s], a2[s], a3[s]);
    }
    if constexpr (kNorm) {
      ss += __shfl_xor(ss, 32, 64);
      if (lg == 0) sSS[h][g][li] = ss;
    }
  }

  const uint32_t panel_bytes = (uint32_t)(min(BM, M - row0) * p.ldc * 4);
  const __amdgpu_buffer_rsrc_t cres = make_rsrc(p.C + (int64_t)row0 * p.ldc, panel_bytes);

  st.template load<0, HW>(wres, tid, sb * 32, p.N, ldws, Kw);
  st.template stage<0, HW>(&sW[0], tid);
  st.template load<HW, NW>(wres, tid, sb * 32, p.N, ldws, Kw);
  st.template stage<HW, NW>(&sW[0], tid);
  if constexpr (kNorm) {
    __syncthreads();  // both halves' sums of squares
    if (h == 0 && lg == 0) sR[g][li] = 1.0f / sqrtf((sSS[0][g][li] + sSS[1][g][li]) / (float)p.K + p.eps);
  }

  // the lower-half wavefronts finish block s: its upper-half partials from
  // LDS, row scale, bias, activation, buffer stores
  floatx16 res;
  auto epilogue = [&](int s) {
    const int col = s * 32 + li;
    const bool cok = col < p.N;
    const float bias = ((FL & kBias) != 0) ? p.bias[cok ? col : 0] : 0.f;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const floatx4 o = *reinterpret_cast<const floatx4*>(&sP[(s - sb) & 1][g][q][lane][0]);
      res[4 * q] += o.x;
      res[4 * q + 1] += o.y;
      res[4 * q + 2] += o.z;
      res[4 * q + 3] += o.w;
    }
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int rl = 8 * (r >> 2) + 4 * lg + (r & 3);
      float v = res[r];
      if constexpr (kNorm) v *= sR[g][rl];
      v += bias;
      if (p.relu) v = fmaxf(v, 0.f);
      const uint32_t off = cok ? (uint32_t)(((g * 32 + rl) * p.ldc + col) * 4) : kOutOfRange;
      __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, v), cres, off, 0, 0);
    }
  };

  // The block loop, compiled once per K half (a wavefront-uniform choice):
  // the lower half's epilogue stores are then only on its own path, so the
  // wait for the W stage's loads (issued before them) need not wait for the
  // stores as well, as it would after a join with the upper half's path.
  auto blocks = [&](auto lower_tag) {
    constexpr bool LOWER = decltype(lower_tag)::value;
    for (int s = sb; s < se; ++s) {
      const int buf = (s - sb) & 1, n0 = s * 32;
      // block s staged and block s-1's partials parked; every wavefront is
      // past block s-1's fragment reads and the partials of block s-2
      __syncthreads();
      const bool more = s + 1 < se;
      // the next block's W in two halves: the first loaded now and staged
      // halfway through the MFMAs, the second loaded then and staged at the end
      if (more) st.template load<0, HW>(wres, tid, n0 + 32, p.N, ldws, Kw);
      if (LOWER && s > sb) epilogue(s - 1);

      floatx16 acc, acc2;
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[r] = acc2[r] = 0.f;
      const uint16_t* wb = &sW[buf * 3 * PART + li * WP + 8 * lg + kh];
      auto wfrag = [&](int part, int ks) {
        return __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(wb + part * PART + 16 * ks));
      };
      // W fragments one k-step ahead of their MFMAs (the other wavefront on
      // the SIMD covers the rest of the LDS latency)
      bf16x8 q[2][3];
#pragma unroll
      for (int j = 0; j < 3; ++j) q[0][j] = wfrag(j, 0);
      __builtin_amdgcn_sched_group_barrier(0x0100, 3, 0);
#pragma unroll
      for (int ks = 0; ks < NSH; ++ks) {
        if (ks + 1 < NSH) {
#pragma unroll
          for (int j = 0; j < 3; ++j) q[(ks + 1) & 1][j] = wfrag(j, ks + 1);
        }
        const bf16x8* w = q[ks & 1];
        acc2 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a3[ks], w[0], acc2, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a2[ks], w[0], acc, 0, 0, 0);
        acc2 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1[ks], w[2], acc2, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1[ks], w[1], acc, 0, 0, 0);
        acc2 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a2[ks], w[1], acc2, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1[ks], w[0], acc, 0, 0, 0);
        if (ks + 1 < NSH) __builtin_amdgcn_sched_group_barrier(0x0100, 3, 0);
        __builtin_amdgcn_sched_group_barrier(0x0008, 6, 0);
        if (ks == NSH / 2 && more) {
          st.template stage<0, HW>(&sW[(buf ^ 1) * 3 * PART], tid);
          st.template load<HW, NW>(wres, tid, n0 + 32, p.N, ldws, Kw);
          __builtin_amdgcn_sched_group_barrier(0x0200, HW, 0);
        }
      }
      if (more) st.template stage<HW, NW>(&sW[(buf ^ 1) * 3 * PART], tid);
      if constexpr (!LOWER) {
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4)
          *reinterpret_cast<floatx4*>(&sP[buf][g][q4][lane][0]) =
              floatx4{acc[4 * q4] + acc2[4 * q4], acc[4 * q4 + 1] + acc2[4 * q4 + 1],
                      acc[4 * q4 + 2] + acc2[4 * q4 + 2], acc[4 * q4 + 3] + acc2[4 * q4 + 3]};
      } else {
#pragma unroll
        for (int r = 0; r < 16; ++r) res[r] = acc[r] + acc2[r];
      }
    }
    __syncthreads();
    if constexpr (LOWER) epilogue(se - 1);
  };
  if (__builtin_amdgcn_readfirstlane(h) == 0)
    blocks(std::true_type{});
  else
    blocks(std::false_type{});
}

// ---------------------------------------------------------------- 16-row panels
template <int KC, int FL>
__global__ __launch_bounds__(kWaves * 64, 1) void gemm_split16_kernel(GemmArgs p, const uint16_t* Ws,
                                                                      int ldws) {
  constexpr int NS = KC * 2;  // 32-k MFMA steps
  constexpr int BM = kWaves * 16;
  using Stage = WStage<16, KC>;
  constexpr int WP = Stage::WP;
  constexpr int PART = 16 * WP;
  static_assert((FL & (kRowNorm | kGather)) == 0, "16-row split panels serve plain, bias and residual GEMMs");

  __shared__ __attribute__((aligned(16))) uint16_t sW[2 * 3 * PART];

  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63;
  const int lr = lane & 15, lq = lane >> 4;
  const int M = p.Mdev ? *p.Mdev : p.Mmax;
  const int row0 = blockIdx.x * BM;
  if (row0 >= M) return;

  const int Kw = (p.K + 7) & ~7;
  const __amdgpu_buffer_rsrc_t wres = make_rsrc(Ws, (uint32_t)__builtin_amdgcn_readfirstlane(3 * p.N * ldws * 2));
  const int nsteps = (p.N + 15) / 16;
  Stage st;
  st.load(wres, tid, 0, p.N, ldws, Kw);

  // prologue: row lr of this wavefront's 16, lane quarter lq's 8 k of every step
  bf16x8 a1[NS], a2[NS], a3[NS];
  {
    const int grow = row0 + wave * 16 + lr;
    const bool rok = grow < M;
    const float* arow = p.A + (rok ? (int64_t)grow * p.lda : 0);
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      floatx4 v0, v1;
      load8(arow, rok, 32 * s + 8 * lq, p.K, v0, v1);
      split8(v0, v1, a1[s], a2[s], a3[s]);
    }
  }

  const uint32_t panel_bytes = (uint32_t)(min(BM, M - row0) * p.ldc * 4);
  const __amdgpu_buffer_rsrc_t cres = make_rsrc(p.C + (int64_t)row0 * p.ldc, panel_bytes);
  const __amdgpu_buffer_rsrc_t rres =
      make_rsrc((p.R ? p.R : p.C) + (int64_t)row0 * p.ldc, (FL & kResid) != 0 ? panel_bytes : 0);

  st.stage(&sW[0], tid);
  for (int s = 0; s < nsteps; ++s) {
    const int buf = s & 1, n0 = s * 16;
    __syncthreads();  // block s visible; the other buffer is free for block s+1
    const bool more = s + 1 < nsteps;
    if (more) st.load(wres, tid, n0 + 16, p.N, ldws, Kw);

    // the residual of this block's outputs, loaded while the MFMAs run
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

    floatx4 acc = floatx4{0.f, 0.f, 0.f, 0.f}, acc2 = acc;  // two chains, as above
    const uint16_t* wb = &sW[buf * 3 * PART + lr * WP + 8 * lq];
    auto wfrag = [&](int part, int ks) {
      return __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(wb + part * PART + 32 * ks));
    };
    bf16x8 q[3][3];
#pragma unroll
    for (int ks = 0; ks < 2 && ks < NS; ++ks)
#pragma unroll
      for (int j = 0; j < 3; ++j) q[ks][j] = wfrag(j, ks);
    __builtin_amdgcn_sched_group_barrier(0x0100, NS > 1 ? 6 : 3, 0);
#pragma unroll
    for (int ks = 0; ks < NS; ++ks) {
      if (ks + 2 < NS) {
#pragma unroll
        for (int j = 0; j < 3; ++j) q[(ks + 2) % 3][j] = wfrag(j, ks + 2);
      }
      const bf16x8* w = q[ks % 3];
      acc2 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a3[ks], w[0], acc2, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a2[ks], w[0], acc, 0, 0, 0);
      acc2 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a1[ks], w[2], acc2, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a1[ks], w[1], acc, 0, 0, 0);
      acc2 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a2[ks], w[1], acc2, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a1[ks], w[0], acc, 0, 0, 0);
      if (ks + 2 < NS) __builtin_amdgcn_sched_group_barrier(0x0100, 3, 0);
      __builtin_amdgcn_sched_group_barrier(0x0008, 6, 0);
      if (ks == NS / 2 && more) {
        st.stage(&sW[(buf ^ 1) * 3 * PART], tid);
        __builtin_amdgcn_sched_group_barrier(0x0200, Stage::NW, 0);
      }
    }

    // epilogue: lane l holds column l % 16 and rows 4*(l/16) + r
    const float bias = ((FL & kBias) != 0) ? p.bias[cok ? col : 0] : 0.f;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      float v = (acc[r] + acc2[r]) + bias + res[r];
      if (p.relu) v = fmaxf(v, 0.f);
      const uint32_t off = cok ? (uint32_t)(((wave * 16 + 4 * lq + r) * p.ldc + col) * 4) : kOutOfRange;
      __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, v), cres, off, 0, 0);
    }
  }
}

// ---------------------------------------------------------------- 32-row panels, all N in registers
// KCH chunks of KC * 64 k; NB 32-column blocks (N <= 32 NB).
template <int KC, int KCH, int NB, int FL>
__global__ __launch_bounds__(kWaves * 64, 1) void gemm_split32acc_kernel(GemmArgs p, const uint16_t* Ws,
                                                                         int ldws) {
  constexpr int NS = KC * 4;  // 16-k MFMA steps per chunk
  constexpr int BM = kWaves * 32;
  using Stage = WStage<32, KC>;
  constexpr int WP = Stage::WP;
  constexpr int PART = 32 * WP;
  static_assert((FL & (kRowNorm | kGather)) == 0, "plain, bias and residual GEMMs only");
  // PAIR: column blocks in pairs whose MFMAs alternate between the two
  // accumulators (no MFMA waits for the one before it), one barrier per
  // pair, W staged through a ring of four one-block LDS buffers
  constexpr bool PAIR = NB >= 4 && KC <= 2;
  constexpr int NBUF = PAIR ? 4 : 2;

  __shared__ __attribute__((aligned(16))) uint16_t sW[NBUF * 3 * PART];

  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63;
  const int li = lane & 31, lg = lane >> 5;
  const int M = p.Mdev ? *p.Mdev : p.Mmax;
  const int row0 = blockIdx.x * BM;
  if (row0 >= M) return;
  // this workgroup's NB column blocks start at column cb (gridDim.y > 1:
  // a small batch's columns split over more workgroups)
  const int cb = blockIdx.y * NB * 32;

  const int Kw = (p.K + 7) & ~7;
  const __amdgpu_buffer_rsrc_t wres = make_rsrc(Ws, (uint32_t)__builtin_amdgcn_readfirstlane(3 * p.N * ldws * 2));
  Stage st;
  st.load(wres, tid, cb, p.N, ldws, Kw, 0);

  const int grow = row0 + wave * 32 + li;
  const bool rok = grow < M;
  const float* arow = p.A + (rok ? (int64_t)grow * p.lda : 0);

  floatx16 acc[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[nb][r] = 0.f;
  st.stage(&sW[0], tid);
  if constexpr (PAIR) {
    st.load(wres, tid, cb + 32, p.N, ldws, Kw, 0);
    st.stage(&sW[3 * PART], tid);
  }

#pragma unroll
  for (int c = 0; c < KCH; ++c) {
    // keep the next chunk's loads of A below this point: hoisted, they would
    // hold a second set of A's parts in registers
    __builtin_amdgcn_sched_barrier(0);
    // this chunk of the wavefront's 32 rows -> three parts in registers
    bf16x8 a1[NS], a2[NS], a3[NS];
#pragma unroll
    for (int s2 = 0; s2 < NS; ++s2) {
      floatx4 v0, v1;
      load8(arow, rok, c * KC * 64 + 16 * s2 + 8 * lg, p.K, v0, v1);
      split8(v0, v1, a1[s2], a2[s2], a3[s2]);
    }
    if constexpr (PAIR) {
#pragma unroll
      for (int pp = 0; pp < NB / 2; ++pp) {
        const int g = c * NB + 2 * pp;  // global index of the pair's first block
        __syncthreads();  // this pair visible; the previous pair's buffers are free
        const bool more = pp + 1 < NB / 2 || c + 1 < KCH;
        const int ncol = cb + (pp + 1 < NB / 2 ? (2 * pp + 2) * 32 : 0);
        const int nk = pp + 1 < NB / 2 ? c * KC * 64 : (c + 1) * KC * 64;
        if (more) st.load(wres, tid, ncol, p.N, ldws, Kw, nk);

        const uint16_t* wb0 = &sW[(g & 3) * 3 * PART + li * WP + 8 * lg];
        const uint16_t* wb1 = &sW[((g + 1) & 3) * 3 * PART + li * WP + 8 * lg];
        auto wfrag = [&](const uint16_t* wb, int part, int ks) {
          return __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(wb + part * PART + 16 * ks));
        };
        bf16x8 q[2][6];
#pragma unroll
        for (int j = 0; j < 3; ++j) {
          q[0][j] = wfrag(wb0, j, 0);
          q[0][3 + j] = wfrag(wb1, j, 0);
        }
        __builtin_amdgcn_sched_group_barrier(0x0100, 6, 0);
        floatx16& x0 = acc[2 * pp];
        floatx16& x1 = acc[2 * pp + 1];
#pragma unroll
        for (int ks = 0; ks < NS; ++ks) {
          if (ks + 1 < NS) {
#pragma unroll
            for (int j = 0; j < 3; ++j) {
              q[(ks + 1) & 1][j] = wfrag(wb0, j, ks + 1);
              q[(ks + 1) & 1][3 + j] = wfrag(wb1, j, ks + 1);
            }
          }
          const bf16x8* w = q[ks & 1];
          x0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a3[ks], w[0], x0, 0, 0, 0);
          x1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a3[ks], w[3], x1, 0, 0, 0);
          x0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a2[ks], w[1], x0, 0, 0, 0);
          x1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a2[ks], w[4], x1, 0, 0, 0);
          x0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1[ks], w[2], x0, 0, 0, 0);
          x1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1[ks], w[5], x1, 0, 0, 0);
          x0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a2[ks], w[0], x0, 0, 0, 0);
          x1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a2[ks], w[3], x1, 0, 0, 0);
          x0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1[ks], w[1], x0, 0, 0, 0);
          x1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1[ks], w[4], x1, 0, 0, 0);
          x0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1[ks], w[0], x0, 0, 0, 0);
          x1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1[ks], w[3], x1, 0, 0, 0);
          if (ks + 1 < NS) __builtin_amdgcn_sched_group_barrier(0x0100, 6, 0);
          __builtin_amdgcn_sched_group_barrier(0x0008, 12, 0);
          // the next pair's two blocks: the first staged a quarter of the
          // way through, the second loaded then and staged at three quarters
          if (ks == NS / 4 && more) {
            st.stage(&sW[((g + 2) & 3) * 3 * PART], tid);
            __builtin_amdgcn_sched_group_barrier(0x0200, Stage::NW, 0);
            st.load(wres, tid, ncol + 32, p.N, ldws, Kw, nk);
          }
          if (ks == 3 * NS / 4 && more) {
            st.stage(&sW[((g + 3) & 3) * 3 * PART], tid);
            __builtin_amdgcn_sched_group_barrier(0x0200, Stage::NW, 0);
          }
        }
      }
    } else {
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      const int buf = (c * NB + nb) & 1;
      __syncthreads();  // this block visible; the other buffer is free for the next
      const bool more = nb + 1 < NB || c + 1 < KCH;
      if (nb + 1 < NB) st.load(wres, tid, cb + (nb + 1) * 32, p.N, ldws, Kw, c * KC * 64);
      else if (c + 1 < KCH) st.load(wres, tid, cb, p.N, ldws, Kw, (c + 1) * KC * 64);

      const uint16_t* wb = &sW[buf * 3 * PART + li * WP + 8 * lg];
      auto wfrag = [&](int part, int ks) {
        return __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(wb + part * PART + 16 * ks));
      };
      // W fragments one k-step ahead (a ring of two: registers are scarce here)
      bf16x8 q[2][3];
#pragma unroll
      for (int j = 0; j < 3; ++j) q[0][j] = wfrag(j, 0);
      __builtin_amdgcn_sched_group_barrier(0x0100, 3, 0);
#pragma unroll
      for (int ks = 0; ks < NS; ++ks) {
        if (ks + 1 < NS) {
#pragma unroll
          for (int j = 0; j < 3; ++j) q[(ks + 1) & 1][j] = wfrag(j, ks + 1);
        }
        const bf16x8* w = q[ks & 1];
        acc[nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a3[ks], w[0], acc[nb], 0, 0, 0);
        acc[nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a2[ks], w[1], acc[nb], 0, 0, 0);
        acc[nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1[ks], w[2], acc[nb], 0, 0, 0);
        acc[nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a2[ks], w[0], acc[nb], 0, 0, 0);
        acc[nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1[ks], w[1], acc[nb], 0, 0, 0);
        acc[nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1[ks], w[0], acc[nb], 0, 0, 0);
        if (ks + 1 < NS) __builtin_amdgcn_sched_group_barrier(0x0100, 3, 0);
        __builtin_amdgcn_sched_group_barrier(0x0008, 6, 0);
        if (ks == NS / 2 && more) {
          st.stage(&sW[(buf ^ 1) * 3 * PART], tid);
          __builtin_amdgcn_sched_group_barrier(0x0200, Stage::NW, 0);
        }
      }
    }
    }
  }

  // epilogue: lane l holds column nb*32 + l % 32 and rows 8*(r/4) + 4*(l/32) + (r%4)
  const uint32_t panel_bytes = (uint32_t)(min(BM, M - row0) * p.ldc * 4);
  const __amdgpu_buffer_rsrc_t cres = make_rsrc(p.C + (int64_t)row0 * p.ldc, panel_bytes);
  const __amdgpu_buffer_rsrc_t rres =
      make_rsrc((p.R ? p.R : p.C) + (int64_t)row0 * p.ldc, (FL & kResid) != 0 ? panel_bytes : 0);
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    const int col = cb + nb * 32 + li;
    const bool cok = col < p.N;
    const float bias = ((FL & kBias) != 0) ? p.bias[cok ? col : 0] : 0.f;
    float res[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int rl = 8 * (r >> 2) + 4 * lg + (r & 3);
      const uint32_t off = cok ? (uint32_t)(((wave * 32 + rl) * p.ldc + col) * 4) : kOutOfRange;
      res[r] = ((FL & kResid) != 0)
                   ? __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rres, off, 0, 0))
                   : 0.f;
    }
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int rl = 8 * (r >> 2) + 4 * lg + (r & 3);
      float v = acc[nb][r] + bias + res[r];
      if (p.relu) v = fmaxf(v, 0.f);
      const uint32_t off = cok ? (uint32_t)(((wave * 32 + rl) * p.ldc + col) * 4) : kOutOfRange;
      __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, v), cres, off, 0, 0);
    }
  }
}

// ---------------------------------------------------------------- x_proj with the conv in front
// The 32-row, all-N-in-registers panel of x_proj, walking K in chunks of 64
// channels whose A chunk is made in the kernel: each wavefront computes the
// causal conv + SiLU of its 32 rows (lane = channel; the 35 input rows, 3 of
// them before the wavefront's first row, are loaded one chunk ahead into
// registers), stores u, parks the chunk in LDS and reads its MFMA fragments
// from there. Two workgroups fit a CU. Taps that reach before a program's
// first token read zero, as in the stand-alone conv kernel, and the taps are
// summed in the same order, so u is the same bits either way.
// Copies the compiler cannot see through: values derived from them per
// chunk (lane masks, per-row offsets) are then built where they are used
// instead of being kept live across all chunks.
__device__ __forceinline__ uint32_t opaque_s(uint32_t v) {
  asm volatile("" : "+s"(v));
  return v;
}
__device__ __forceinline__ uint32_t opaque_v(uint32_t v) {
  asm volatile("" : "+v"(v));
  return v;
}

template <int KCH, bool XB>
__global__ __launch_bounds__(kWaves * 64, 2) void gemm_split32conv_kernel(GemmArgs p, ConvIn cv, const uint16_t* Ws,
                                                                          int ldws) {
  constexpr int NS = 4;               // 16-k MFMA steps per chunk
  constexpr int CW = 64;              // channels per chunk
  constexpr int PA = CW + 4;          // fp32 pitch of a parked row (conflict-free 16-byte reads)
  constexpr int XR = 32 + 3;          // conv input rows per wavefront
  constexpr int BM = kWaves * 32;
  using Stage = WStage<32, 1>;
  constexpr int WP = Stage::WP;
  constexpr int PART = 32 * WP;

  __shared__ __attribute__((aligned(16))) uint16_t sW[2 * 3 * PART];
  __shared__ __attribute__((aligned(16))) float sA[BM * PA];

  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63;
  const int li = lane & 31, lg = lane >> 5;
  const int M = p.Mdev ? *p.Mdev : p.Mmax;
  const int row0 = blockIdx.x * BM;
  if (row0 >= M) return;
  const int E = p.K;

  // W goes through LDS in two 32-column blocks per chunk; a block's loads
  // are issued a block or more ahead (before the conv inputs of the next
  // chunk, so that waiting for them never waits for those)
  const int Kw = (p.K + 7) & ~7;
  const __amdgpu_buffer_rsrc_t wres = make_rsrc(Ws, (uint32_t)__builtin_amdgcn_readfirstlane(3 * p.N * ldws * 2));
  Stage st0, st1;
  st0.load(wres, tid, 0, p.N, ldws, Kw, 0);

  // rows of this wavefront: wb .. wb + 31. p0 = position of row wb in its
  // program (clamped to 3); bit r of `starts` (r >= 1): row wb + r is a
  // program's first row
  const int wb = row0 + wave * 32;
  int tp = 3;
  if (lane < 32 && wb + lane < M) tp = min((int)cv.tpos[wb + lane], 3);
  const uint32_t p0 = (uint32_t)__builtin_amdgcn_readfirstlane(tp);
  const uint32_t starts = (uint32_t)__builtin_amdgcn_ballot_w64(lane >= 1 && lane < 32 && tp == 0);
  // conv input rows max(row0 - 3, 0) .. min(M, row0 + BM) - 1: a row before
  // the first or past the last reads zero through the resource
  const int xr0 = max(row0 - 3, 0);
  const int xrows = min(M, row0 + BM) - xr0;
  // (XB: x channel-blocked, each chunk's rows contiguous at 256 bytes a row)
  const __amdgpu_buffer_rsrc_t xres =
      make_rsrc(cv.x + (int64_t)xr0 * (XB ? 64 : cv.ldx), (uint32_t)(xrows * (XB ? 64 : cv.ldx) * 4));
  const __amdgpu_buffer_rsrc_t ures = make_rsrc(cv.u + (int64_t)row0 * E, (uint32_t)(min(BM, M - row0) * E * 4));
  const __amdgpu_buffer_rsrc_t cwres = make_rsrc(cv.w, (uint32_t)(E * 4 * 4));
  const __amdgpu_buffer_rsrc_t cbres = make_rsrc(cv.b, (uint32_t)(E * 4));

  const uint32_t ldx4 = (uint32_t)(cv.ldx * 4);
  uint32_t xw[XR];
  u32x4 cw;
  uint32_t cb;
  auto load_chunk = [&](int c) {
    const uint32_t e = c * CW + lane;
    const uint32_t ve = opaque_v(e * 4);
    const uint32_t ld = opaque_s(XB ? 256u : ldx4), vx = XB ? opaque_v((uint32_t)lane * 4) : ve;
    const __amdgpu_buffer_rsrc_t xr =
        XB ? make_rsrc(cv.x + ((int64_t)c * cv.xblk_rows + xr0) * 64, (uint32_t)(xrows * 64 * 4)) : xres;
#pragma unroll
    for (int i = 0; i < XR; ++i) {
      const int row = wb - 3 + i;
      const uint32_t off = row >= 0 ? (uint32_t)(row - xr0) * ld + vx : kOutOfRange;
      xw[i] = __builtin_amdgcn_raw_buffer_load_b32(xr, off, 0, 0);
    }
    cw = __builtin_amdgcn_raw_buffer_load_b128(cwres, ve * 4, 0, 0);
    cb = __builtin_amdgcn_raw_buffer_load_b32(cbres, ve, 0, 0);
  };
  load_chunk(0);

  floatx16 acc[2];
#pragma unroll
  for (int nb = 0; nb < 2; ++nb)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[nb][r] = 0.f;
  st0.stage(&sW[0], tid);

  float* myA = &sA[wave * 32 * PA];
#pragma unroll
  for (int c = 0; c < KCH; ++c) {
    __builtin_amdgcn_sched_barrier(0);
    // W of this chunk's second block and of the next chunk's first
    st1.load(wres, tid, 32, p.N, ldws, Kw, c * CW);
    if (c + 1 < KCH) st0.load(wres, tid, 0, p.N, ldws, Kw, (c + 1) * CW);
    // conv + SiLU of rows wb .. wb + 31 at channel c CW + lane, parked in LDS
    {
      const float w0 = __uint_as_float(cw.x), w1 = __uint_as_float(cw.y), w2 = __uint_as_float(cw.z),
                  w3 = __uint_as_float(cw.w), bias = __uint_as_float(cb);
      const uint32_t pc = opaque_s(p0), sc = opaque_s(starts);
      // the rows before the wavefront's first row that lie in an earlier program
      if (pc < 3) xw[0] = 0u;
      if (pc < 2) xw[1] = 0u;
      if (pc < 1) xw[2] = 0u;
#pragma unroll
      for (int r = 0; r < 32; ++r) {
        // row wb + r starts a program: the three rows before it are no
        // longer anyone's taps
        if (r > 0 && ((sc >> r) & 1u)) xw[r] = xw[r + 1] = xw[r + 2] = 0u;
        float a = bias;
        a = fmaf(w0, __uint_as_float(xw[r]), a);
        a = fmaf(w1, __uint_as_float(xw[r + 1]), a);
        a = fmaf(w2, __uint_as_float(xw[r + 2]), a);
        a = fmaf(w3, __uint_as_float(xw[r + 3]), a);
        myA[r * PA + lane] = silu(a);
      }
    }
    // the next chunk's conv inputs load while this chunk's MFMAs run
    if (c + 1 < KCH) load_chunk(c + 1);
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    // u: the parked rows stored 16 bytes per lane (four rows per instruction)
    {
      const uint32_t uo = opaque_v((uint32_t)((wave * 32 + (lane >> 4)) * E + c * CW + 4 * (lane & 15)) * 4);
      const uint32_t ur = opaque_s((uint32_t)E * 16);
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const u32x4 v = *reinterpret_cast<const u32x4*>(&myA[(4 * i + (lane >> 4)) * PA + 4 * (lane & 15)]);
        __builtin_amdgcn_raw_buffer_store_b128(v, ures, uo + i * ur, 0, 0);
      }
    }
    bf16x8 a1[NS], a2[NS], a3[NS];
#pragma unroll
    for (int s2 = 0; s2 < NS; ++s2) {
      const float* ap = &myA[li * PA + 16 * s2 + 8 * lg];
      split8(*reinterpret_cast<const floatx4*>(ap), *reinterpret_cast<const floatx4*>(ap + 4), a1[s2], a2[s2],
             a3[s2]);
    }
    // every lane's reads of the parked rows are done before the next chunk's rows are parked
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
    for (int nb = 0; nb < 2; ++nb) {
      const int buf = (c * 2 + nb) & 1;
      __syncthreads();  // this block visible; the other buffer is free for the next
      const bool more = nb == 0 || c + 1 < KCH;
      const uint16_t* wbp = &sW[buf * 3 * PART + li * WP + 8 * lg];
      auto wfrag = [&](int part, int ks) {
        return __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(wbp + part * PART + 16 * ks));
      };
      bf16x8 q[2][3];
#pragma unroll
      for (int j = 0; j < 3; ++j) q[0][j] = wfrag(j, 0);
      __builtin_amdgcn_sched_group_barrier(0x0100, 3, 0);
#pragma unroll
      for (int ks = 0; ks < NS; ++ks) {
        if (ks + 1 < NS) {
#pragma unroll
          for (int j = 0; j < 3; ++j) q[(ks + 1) & 1][j] = wfrag(j, ks + 1);
        }
        const bf16x8* w = q[ks & 1];
        acc[nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a3[ks], w[0], acc[nb], 0, 0, 0);
        acc[nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a2[ks], w[1], acc[nb], 0, 0, 0);
        acc[nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1[ks], w[2], acc[nb], 0, 0, 0);
        acc[nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a2[ks], w[0], acc[nb], 0, 0, 0);
        acc[nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1[ks], w[1], acc[nb], 0, 0, 0);
        acc[nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1[ks], w[0], acc[nb], 0, 0, 0);
        if (ks + 1 < NS) __builtin_amdgcn_sched_group_barrier(0x0100, 3, 0);
        __builtin_amdgcn_sched_group_barrier(0x0008, 6, 0);
        if (ks == NS / 2 && more) {
          if (nb == 0) st1.stage(&sW[(buf ^ 1) * 3 * PART], tid);
          else st0.stage(&sW[(buf ^ 1) * 3 * PART], tid);
          __builtin_amdgcn_sched_group_barrier(0x0200, Stage::NW, 0);
        }
      }
    }
  }

  // epilogue: lane l holds column nb*32 + l % 32 and rows 8*(r/4) + 4*(l/32) + (r%4)
  const __amdgpu_buffer_rsrc_t cres =
      make_rsrc(p.C + (int64_t)row0 * p.ldc, (uint32_t)(min(BM, M - row0) * p.ldc * 4));
#pragma unroll
  for (int nb = 0; nb < 2; ++nb) {
    const int col = nb * 32 + li;
    const bool cok = col < p.N;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int rl = 8 * (r >> 2) + 4 * lg + (r & 3);
      const uint32_t off = cok ? (uint32_t)(((wave * 32 + rl) * p.ldc + col) * 4) : kOutOfRange;
      // (a bit cast straight from the vector element would read element 0)
      __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(acc[nb][r]), cres, off, 0, 0);
    }
  }
}

template <int FL>
hipError_t launch32(const GemmArgs& a, const uint16_t* Ws, int ldws, hipStream_t s) {
  const int grid = (a.Mmax + kWaves * 32 - 1) / (kWaves * 32);
  if (grid <= 0) return hipSuccess;
#define TCL_SPLIT32(KC)                                                                            \
  hipLaunchKernelGGL((gemm_split32_kernel<KC, FL>), dim3(grid), dim3(kWaves * 64), 0, s, a, Ws, ldws); \
  break
  switch ((a.K + 63) / 64) {
    case 1: TCL_SPLIT32(1);
    case 2: TCL_SPLIT32(2);
    case 3: TCL_SPLIT32(3);
    case 4: TCL_SPLIT32(4);
    default: return hipErrorInvalidValue;
  }
#undef TCL_SPLIT32
  return hipGetLastError();
}

template <int FL>
hipError_t launch32h(const GemmArgs& a, const uint16_t* Ws, int ldws, hipStream_t s) {
  const int grid = (a.Mmax + 127) / 128;
  if (grid <= 0) return hipSuccess;
  // a batch with fewer panels than two per CU also splits the columns, up to
  // 8 ways (each workgroup repeats the short A prologue of its panel)
  const int nblk = (a.N + 31) / 32;
  const int cs = std::max(1, std::min({8, nblk, 512 / grid}));
  const dim3 g(grid, cs);
  switch ((a.K + 127) / 128) {
    case 1: hipLaunchKernelGGL((gemm_split32h_kernel<1, FL>), g, dim3(kWavesH * 64), 0, s, a, Ws, ldws); break;
    case 2: hipLaunchKernelGGL((gemm_split32h_kernel<2, FL>), g, dim3(kWavesH * 64), 0, s, a, Ws, ldws); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <int FL>
hipError_t launch16(const GemmArgs& a, const uint16_t* Ws, int ldws, hipStream_t s) {
  const int grid = (a.Mmax + kWaves * 16 - 1) / (kWaves * 16);
  if (grid <= 0) return hipSuccess;
#define TCL_SPLIT16(KC)                                                                            \
  hipLaunchKernelGGL((gemm_split16_kernel<KC, FL>), dim3(grid), dim3(kWaves * 64), 0, s, a, Ws, ldws); \
  break
  switch ((a.K + 63) / 64) {
    case 1: TCL_SPLIT16(1);
    case 2: TCL_SPLIT16(2);
    case 4: TCL_SPLIT16(4);
    case 8: TCL_SPLIT16(8);
    default: return hipErrorInvalidValue;
  }
#undef TCL_SPLIT16
  return hipGetLastError();
}

template <int KC, int KCH, int FL>
hipError_t launch32acc_nb(const GemmArgs& a, const uint16_t* Ws, int ldws, int grid, hipStream_t s) {
  const int nb = (a.N + 31) / 32;
  // a batch with fewer panels than two per CU splits the columns over 2 or
  // 4 workgroups per panel (each repeats its panel's A chunks)
  const int cs = 512 / grid >= 4 ? 4 : 512 / grid >= 2 ? 2 : 1;
#define TCL_SPLIT32ACC(NB, CS)                                                                           \
  hipLaunchKernelGGL((gemm_split32acc_kernel<KC, KCH, NB, FL>), dim3(grid, CS), dim3(kWaves * 64), 0, s, a, \
                     Ws, ldws)
  if (nb <= 2) TCL_SPLIT32ACC(2, 1);
  else if (nb <= 4) {
    if (cs >= 2) TCL_SPLIT32ACC(2, 2);
    else TCL_SPLIT32ACC(4, 1);
  } else if (nb <= 8) {
    if (cs >= 4) TCL_SPLIT32ACC(2, 4);
    else if (cs == 2) TCL_SPLIT32ACC(4, 2);
    else TCL_SPLIT32ACC(8, 1);
  } else return hipErrorInvalidValue;
#undef TCL_SPLIT32ACC
  return hipGetLastError();
}

template <int FL>
hipError_t launch32acc(const GemmArgs& a, const uint16_t* Ws, int ldws, hipStream_t s) {
  const int grid = (a.Mmax + kWaves * 32 - 1) / (kWaves * 32);
  if (grid <= 0) return hipSuccess;
  switch ((a.K + 63) / 64) {
    case 1: return launch32acc_nb<1, 1, FL>(a, Ws, ldws, grid, s);
    case 2: return launch32acc_nb<2, 1, FL>(a, Ws, ldws, grid, s);
    case 3: return launch32acc_nb<3, 1, FL>(a, Ws, ldws, grid, s);
    case 4: return launch32acc_nb<4, 1, FL>(a, Ws, ldws, grid, s);
    // K > 256: chunks of 128 (A's parts of a 256-k chunk, 128 accumulators
    // and the W stage's registers would not fit together)
    case 5: case 6: return launch32acc_nb<2, 3, FL>(a, Ws, ldws, grid, s);
    case 7: case 8: return launch32acc_nb<2, 4, FL>(a, Ws, ldws, grid, s);
    default: return hipErrorInvalidValue;
  }
}

// W -> its three bf16 parts, [3][N][ldw], the padding k >= K zero
__global__ __launch_bounds__(256) void split_weights_kernel(const float* __restrict__ W, int N, int K,
                                                            int ldw, uint16_t* __restrict__ out) {
  const int64_t n_all = (int64_t)N * ldw;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n_all; i += (int64_t)gridDim.x * 256) {
    const int n = (int)(i / ldw), k = (int)(i % ldw);
    const float v = k < K ? W[(int64_t)n * K + k] : 0.f;
    uint32_t h, m, l;
    split3_pair(v, 0.f, h, m, l);
    out[i] = (uint16_t)h;
    out[n_all + i] = (uint16_t)m;
    out[2 * n_all + i] = (uint16_t)l;
  }
}

}  // namespace

bool gemm_split_supports(const GemmArgs& a, int flags, int variant) {
  const bool al = a.K % 4 == 0 && a.lda % 4 == 0 && reinterpret_cast<uintptr_t>(a.A) % 16 == 0 &&
                  // byte offsets of the buffer resources stay below 2^31
                  (int64_t)3 * a.N * ((a.K + 7) & ~7) * 2 < (1ll << 31) &&
                  (int64_t)kWaves * 32 * a.ldc * 4 < (1ll << 31);
  if (!al || a.K < 1) return false;
  const int kc = (a.K + 63) / 64;
  const bool plain = (flags & (kRowNorm | kGather)) == 0;
  switch (variant) {
    case kSplit32: return (flags & kResid) == 0 && kc <= 4;
    case kSplit32H: return (flags & kResid) == 0 && kc <= 4 && (int64_t)128 * a.ldc * 4 < (1ll << 31);
    case kSplit16: return plain && (kc == 1 || kc == 2 || kc == 4 || kc == 8);
    case kSplit32Acc: return plain && kc <= 8 && a.N <= 256;
    default: return false;
  }
}

int gemm_split_variant(const GemmArgs& a, int flags) {
  // 32-row panels first (half the LDS traffic per flop of 16-row ones);
  // streaming N blocks when K fits one chunk, else all of N in registers
  // K in (192, 256]: the K halves on two wavefronts per SIMD (measured on
  // MI355X for in_proj, 61,715 x 1024 x 256 with the RMSNorm: 17% faster than
  // one wavefront per row group); below that the upper half would be mostly
  // padding (the input Linear, K = 164: 12% slower)
  if ((a.K + 63) / 64 == 4 && gemm_split_supports(a, flags, kSplit32H)) return kSplit32H;
  if ((flags & kResid) == 0 && gemm_split_supports(a, flags, kSplit32)) return kSplit32;
  if (gemm_split_supports(a, flags, kSplit32Acc)) return kSplit32Acc;
  if (gemm_split_supports(a, flags, kSplit16)) return kSplit16;
  return -1;
}

hipError_t launch_gemm_split(const GemmArgs& a, const uint16_t* Ws, int ldws, int flags, int variant,
                             hipStream_t s) {
  if (variant < 0) variant = gemm_split_variant(a, flags);
  if (!gemm_split_supports(a, flags, variant)) return hipErrorInvalidValue;
  if (variant == kSplit32Acc) {
    switch (flags) {
      case 0: return launch32acc<0>(a, Ws, ldws, s);
      case kBias: return launch32acc<kBias>(a, Ws, ldws, s);
      case kResid: return launch32acc<kResid>(a, Ws, ldws, s);
      default: return hipErrorInvalidValue;
    }
  }
  if (variant == kSplit32H) {
    switch (flags) {
      case 0: return launch32h<0>(a, Ws, ldws, s);
      case kBias: return launch32h<kBias>(a, Ws, ldws, s);
      case kRowNorm: return launch32h<kRowNorm>(a, Ws, ldws, s);
      case kBias | kGather: return launch32h<kBias | kGather>(a, Ws, ldws, s);
      default: return hipErrorInvalidValue;
    }
  }
  if (variant == kSplit32) {
    switch (flags) {
      case 0: return launch32<0>(a, Ws, ldws, s);
      case kBias: return launch32<kBias>(a, Ws, ldws, s);
      case kRowNorm: return launch32<kRowNorm>(a, Ws, ldws, s);
      case kBias | kGather: return launch32<kBias | kGather>(a, Ws, ldws, s);
      default: return hipErrorInvalidValue;
    }
  }
  if (variant == kSplit16) {
    switch (flags) {
      case 0: return launch16<0>(a, Ws, ldws, s);
      case kBias: return launch16<kBias>(a, Ws, ldws, s);
      case kResid: return launch16<kResid>(a, Ws, ldws, s);
      default: return hipErrorInvalidValue;
    }
  }
  return hipErrorInvalidValue;
}

bool gemm_split_conv_supports(const GemmArgs& a, const ConvIn& cv, int d_conv) {
  const auto a16 = [](const void* q) { return reinterpret_cast<uintptr_t>(q) % 16 == 0; };
  const bool xin = cv.xblk_rows > 0 ? cv.xblk_rows >= a.Mmax
                                    : cv.ldx % 4 == 0 && cv.ldx >= a.K &&
                                          (int64_t)(kWaves * 32 + 3) * cv.ldx * 4 < (1ll << 31);
  return d_conv == 4 && !a.relu && a.K % 64 == 0 && a.K >= 64 && a.K <= 512 && a.N >= 1 && a.N <= 64 && cv.x && cv.w &&
         cv.b && cv.tpos && cv.u && a16(cv.x) && a16(cv.w) && a16(cv.u) && xin &&
         // byte offsets of the buffer resources stay below 2^31
         (int64_t)kWaves * 32 * a.K * 4 < (1ll << 31) && (int64_t)kWaves * 32 * a.ldc * 4 < (1ll << 31) &&
         (int64_t)3 * a.N * ((a.K + 7) & ~7) * 2 < (1ll << 31);
}

hipError_t launch_gemm_split_conv(const GemmArgs& a, const ConvIn& cv, const uint16_t* Ws, int ldws, hipStream_t s) {
  if (!gemm_split_conv_supports(a, cv, 4)) return hipErrorInvalidValue;
  const int grid = (a.Mmax + kWaves * 32 - 1) / (kWaves * 32);
  if (grid <= 0) return hipSuccess;
#define TCL_SPLITCONV(KCH)                                                                                    \
  if (cv.xblk_rows > 0)                                                                                     \
    hipLaunchKernelGGL((gemm_split32conv_kernel<KCH, true>), dim3(grid), dim3(kWaves * 64), 0, s, a, cv, Ws, ldws); \
  else                                                                                                      \
    hipLaunchKernelGGL((gemm_split32conv_kernel<KCH, false>), dim3(grid), dim3(kWaves * 64), 0, s, a, cv, Ws, ldws)
  switch (a.K / 64) {
    case 1: TCL_SPLITCONV(1); break;
    case 2: TCL_SPLITCONV(2); break;
    case 3: TCL_SPLITCONV(3); break;
    case 4: TCL_SPLITCONV(4); break;
    case 5: TCL_SPLITCONV(5); break;
    case 6: TCL_SPLITCONV(6); break;
    case 7: TCL_SPLITCONV(7); break;
    case 8: TCL_SPLITCONV(8); break;
    default: return hipErrorInvalidValue;
  }
#undef TCL_SPLITCONV
  return hipGetLastError();
}

hipError_t launch_split_weights(const float* W, int N, int K, int ldw, uint16_t* out, hipStream_t s) {
  if (N <= 0 || K <= 0 || ldw < K) return hipErrorInvalidValue;
  const int64_t n_all = (int64_t)N * ldw;
  const int grid = (int)std::min<int64_t>((n_all + 255) / 256, 4096);
  hipLaunchKernelGGL(split_weights_kernel, dim3(grid), dim3(256), 0, s, W, N, K, ldw, out);
  return hipGetLastError();
}

}  // namespace tcl
