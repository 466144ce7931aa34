// fp32 projections on the gfx950 matrix cores (v_mfma_f32_32x32x2_f32).
//
// C = A W^T with both operands K-contiguous (activations are row-major
// [tokens, K]; weights keep the [out, in] layout). A workgroup computes a
// BM x BN tile; each wavefront owns a (TM*32) x (TN*32) sub-tile made of
// 32x32 MFMA blocks with their accumulators in registers. K is consumed in
// chunks of 32 staged through LDS; the next chunk's global loads are issued
// before the current chunk's MFMAs so that their latency overlaps compute.
//
// Operand k-order: v_mfma_f32_32x32x2_f32 multiplies A[32x2] by B[2x32];
// lane l supplies row (l % 32) of A and column (l % 32) of B at the k
// index (l / 32). The sum over k does not depend on which k each step
// uses, so lane half g = l/32 walks k = 16g .. 16g+15 of the chunk while
// lane half 0 walks k = 0..15: each lane then reads 16 contiguous floats
// of its row with four 128-bit LDS loads instead of 16 scalar loads.
//
// Tile order is XCD-aware: workgroup i runs on XCD i % 8, and the mapping
// below gives each XCD a stripe of M-tiles whose N-tiles it walks in
// order, so the A rows of a tile are fetched into that XCD's L2 once.
#include "common.h"
#include "kernels.h"

namespace tcl {
namespace {

// Occupancy target: 3 wavefronts per SIMD for K chunks of 32 (the register
// file then holds three workgroups' tiles), 2 for chunks of 64.
template <int WM, int WN, int TM, int TN, int BK, int FL>
__global__ __launch_bounds__(WM* WN * 64, BK == 32 ? 3 : 2) void gemm_f32_kernel(GemmArgs p, int ntm,
                                                                                 int ntn) {
  // BK + 4 floats per LDS row: 144- or 272-byte rows keep 8 lanes of b128 reads conflict-free
  constexpr int PITCH = BK + 4;
  constexpr int Q = BK / 4;        // float4 per row chunk
  constexpr int KH = BK / 2;       // k per lane half within a chunk
  constexpr int NT = WM * WN * 64;
  constexpr int BM = WM * TM * 32;
  constexpr int BN = WN * TN * 32;
  constexpr int NA = BM * Q / NT;
  constexpr int NB = BN * Q / NT;
  static_assert((BM * Q) % NT == 0 && (BN * Q) % NT == 0, "tile/thread mismatch");
  static_assert(NT % Q == 0, "k offset must be thread-invariant");
  constexpr bool kNorm = (FL & kRowNorm) != 0;

  __shared__ __attribute__((aligned(16))) float sA[BM * PITCH];
  __shared__ __attribute__((aligned(16))) float sB[BN * PITCH];
  __shared__ float sR[kNorm ? BM : 1];

  const int tid = threadIdx.x;
  const int M = p.Mdev ? *p.Mdev : p.Mmax;

  const int bid = blockIdx.x;
  const int xcd = bid & 7, j = bid >> 3;
  const int mt = xcd + 8 * (j / ntn), nt = j % ntn;
  if (mt >= ntm) return;
  const int row0 = mt * BM;
  if (row0 >= M) return;
  const int col0 = nt * BN;

  const int q4 = (tid % Q) * 4;  // k offset of this thread's float4 within a chunk

  const float* aptr[NA];
  bool aval[NA];
#pragma unroll
  for (int i = 0; i < NA; ++i) {
    const int r = (tid + i * NT) / Q;
    const int grow = row0 + r;
    aval[i] = grow < M;
    int64_t src = grow;
    if constexpr ((FL & kGather) != 0) {
      if (aval[i]) {
        int lo = 0, hi = p.B;  // largest b with offs[b] <= grow
        while (hi - lo > 1) {
          const int mid = (lo + hi) >> 1;
          if (p.offs[mid] <= grow) lo = mid; else hi = mid;
        }
        src = (int64_t)lo * p.L + (grow - p.offs[lo]);
      }
    }
    aptr[i] = p.A + (aval[i] ? src : 0) * p.lda + q4;
  }
  const float* bptr[NB];
  bool bval[NB];
#pragma unroll
  for (int i = 0; i < NB; ++i) {
    const int n = col0 + (tid + i * NT) / Q;
    bval[i] = n < p.N;
    bptr[i] = p.W + (bval[i] ? (int64_t)n : 0) * p.ldw + q4;
  }

  floatx4 ra[NA], rb[NB];
  float ss[NA];
#pragma unroll
  for (int i = 0; i < NA; ++i) ss[i] = 0.f;

  // Loads go to clamped in-bounds addresses (no branch per load); units
  // outside A, W or K are zeroed when staged, and the RMSNorm sum of squares
  // is taken there too, so nothing waits for a load before the MFMAs that
  // should hide it.
  auto gload = [&](int k0) {
    const bool kin = k0 + q4 < p.K;  // K % 4 == 0: a float4 is all in or all out
#pragma unroll
    for (int i = 0; i < NA; ++i) ra[i] = *reinterpret_cast<const floatx4*>(aptr[i] + (kin ? k0 : 0));
#pragma unroll
    for (int i = 0; i < NB; ++i) rb[i] = *reinterpret_cast<const floatx4*>(bptr[i] + (kin ? k0 : 0));
  };

  const int wave = tid >> 6, lane = tid & 63;
  const int wm = wave / WN, wn = wave % WN;
  const int li = lane & 31, lg = lane >> 5;

  floatx16 acc[TM][TN];
#pragma unroll
  for (int a = 0; a < TM; ++a)
#pragma unroll
    for (int b = 0; b < TN; ++b)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[a][b][r] = 0.f;

  gload(0);
  for (int k0 = 0; k0 < p.K; k0 += BK) {
    __syncthreads();
    const bool kin = k0 + q4 < p.K;
#pragma unroll
    for (int i = 0; i < NA; ++i) {
      const int r = (tid + i * NT) / Q;
      const floatx4 v = (aval[i] && kin) ? ra[i] : floatx4{0.f, 0.f, 0.f, 0.f};
      if constexpr (kNorm) ss[i] += v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
      *reinterpret_cast<floatx4*>(&sA[r * PITCH + q4]) = v;
    }
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      const int r = (tid + i * NT) / Q;
      *reinterpret_cast<floatx4*>(&sB[r * PITCH + q4]) =
          (bval[i] && kin) ? rb[i] : floatx4{0.f, 0.f, 0.f, 0.f};
    }
    __syncthreads();
    if (k0 + BK < p.K) gload(k0 + BK);

    // fragments are read four k at a time, just ahead of the MFMAs that use them
    const float* srcA = &sA[(wm * TM * 32 + li) * PITCH + lg * KH];
    const float* srcB = &sB[(wn * TN * 32 + li) * PITCH + lg * KH];
#pragma unroll
    for (int c = 0; c < KH / 4; ++c) {
      floatx4 a4[TM], b4[TN];
#pragma unroll
      for (int a = 0; a < TM; ++a) a4[a] = *reinterpret_cast<const floatx4*>(srcA + a * 32 * PITCH + 4 * c);
#pragma unroll
      for (int b = 0; b < TN; ++b) b4[b] = *reinterpret_cast<const floatx4*>(srcB + b * 32 * PITCH + 4 * c);
#pragma unroll
      for (int e = 0; e < 4; ++e)
#pragma unroll
        for (int a = 0; a < TM; ++a)
#pragma unroll
          for (int b = 0; b < TN; ++b)
            acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x2f32(a4[a][e], b4[b][e], acc[a][b], 0, 0, 0);
    }
  }

  if constexpr (kNorm) {
    // the Q threads that loaded a row's k-slices are adjacent lanes
#pragma unroll
    for (int i = 0; i < NA; ++i) {
      float v = ss[i];
#pragma unroll
      for (int o = 1; o < Q; o <<= 1) v += __shfl_xor(v, o, 64);
      if ((tid % Q) == 0) {
        const int r = (tid + i * NT) / Q;
        sR[r] = 1.0f / sqrtf(v / (float)p.K + p.eps);
      }
    }
    __syncthreads();
  }

  // Accumulator layout of a 32x32 block: lane l holds column l % 32 and rows
  // 8*(r/4) + 4*(l/32) + (r%4) for r = 0..15. With a residual, every block's
  // residuals are loaded before the first store (C may be read in place, so
  // loads cannot move past earlier stores, and each would wait for them).
  float res[(FL & kResid) != 0 ? TM : 1][(FL & kResid) != 0 ? TN : 1][16];
  if constexpr ((FL & kResid) != 0) {
    const float* R = p.R ? p.R : p.C;
#pragma unroll
    for (int a = 0; a < TM; ++a)
#pragma unroll
      for (int b = 0; b < TN; ++b) {
        const int col = col0 + wn * TN * 32 + b * 32 + li;
        const bool cok = col < p.N;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int row = row0 + wm * TM * 32 + a * 32 + 8 * (r >> 2) + 4 * lg + (r & 3);
          res[a][b][r] = (cok && row < M) ? R[(int64_t)row * p.ldc + col] : 0.f;
        }
      }
  }
#pragma unroll
  for (int a = 0; a < TM; ++a) {
#pragma unroll
    for (int b = 0; b < TN; ++b) {
      const int col = col0 + wn * TN * 32 + b * 32 + li;
      const bool cok = col < p.N;
      if (!cok) continue;
      const float bias = (FL & kBias) ? p.bias[col] : 0.f;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int rl = wm * TM * 32 + a * 32 + 8 * (r >> 2) + 4 * lg + (r & 3);
        const int row = row0 + rl;
        if (row >= M) continue;
        float v = acc[a][b][r];
        if constexpr (kNorm) v *= sR[rl];
        v += bias;
        if constexpr ((FL & kResid) != 0) v += res[a][b][r];
        if (p.relu) v = fmaxf(v, 0.f);
        p.C[(int64_t)row * p.ldc + col] = v;
      }
    }
  }
}

template <int WM, int WN, int TM, int TN, int BK, int FL>
hipError_t launch_t(const GemmArgs& a, hipStream_t s) {
  constexpr int BM = WM * TM * 32, BN = WN * TN * 32;
  const int ntm = (a.Mmax + BM - 1) / BM;
  const int ntn = (a.N + BN - 1) / BN;
  const int grid = 8 * ntn * ((ntm + 7) / 8);
  if (grid <= 0) return hipSuccess;
  hipLaunchKernelGGL((gemm_f32_kernel<WM, WN, TM, TN, BK, FL>), dim3(grid), dim3(WM * WN * 64), 0, s,
                     a, ntm, ntn);
  return hipGetLastError();
}

template <int WM, int WN, int TM, int TN, int BK>
hipError_t dispatch_flags(const GemmArgs& a, int flags, hipStream_t s) {
  switch (flags) {
    case 0: return launch_t<WM, WN, TM, TN, BK, 0>(a, s);
    case kBias: return launch_t<WM, WN, TM, TN, BK, kBias>(a, s);
    case kResid: return launch_t<WM, WN, TM, TN, BK, kResid>(a, s);
    case kRowNorm: return launch_t<WM, WN, TM, TN, BK, kRowNorm>(a, s);
    case kBias | kGather: return launch_t<WM, WN, TM, TN, BK, kBias | kGather>(a, s);
    default: return hipErrorInvalidValue;
  }
}

constexpr int kPanelMinRows = 32768;

}  // namespace

GemmTile pick_gemm_f32_tile(const GemmArgs& a, int flags) {
  // Measured on MI355X with the model's epilogues (fp32 MFMA, TFLOP/s, three
  // wavefronts per SIMD): at ~62K rows 64x128 tiles win (in_proj with the
  // RMSNorm prologue 104 vs 98 for 128x128; out_proj with the residual 100 vs
  // 78), because the last partial round of workgroups is shorter; the
  // gathered input Linear (K = 164) prefers 128x128 with K chunks of 64
  // (81 vs 67). At ~1.3M rows 128x128 is best for in_proj (115) and 64x128
  // for out_proj (113). Row panels replace the tiles once there are enough
  // rows to give every CU two panels: in_proj 117 (B = 4096) and 127
  // (L = 256) TFLOP/s, the input Linear 97; 16-row panels for out_proj 106
  // and 114, and for x_proj (N = 48) 72 and 81 against 62 and 65 for 64x64.
  const int Mmax = a.Mmax, N = a.N, K = a.K;
  if (Mmax >= kPanelMinRows && gemm_f32_panel_fits(a, flags)) return kPanel;
  if (Mmax >= kPanelMinRows && gemm_f32_panel16_fits(a, flags)) return kPanel16;
  if (N <= 64) return kNarrow;
  if (K % 64 != 0) return Mmax >= 500000 ? kWide : kTile128x128K64;
  if (Mmax >= 500000 && N >= 1024) return kWide;
  return kTile64x128;
}

hipError_t launch_gemm_f32(const GemmArgs& a, int flags, int tile_id, hipStream_t s) {
  const GemmTile tile = tile_id < 0 ? pick_gemm_f32_tile(a, flags) : static_cast<GemmTile>(tile_id);
  if (tile == kPanel) {
    if (!gemm_f32_panel_fits(a, flags)) return hipErrorInvalidValue;
    return launch_gemm_f32_panel(a, flags, s);
  }
  if (tile == kPanel16) {
    if (!gemm_f32_panel16_fits(a, flags)) return hipErrorInvalidValue;
    return launch_gemm_f32_panel16(a, flags, s);
  }
  switch (tile) {
    case kWide: return dispatch_flags<2, 2, 2, 2, 32>(a, flags, s);
    case kNarrow: return dispatch_flags<2, 2, 1, 1, 32>(a, flags, s);
    case kTile64x128: return dispatch_flags<2, 2, 1, 2, 32>(a, flags, s);
    case kTile128x64: return dispatch_flags<2, 2, 2, 1, 32>(a, flags, s);
    case kTile128x256: return dispatch_flags<2, 4, 2, 2, 32>(a, flags, s);
    case kTile128x128K64: return dispatch_flags<2, 2, 2, 2, 64>(a, flags, s);
    case kTile64x128K64: return dispatch_flags<2, 2, 1, 2, 64>(a, flags, s);
    case kTile128x64K64: return dispatch_flags<2, 2, 2, 1, 64>(a, flags, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace tcl
