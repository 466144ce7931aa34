// bf16 projections on the gfx950 matrix cores (v_mfma_f32_32x32x16_bf16),
// fp32 accumulation.
//
// Same structure as the fp32 GEMM: C = A W^T, K-contiguous operands, a
// workgroup tile of (WM*TM*32) x (WN*TN*32) built from 32x32 MFMA blocks
// held in registers, K staged through LDS in chunks of 64, next chunk's
// global loads issued before the current chunk's MFMAs, XCD-aware tile
// order. The A operand may be fp32 (the residual stream or the input
// features; converted to bf16, round-to-nearest-even, as it is staged -- with
// the RMSNorm gain applied first when kRowNorm is set) or bf16 (activations
// written by earlier kernels). W is bf16, zero-padded to a multiple of 8 in
// K. C is fp32 or bf16.
//
// Operand k-order: lane l of v_mfma_f32_32x32x16_bf16 supplies 8
// consecutive k of row (l % 32) in intrinsic positions 8*(l/32)..+7. Within
// a 64-wide chunk, lane half g takes k = 32g + 8j .. +7 in MFMA j (j=0..3),
// for A and W alike, so each lane reads its 32 contiguous bf16 with four
// 128-bit LDS loads.
#include "common.h"
#include "kernels.h"

namespace tcl {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int BK = 64;          // k per chunk (bf16 elements)
constexpr int PITCH = BK + 8;   // bf16 per LDS row: 144 bytes, conflict-free 8-lane b128 reads
constexpr int Q = BK / 8;       // 16-byte units per row chunk

__device__ __forceinline__ uint32_t pack2(float a, float b) { return f32x2_to_bf16x2(a, b); }

template <typename TA, typename TC, int WM, int WN, int TM, int TN, int FL>
__global__ __launch_bounds__(WM* WN * 64) void gemm_bf16_kernel(GemmArgsBF16 p, int ntm, int ntn) {
  constexpr int NT = WM * WN * 64;
  constexpr int BM = WM * TM * 32;
  constexpr int BN = WN * TN * 32;
  constexpr int NA = BM * Q / NT;
  constexpr int NB = BN * Q / NT;
  static_assert((BM * Q) % NT == 0 && (BN * Q) % NT == 0, "tile/thread mismatch");
  static_assert(NT % Q == 0, "k offset must be thread-invariant");
  constexpr bool kF32A = sizeof(TA) == 4;
  constexpr bool kNorm = (FL & kRowNorm) != 0;
  static_assert(!kNorm || kF32A, "RMSNorm prologue needs the fp32 residual stream");

  __shared__ __attribute__((aligned(16))) uint16_t sA[BM * PITCH];
  __shared__ __attribute__((aligned(16))) uint16_t sB[BN * PITCH];
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
  const int q8 = (tid % Q) * 8;  // k offset (elements) of this thread's unit within a chunk
  const int Kw = (p.K + 7) & ~7; // W is zero-padded to here

  const TA* aptr[NA];
  bool aval[NA];
#pragma unroll
  for (int i = 0; i < NA; ++i) {
    const int r = (tid + i * NT) / Q;
    const int grow = row0 + r;
    aval[i] = grow < M;
    int64_t src = grow;
    if constexpr ((FL & kGather) != 0) {
      if (aval[i]) {
        int lo = 0, hi = p.B;
        while (hi - lo > 1) {
          const int mid = (lo + hi) >> 1;
          if (p.offs[mid] <= grow) lo = mid; else hi = mid;
        }
        src = (int64_t)lo * p.L + (grow - p.offs[lo]);
      }
    }
    aptr[i] = reinterpret_cast<const TA*>(p.A) + (aval[i] ? src : 0) * p.lda + q8;
  }
  const uint16_t* bptr[NB];
  bool bval[NB];
#pragma unroll
  for (int i = 0; i < NB; ++i) {
    const int n = col0 + (tid + i * NT) / Q;
    bval[i] = n < p.N;
    bptr[i] = p.W + (bval[i] ? (int64_t)n : 0) * p.ldw + q8;
  }

  u32x4 ra[NA], rb[NB];
  float ss[NA];
#pragma unroll
  for (int i = 0; i < NA; ++i) ss[i] = 0.f;

  auto gload = [&](int k0) {
    const int k = k0 + q8;
    // the gain slice is the same for every row this thread stages
    floatx4 g0 = floatx4{1.f, 1.f, 1.f, 1.f}, g1 = g0;
    if constexpr (kNorm) {
      if (k < p.K) {
        g0 = *reinterpret_cast<const floatx4*>(p.gain + k);
        g1 = *reinterpret_cast<const floatx4*>(p.gain + k + 4);
      }
    }
#pragma unroll
    for (int i = 0; i < NA; ++i) {
      if constexpr (kF32A) {
        // two float4 per unit; K % 4 == 0 so each float4 is all in or all out
        floatx4 lo = floatx4{0.f, 0.f, 0.f, 0.f}, hi = lo;
        const float* src = reinterpret_cast<const float*>(aptr[i]) + k0;
        if (aval[i] && k < p.K) lo = *reinterpret_cast<const floatx4*>(src);
        if (aval[i] && k + 4 < p.K) hi = *reinterpret_cast<const floatx4*>(src + 4);
        if constexpr (kNorm) {
          ss[i] += lo.x * lo.x + lo.y * lo.y + lo.z * lo.z + lo.w * lo.w +
                   hi.x * hi.x + hi.y * hi.y + hi.z * hi.z + hi.w * hi.w;
          lo *= g0;
          hi *= g1;
        }
        ra[i] = u32x4{pack2(lo.x, lo.y), pack2(lo.z, lo.w), pack2(hi.x, hi.y), pack2(hi.z, hi.w)};
      } else {
        ra[i] = (aval[i] && k < p.K) ? *reinterpret_cast<const u32x4*>(aptr[i] + k0)
                                     : u32x4{0u, 0u, 0u, 0u};
      }
    }
#pragma unroll
    for (int i = 0; i < NB; ++i)
      rb[i] = (bval[i] && k < Kw) ? *reinterpret_cast<const u32x4*>(bptr[i] + k0) : u32x4{0u, 0u, 0u, 0u};
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
#pragma unroll
    for (int i = 0; i < NA; ++i) {
      const int r = (tid + i * NT) / Q;
      *reinterpret_cast<u32x4*>(&sA[r * PITCH + q8]) = ra[i];
    }
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      const int r = (tid + i * NT) / Q;
      *reinterpret_cast<u32x4*>(&sB[r * PITCH + q8]) = rb[i];
    }
    __syncthreads();
    if (k0 + BK < p.K) gload(k0 + BK);

    bf16x8 a8[TM][4], b8[TN][4];
#pragma unroll
    for (int a = 0; a < TM; ++a) {
      const uint16_t* src = &sA[(wm * TM * 32 + a * 32 + li) * PITCH + lg * 32];
#pragma unroll
      for (int c = 0; c < 4; ++c)
        a8[a][c] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(src + 8 * c));
    }
#pragma unroll
    for (int b = 0; b < TN; ++b) {
      const uint16_t* src = &sB[(wn * TN * 32 + b * 32 + li) * PITCH + lg * 32];
#pragma unroll
      for (int c = 0; c < 4; ++c)
        b8[b][c] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(src + 8 * c));
    }
#pragma unroll
    for (int c = 0; c < 4; ++c)
#pragma unroll
      for (int a = 0; a < TM; ++a)
#pragma unroll
        for (int b = 0; b < TN; ++b)
          acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a8[a][c], b8[b][c], acc[a][b], 0, 0, 0);
  }

  if constexpr (kNorm) {
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

  // 32x32 accumulator layout: lane l holds column l % 32 and rows
  // 8*(r/4) + 4*(l/32) + (r%4), r = 0..15.
#pragma unroll
  for (int a = 0; a < TM; ++a) {
#pragma unroll
    for (int b = 0; b < TN; ++b) {
      const int col = col0 + wn * TN * 32 + b * 32 + li;
      const bool cok = col < p.N;
      // a block's residual loads go before its stores (C may be read in place)
      float res[16];
      if constexpr ((FL & kResid) != 0 && sizeof(TC) == 4) {
        const float* R = p.R ? p.R : reinterpret_cast<const float*>(p.C);
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int row = row0 + wm * TM * 32 + a * 32 + 8 * (r >> 2) + 4 * lg + (r & 3);
          res[r] = (cok && row < M) ? R[(int64_t)row * p.ldc + col] : 0.f;
        }
      }
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
        TC* dst = reinterpret_cast<TC*>(p.C) + (int64_t)row * p.ldc + col;
        if constexpr (sizeof(TC) == 4) {
          if constexpr ((FL & kResid) != 0) v += res[r];
          *reinterpret_cast<float*>(dst) = v;
        } else {
          *reinterpret_cast<uint16_t*>(dst) = f32_to_bf16(v);
        }
      }
    }
  }
}

template <typename TA, typename TC, int WM, int WN, int TM, int TN, int FL>
hipError_t launch_t(const GemmArgsBF16& a, hipStream_t s) {
  constexpr int BM = WM * TM * 32, BN = WN * TN * 32;
  const int ntm = (a.Mmax + BM - 1) / BM;
  const int ntn = (a.N + BN - 1) / BN;
  const int grid = 8 * ntn * ((ntm + 7) / 8);
  if (grid <= 0) return hipSuccess;
  hipLaunchKernelGGL((gemm_bf16_kernel<TA, TC, WM, WN, TM, TN, FL>), dim3(grid), dim3(WM * WN * 64), 0,
                     s, a, ntm, ntn);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_gemm_bf16(const GemmArgsBF16& a, GemmBF16Kind kind, hipStream_t s) {
  switch (kind) {
    case kInputF32toF32:  // features (fp32, gathered) -> H fp32, + bias
      return launch_t<float, float, 2, 2, 2, 2, kBias | kGather>(a, s);
    case kNormF32toBF16:  // residual stream fp32 -> RMSNorm -> xz bf16
      return launch_t<float, uint16_t, 2, 2, 2, 2, kRowNorm>(a, s);
    case kBF16toF32Narrow:  // u bf16 -> xdbl fp32 (small N)
      return launch_t<uint16_t, float, 2, 2, 1, 1, 0>(a, s);
    case kBF16ResidF32:  // y bf16 -> H fp32 += result
      return launch_t<uint16_t, float, 2, 2, 2, 2, kResid>(a, s);
    case kBF16toF32:  // plain bf16 x bf16 -> fp32 (tests)
      return launch_t<uint16_t, float, 2, 2, 2, 2, 0>(a, s);
    case kBF16toF32Bias:
      return launch_t<uint16_t, float, 2, 2, 2, 2, kBias>(a, s);
    case kBF16toBF16:
      return launch_t<uint16_t, uint16_t, 2, 2, 2, 2, 0>(a, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace tcl
