// bf16 projections on the gfx950 matrix cores (v_mfma_f32_32x32x16_bf16),
// fp32 accumulation.
//
// Same structure as the fp32 GEMM: C = A W^T, K-contiguous operands, a
// workgroup tile of (WM*TM*32) x (WN*TN*32) built from 32x32 MFMA blocks
// held in accumulator registers, K staged through LDS in chunks of 64,
// XCD-aware tile order. The A operand may be fp32 (the residual stream or
// the input features) or bf16 (activations written by earlier kernels). W is
// bf16, zero-padded to a multiple of 8 in K. C is fp32 or bf16.
//
// Pipeline: the next chunk's global loads are issued right after the current
// chunk is in LDS and land in registers while the MFMAs run. An fp32 A chunk
// stays raw in those registers; it is converted to bf16 (round-to-nearest-
// even, after the RMSNorm gain when kRowNorm is set, whose sum of squares is
// accumulated from the same registers) only when it is written to LDS, so
// no load is waited on before the MFMAs that should hide it.
//
// Operand k-order: lane l of v_mfma_f32_32x32x16_bf16 supplies 8
// consecutive k of row (l % 32) in intrinsic positions 8*(l/32)..+7. Within
// a 64-wide chunk, lane half g takes k = 32g + 8j .. +7 in MFMA j (j=0..3),
// for A and W alike, so each lane reads its 32 contiguous bf16 with four
// 128-bit LDS loads.
//
// Epilogue: each wavefront writes one 32-row slice of its accumulators to
// LDS (the operand buffers are free by then), reads it back along rows and
// finishes four consecutive columns per lane: row scale, bias, residual
// (16-byte loads), conversion, and 16-byte (fp32) or 8-byte (bf16) stores
// that cover whole row segments. N and ldc are multiples of 4.
#include "common.h"
#include "kernels.h"

namespace tcl {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int BK = 64;          // k per chunk (bf16 elements)
constexpr int PITCH = BK + 8;   // bf16 per LDS row: 144 bytes, conflict-free 8-lane b128 reads
constexpr int Q = BK / 8;       // 16-byte units per row chunk

__device__ __forceinline__ uint32_t pack2(float a, float b) { return f32x2_to_bf16x2(a, b); }

constexpr int cmax(int a, int b) { return a > b ? a : b; }

// wavefronts per SIMD to aim for: fewer accumulators leave room for more;
// a raw fp32 A prefetch takes twice the registers of a bf16 one
constexpr int occupancy_for(int tm, int tn, bool f32a) {
  return tm * tn <= 1 ? 4 : tm * tn <= 2 ? (f32a ? 3 : 4) : tm * tn <= 4 ? (f32a ? 2 : 3) : 1;
}

template <typename TA, typename TC, int WM, int WN, int TM, int TN, int FL>
__global__ __launch_bounds__(WM* WN * 64, occupancy_for(TM, TN, sizeof(TA) == 4)) void gemm_bf16_kernel(
    GemmArgsBF16 p, int ntm, int ntn) {
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

  constexpr int SP = TN * 32 + 4;  // staging pitch (floats) of the epilogue
  constexpr int kOperandBytes = (BM + BN) * PITCH * 2;
  constexpr int kStageBytes = WM * WN * 32 * SP * 4;
  __shared__ __attribute__((aligned(16))) unsigned char lds[cmax(kOperandBytes, kStageBytes)];
  __shared__ float sR[kNorm ? BM : 1];
  uint16_t* sA = reinterpret_cast<uint16_t*>(lds);
  uint16_t* sB = sA + BM * PITCH;

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

  // prefetch registers: raw fp32 A (two float4 per unit) or bf16 A, bf16 W
  constexpr int NAF = kF32A ? NA : 1;
  constexpr int NAH = kF32A ? 1 : NA;
  floatx4 alo[NAF], ahi[NAF];
  u32x4 ra[NAH], rb[NB];
  floatx4 gl0 = floatx4{1.f, 1.f, 1.f, 1.f}, gl1 = gl0;
  float ss[NA];
#pragma unroll
  for (int i = 0; i < NA; ++i) ss[i] = 0.f;

  auto gload = [&](int k0) {
    const int k = k0 + q8;
    if constexpr (kNorm) {
      // the gain slice is the same for every row this thread stages
      gl0 = k < p.K ? *reinterpret_cast<const floatx4*>(p.gain + k) : floatx4{0.f, 0.f, 0.f, 0.f};
      gl1 = k + 4 < p.K ? *reinterpret_cast<const floatx4*>(p.gain + k + 4) : floatx4{0.f, 0.f, 0.f, 0.f};
    }
#pragma unroll
    for (int i = 0; i < NA; ++i) {
      if constexpr (kF32A) {
        // K % 4 == 0, so each float4 is all in or all out
        const float* src = reinterpret_cast<const float*>(aptr[i]) + k0;
        alo[i] = (aval[i] && k < p.K) ? *reinterpret_cast<const floatx4*>(src) : floatx4{0.f, 0.f, 0.f, 0.f};
        ahi[i] = (aval[i] && k + 4 < p.K) ? *reinterpret_cast<const floatx4*>(src + 4)
                                          : floatx4{0.f, 0.f, 0.f, 0.f};
      } else {
        ra[i] = (aval[i] && k < p.K) ? *reinterpret_cast<const u32x4*>(aptr[i] + k0)
                                     : u32x4{0u, 0u, 0u, 0u};
      }
    }
#pragma unroll
    for (int i = 0; i < NB; ++i)
      rb[i] = (bval[i] && k < Kw) ? *reinterpret_cast<const u32x4*>(bptr[i] + k0) : u32x4{0u, 0u, 0u, 0u};
  };

  auto stage = [&]() {
#pragma unroll
    for (int i = 0; i < NA; ++i) {
      const int r = (tid + i * NT) / Q;
      u32x4 v;
      if constexpr (kF32A) {
        floatx4 lo = alo[i], hi = ahi[i];
        if constexpr (kNorm) {
          ss[i] += lo.x * lo.x + lo.y * lo.y + lo.z * lo.z + lo.w * lo.w +
                   hi.x * hi.x + hi.y * hi.y + hi.z * hi.z + hi.w * hi.w;
          lo *= gl0;
          hi *= gl1;
        }
        v = u32x4{pack2(lo.x, lo.y), pack2(lo.z, lo.w), pack2(hi.x, hi.y), pack2(hi.z, hi.w)};
      } else {
        v = ra[i];
      }
      *reinterpret_cast<u32x4*>(&sA[r * PITCH + q8]) = v;
    }
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      const int r = (tid + i * NT) / Q;
      *reinterpret_cast<u32x4*>(&sB[r * PITCH + q8]) = rb[i];
    }
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
    if (k0 > 0) __syncthreads();  // every wavefront is done with the previous chunk
    stage();
    __syncthreads();
    if (k0 + BK < p.K) gload(k0 + BK);

#pragma unroll
    for (int c = 0; c < 4; ++c) {
      bf16x8 a8[TM], b8[TN];
#pragma unroll
      for (int a = 0; a < TM; ++a)
        a8[a] = __builtin_bit_cast(
            bf16x8, *reinterpret_cast<const u32x4*>(&sA[(wm * TM * 32 + a * 32 + li) * PITCH + lg * 32 + 8 * c]));
#pragma unroll
      for (int b = 0; b < TN; ++b)
        b8[b] = __builtin_bit_cast(
            bf16x8, *reinterpret_cast<const u32x4*>(&sB[(wn * TN * 32 + b * 32 + li) * PITCH + lg * 32 + 8 * c]));
#pragma unroll
      for (int a = 0; a < TM; ++a)
#pragma unroll
        for (int b = 0; b < TN; ++b)
          acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a8[a], b8[b], acc[a][b], 0, 0, 0);
    }
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
  }
  __syncthreads();  // operand buffers free for staging; row scales visible

  float* stg = reinterpret_cast<float*>(lds) + wave * 32 * SP;
  constexpr int C4 = TN * 8;  // float4 groups per staged row
  const float* R = p.R ? p.R : reinterpret_cast<const float*>(p.C);
#pragma unroll
  for (int a = 0; a < TM; ++a) {
    if (a > 0) __syncthreads();  // the previous slice has been read back
    // 32x32 accumulator layout: lane l holds column l % 32 and rows
    // 8*(r/4) + 4*(l/32) + (r%4), r = 0..15.
#pragma unroll
    for (int b = 0; b < TN; ++b)
#pragma unroll
      for (int r = 0; r < 16; ++r)
        stg[(8 * (r >> 2) + 4 * lg + (r & 3)) * SP + b * 32 + li] = acc[a][b][r];
    __syncthreads();
    constexpr int NI = 32 * C4 / 64;
    // the slice's residuals are loaded before its first store: read in
    // place (R = C), they would otherwise each wait for the stores before
    floatx4 rv[(FL & kResid) != 0 ? NI : 1];
    if constexpr ((FL & kResid) != 0) {
#pragma unroll
      for (int i = 0; i < NI; ++i) {
        const int idx = lane + 64 * i;
        const int rr = idx / C4, c4 = idx % C4;
        const int row = row0 + wm * TM * 32 + a * 32 + rr;
        const int col = col0 + wn * TN * 32 + c4 * 4;
        rv[i] = (row < M && col < p.N) ? *reinterpret_cast<const floatx4*>(R + (int64_t)row * p.ldc + col)
                                       : floatx4{0.f, 0.f, 0.f, 0.f};
      }
    }
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int idx = lane + 64 * i;
      const int rr = idx / C4, c4 = idx % C4;
      const int rl = wm * TM * 32 + a * 32 + rr;
      const int row = row0 + rl;
      const int col = col0 + wn * TN * 32 + c4 * 4;
      if (row >= M || col >= p.N) continue;
      floatx4 v = *reinterpret_cast<const floatx4*>(&stg[rr * SP + c4 * 4]);
      if constexpr (kNorm) v *= sR[rl];
      if constexpr ((FL & kBias) != 0)
        v += floatx4{p.bias[col], p.bias[col + 1], p.bias[col + 2], p.bias[col + 3]};
      const int64_t off = (int64_t)row * p.ldc + col;
      if constexpr (sizeof(TC) == 4) {
        if constexpr ((FL & kResid) != 0) v += rv[i];
        *reinterpret_cast<floatx4*>(reinterpret_cast<float*>(p.C) + off) = v;
      } else {
        *reinterpret_cast<u32x2*>(reinterpret_cast<uint16_t*>(p.C) + off) =
            u32x2{pack2(v.x, v.y), pack2(v.z, v.w)};
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

template <typename TA, typename TC, int FL>
hipError_t dispatch_tile(const GemmArgsBF16& a, GemmBF16Tile tile, hipStream_t s) {
  switch (tile) {
    case kB128x128: return launch_t<TA, TC, 2, 2, 2, 2, FL>(a, s);
    case kB64x64: return launch_t<TA, TC, 2, 2, 1, 1, FL>(a, s);
    case kB64x128: return launch_t<TA, TC, 2, 2, 1, 2, FL>(a, s);
    case kB128x64: return launch_t<TA, TC, 2, 2, 2, 1, FL>(a, s);
    case kB128x256: return launch_t<TA, TC, 2, 4, 2, 2, FL>(a, s);
    case kB256x128: return launch_t<TA, TC, 4, 2, 2, 2, FL>(a, s);
    case kB256x128W4: return launch_t<TA, TC, 2, 2, 4, 2, FL>(a, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

GemmBF16Tile pick_gemm_bf16_tile(GemmBF16Kind kind, int Mmax, int N, int K) {
  // Measured on MI355X (microseconds per call, ~983K rows unless noted):
  // in_proj (RMSNorm, N = 1024, K = 256) row panels 923 vs 1489 for the best
  // tile, and at 492K rows 128-row panels (whole-line bf16 stores) 448 vs
  // 496 for 256-row ones; gathered input Linear (N = 256, K = 164) 128-row
  // panels 376 vs 391 for 256-row ones and 591 for the best tile; out_proj
  // (K = 512, no panel) 128x128 629; x_proj (N = 48) 64x64 227. At ~15K rows
  // (distillation) 128x64 wins for N <= 256 (7.2 vs 9.4 at N = 128, 11.9 vs
  // 13.5 at 256).
  if (N <= 64) return kB64x64;
  if (K <= 256 && Mmax >= 131072 && kind != kF32toF32 && kind != kF32ResidF32)
    return kind == kInputF32toF32 || kind == kNormF32toBF16 || kind == kBF16toBF16 ? kBPanel128 : kBPanel;
  if (Mmax < 131072 && N <= 256) return kB128x64;
  return kB128x128;
}

hipError_t launch_gemm_bf16(const GemmArgsBF16& a, GemmBF16Kind kind, int tile, hipStream_t s) {
  // the vectorised epilogue finishes four columns at a time
  if (a.N % 4 || a.ldc % 4) return hipErrorInvalidValue;
  GemmBF16Tile t = tile < 0 ? pick_gemm_bf16_tile(kind, a.Mmax, a.N, a.K) : static_cast<GemmBF16Tile>(tile);
  if (t == kBPanel || t == kBPanel128) {
    const bool bf16_out = kind == kNormF32toBF16 || kind == kBF16toBF16;
    if (gemm_bf16_panel_fits(a, bf16_out)) return launch_gemm_bf16_panel(a, kind, t == kBPanel ? 64 : 32, s);
    if (tile >= 0) return hipErrorInvalidValue;
    t = kB128x128;
  }
  switch (kind) {
    case kInputF32toF32:  // features (fp32, gathered) -> H fp32, + bias
      return dispatch_tile<float, float, kBias | kGather>(a, t, s);
    case kNormF32toBF16:  // residual stream fp32 -> RMSNorm -> xz bf16
      return dispatch_tile<float, uint16_t, kRowNorm>(a, t, s);
    case kBF16ResidF32:  // y bf16 -> H fp32 += result
      return dispatch_tile<uint16_t, float, kResid>(a, t, s);
    case kBF16toF32:
      return dispatch_tile<uint16_t, float, 0>(a, t, s);
    case kBF16toF32Bias:
      return dispatch_tile<uint16_t, float, kBias>(a, t, s);
    case kBF16toBF16:
      return dispatch_tile<uint16_t, uint16_t, 0>(a, t, s);
    case kF32toF32:  // fp32 gradients -> fp32 (the backward's data gradients)
      return dispatch_tile<float, float, 0>(a, t, s);
    case kF32ResidF32:
      return dispatch_tile<float, float, kResid>(a, t, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace tcl
