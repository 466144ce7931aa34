// Weight-gradient GEMM: P[s] = sum over tokens m in split s of
// A[m, i] * B[m, j], i.e. dW = dY^T X restricted to one slice of the tokens,
// on the fp32 matrix cores (v_mfma_f32_32x32x2_f32).
//
// Both operands are token-major (row m = token), which is exactly what the
// fp32 MFMA wants here: lane l supplies A^T[i = l%32][k = l/32] =
// A[m0 + l/32][i0 + l%32], so 32 lanes read 32 consecutive features of one
// token -- a contiguous row segment -- and no transpose is needed. Inputs
// may be fp32 or bf16 (widened exactly); B may be gathered from the padded
// feature tensor. Each split writes its own fp32 partial tile; a separate
// reduction sums the splits in a fixed order, so the result is
// deterministic. Splits that start past the packed token count write zeros.
#include "common.h"
#include "kernels.h"

namespace tcl {
namespace {

constexpr int BK = 32;            // tokens per chunk
constexpr int TW = 64;            // tile width in i and in j
constexpr int PITCH = TW + 4;     // floats per LDS row

__device__ __forceinline__ void load8(const float* p, float* v) {
  const floatx4 a = *reinterpret_cast<const floatx4*>(p);
  const floatx4 b = *reinterpret_cast<const floatx4*>(p + 4);
  v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
  v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
}
__device__ __forceinline__ void load8(const uint16_t* p, float* v) {
  typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
  const u32x4 x = *reinterpret_cast<const u32x4*>(p);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    v[2 * i] = __uint_as_float(x[i] << 16);
    v[2 * i + 1] = __uint_as_float(x[i] & 0xFFFF0000u);
  }
}

// Stage rows [m0, m0 + BK) x columns [c0, c0 + TW) of X into LDS as fp32.
// Thread t loads 8 consecutive columns of one row; out-of-range rows or
// columns read as zero. A full group of 8 is read with 16-byte loads when
// the row pitch keeps them aligned, else element by element.
template <typename T, bool GATHER>
__device__ __forceinline__ void stage(float* s, const T* X, int64_t ldx, int ncols, int m0, int M,
                                      int c0, const int* offs, int B, int L) {
  const int tid = threadIdx.x;          // 256 threads: 32 rows x 8 column groups
  const int r = tid >> 3, cg = (tid & 7) * 8;
  const int m = m0 + r;
  float v[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) v[i] = 0.f;
  if (m < M) {
    int64_t src = m;
    if constexpr (GATHER) {
      int lo = 0, hi = B;
      while (hi - lo > 1) {
        const int mid = (lo + hi) >> 1;
        if (offs[mid] <= m) lo = mid; else hi = mid;
      }
      src = (int64_t)lo * L + (m - offs[lo]);
    }
    const T* row = X + src * ldx + c0 + cg;
    if (c0 + cg + 8 <= ncols && (ldx % (16 / sizeof(T))) == 0) {
      load8(row, v);
    } else {
#pragma unroll
      for (int i = 0; i < 8; ++i)
        if (c0 + cg + i < ncols) {
          if constexpr (sizeof(T) == 4) v[i] = row[i];
          else v[i] = bf16_to_f32(row[i]);
        }
    }
  }
#pragma unroll
  for (int i = 0; i < 8; ++i) s[r * PITCH + cg + i] = v[i];
}

template <typename TA, typename TB, bool GATHER_B>
__global__ __launch_bounds__(256) void gemm_tn_kernel(GemmTNArgs p, int nti, int ntj, int rows_per_split) {
  __shared__ __attribute__((aligned(16))) float sA[BK * PITCH];
  __shared__ __attribute__((aligned(16))) float sB[BK * PITCH];
  const int tile = blockIdx.x;
  const int split = blockIdx.y;
  const int ti = tile / ntj, tj = tile % ntj;
  const int i0 = ti * TW, j0 = tj * TW;
  const int M = p.Mdev ? *p.Mdev : p.Mmax;
  const int m_begin = split * rows_per_split;
  const int m_end = min(m_begin + rows_per_split, M);

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int wi = wave >> 1, wj = wave & 1;
  const int li = lane & 31, lg = lane >> 5;
  floatx16 acc;
#pragma unroll
  for (int r = 0; r < 16; ++r) acc[r] = 0.f;

  for (int m0 = m_begin; m0 < m_end; m0 += BK) {
    __syncthreads();
    stage<TA, false>(sA, reinterpret_cast<const TA*>(p.A), p.lda, p.NI, m0, m_end, i0, nullptr, 0, 0);
    stage<TB, GATHER_B>(sB, reinterpret_cast<const TB*>(p.Bm), p.ldb, p.NJ, m0, m_end, j0, p.offs, p.B,
                        p.L);
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < BK / 2; ++kk) {
      const float a = sA[(2 * kk + lg) * PITCH + wi * 32 + li];
      const float b = sB[(2 * kk + lg) * PITCH + wj * 32 + li];
      acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, acc, 0, 0, 0);
    }
  }

  // D[i][j]: lane holds j = li, i = 8*(r/4) + 4*lg + (r%4)
  float* out = p.P + (int64_t)split * p.NI * p.NJ;
  const int j = j0 + wj * 32 + li;
  if (j < p.NJ) {
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int i = i0 + wi * 32 + 8 * (r >> 2) + 4 * lg + (r & 3);
      if (i < p.NI) out[(int64_t)i * p.NJ + j] = acc[r];
    }
  }
}

}  // namespace

int gemm_tn_splits(int Mmax, int NI, int NJ) {
  const int tiles = ((NI + TW - 1) / TW) * ((NJ + TW - 1) / TW);
  int s = (512 + tiles - 1) / tiles;              // aim for >= 512 workgroups
  const int max_s = (Mmax + BK - 1) / BK;         // at least one chunk per split
  if (s > max_s) s = max_s;
  if (s < 1) s = 1;
  return s;
}

hipError_t launch_gemm_tn(const GemmTNArgs& a, TNKind kind, int splits, hipStream_t s) {
  const int nti = (a.NI + TW - 1) / TW, ntj = (a.NJ + TW - 1) / TW;
  int rps = (a.Mmax + splits - 1) / splits;
  rps = (rps + BK - 1) / BK * BK;
  dim3 grid(nti * ntj, splits);
  switch (kind) {
    case kTN_F32_F32:
      hipLaunchKernelGGL((gemm_tn_kernel<float, float, false>), grid, dim3(256), 0, s, a, nti, ntj, rps);
      break;
    case kTN_F32_BF16:
      hipLaunchKernelGGL((gemm_tn_kernel<float, uint16_t, false>), grid, dim3(256), 0, s, a, nti, ntj, rps);
      break;
    case kTN_F32_GatherF32:
      hipLaunchKernelGGL((gemm_tn_kernel<float, float, true>), grid, dim3(256), 0, s, a, nti, ntj, rps);
      break;
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace tcl
