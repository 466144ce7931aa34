// Weight-gradient GEMM: P[s] = sum over tokens m in split s of
// A[m, i] * B[m, j], i.e. dW = dY^T X restricted to one slice of the tokens,
// on the fp32 matrix cores (v_mfma_f32_32x32x2_f32).
//
// Both operands are token-major (row m = token), which is exactly what the
// fp32 MFMA wants here: lane l supplies A^T[i = l%32][k = l/32] =
// A[m0 + l/32][i0 + l%32], so 32 lanes read 32 consecutive features of one
// token -- a contiguous row segment -- and no transpose is needed. Inputs
// may be fp32 or bf16 (widened exactly); B may be gathered from the padded
// feature tensor. The packed tokens are divided evenly over the splits (from
// the device-side token count), and the next 32-token chunk is loaded while
// the current one's MFMAs run. Each split writes its own fp32 partial tile;
// a separate reduction sums the splits in a fixed order, so the result is
// deterministic. Splits that start past the packed token count write zeros.
#include "common.h"
#include "kernels.h"

namespace tcl {
namespace {

constexpr int BK = 32;            // tokens per chunk
constexpr int TW = 64;            // tile width in i and in j
constexpr int PITCH = TW + 4;     // floats per LDS row

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Eight consecutive values of one row as loaded, before conversion (the
// conversion is done when the chunk is parked in LDS, so that it does not
// make the compiler wait for the load right after issuing it).
template <typename T> struct Raw;
template <> struct Raw<float> {
  floatx4 a, b;
  __device__ __forceinline__ void zero() { a = b = floatx4{0.f, 0.f, 0.f, 0.f}; }
  __device__ __forceinline__ void vec(const float* p) {
    a = *reinterpret_cast<const floatx4*>(p);
    b = *reinterpret_cast<const floatx4*>(p + 4);
  }
  __device__ __forceinline__ void one(int i, const float* p) {
    if (i < 4) a[i] = *p; else b[i - 4] = *p;
  }
  __device__ __forceinline__ void to_f32(float* v) const {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      v[i] = a[i];
      v[4 + i] = b[i];
    }
  }
};
template <> struct Raw<uint16_t> {
  u32x4 a;
  __device__ __forceinline__ void zero() { a = u32x4{0u, 0u, 0u, 0u}; }
  __device__ __forceinline__ void vec(const uint16_t* p) { a = *reinterpret_cast<const u32x4*>(p); }
  __device__ __forceinline__ void one(int i, const uint16_t* p) { a[i >> 1] |= (uint32_t)*p << (16 * (i & 1)); }
  __device__ __forceinline__ void to_f32(float* v) const {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      v[2 * i] = __uint_as_float(a[i] << 16);
      v[2 * i + 1] = __uint_as_float(a[i] & 0xFFFF0000u);
    }
  }
};

// Rows [m0, m0 + BK) x columns [c0, c0 + TW) of X: thread t fetches 8
// consecutive columns of one row; out-of-range rows or columns read as
// zero. A full group of 8 is read with 16-byte loads when the row pitch
// keeps them aligned, else element by element.
template <typename T, bool GATHER>
__device__ __forceinline__ void fetch(Raw<T>& raw, const T* X, int64_t ldx, int ncols, int m0, int M, int c0,
                                      const int* offs, int B, int L) {
  const int tid = threadIdx.x;          // 256 threads: 32 rows x 8 column groups
  const int r = tid >> 3, cg = (tid & 7) * 8;
  const int m = m0 + r;
  raw.zero();
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
      raw.vec(row);
    } else {
#pragma unroll
      for (int i = 0; i < 8; ++i)
        if (c0 + cg + i < ncols) raw.one(i, row + i);
    }
  }
}

template <typename T>
__device__ __forceinline__ void park(float* s, const Raw<T>& raw) {
  const int tid = threadIdx.x;
  const int r = tid >> 3, cg = (tid & 7) * 8;
  float v[8];
  raw.to_f32(v);
  *reinterpret_cast<floatx4*>(&s[r * PITCH + cg]) = floatx4{v[0], v[1], v[2], v[3]};
  *reinterpret_cast<floatx4*>(&s[r * PITCH + cg + 4]) = floatx4{v[4], v[5], v[6], v[7]};
}

template <typename TA, typename TB, bool GATHER_B>
__global__ __launch_bounds__(256) void gemm_tn_kernel(GemmTNArgs p, int nti, int ntj) {
  __shared__ __attribute__((aligned(16))) float sA[BK * PITCH];
  __shared__ __attribute__((aligned(16))) float sB[BK * PITCH];
  const int tile = blockIdx.x;
  const int split = blockIdx.y;
  const int ti = tile / ntj, tj = tile % ntj;
  const int i0 = ti * TW, j0 = tj * TW;
  const int M = p.Mdev ? *p.Mdev : p.Mmax;
  // the packed rows are divided evenly over the splits from the device row
  // count (the grid is sized for the row bound)
  int rps = (M + (int)gridDim.y - 1) / (int)gridDim.y;
  rps = (rps + BK - 1) / BK * BK;
  const int m_begin = split * rps;
  const int m_end = min(m_begin + rps, M);

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int wi = wave >> 1, wj = wave & 1;
  const int li = lane & 31, lg = lane >> 5;
  floatx16 acc;
#pragma unroll
  for (int r = 0; r < 16; ++r) acc[r] = 0.f;

  // chunk m0 + BK is fetched while chunk m0's MFMAs run
  Raw<TA> ra;
  Raw<TB> rb;
  const TA* Ap = reinterpret_cast<const TA*>(p.A);
  const TB* Bp = reinterpret_cast<const TB*>(p.Bm);
  if (m_begin < m_end) {
    fetch<TA, false>(ra, Ap, p.lda, p.NI, m_begin, m_end, i0, nullptr, 0, 0);
    fetch<TB, GATHER_B>(rb, Bp, p.ldb, p.NJ, m_begin, m_end, j0, p.offs, p.B, p.L);
  }
  for (int m0 = m_begin; m0 < m_end; m0 += BK) {
    __syncthreads();
    park(sA, ra);
    park(sB, rb);
    __syncthreads();
    if (m0 + BK < m_end) {
      fetch<TA, false>(ra, Ap, p.lda, p.NI, m0 + BK, m_end, i0, nullptr, 0, 0);
      fetch<TB, GATHER_B>(rb, Bp, p.ldb, p.NJ, m0 + BK, m_end, j0, p.offs, p.B, p.L);
    }
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
  dim3 grid(nti * ntj, splits);
  switch (kind) {
    case kTN_F32_F32:
      hipLaunchKernelGGL((gemm_tn_kernel<float, float, false>), grid, dim3(256), 0, s, a, nti, ntj);
      break;
    case kTN_F32_BF16:
      hipLaunchKernelGGL((gemm_tn_kernel<float, uint16_t, false>), grid, dim3(256), 0, s, a, nti, ntj);
      break;
    case kTN_F32_GatherF32:
      hipLaunchKernelGGL((gemm_tn_kernel<float, float, true>), grid, dim3(256), 0, s, a, nti, ntj);
      break;
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace tcl
