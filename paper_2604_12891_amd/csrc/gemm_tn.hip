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
// the device-side token count), and the next three 32-token chunks are in
// flight while the current one's MFMAs run (a split walks its chunks one
// after another, so memory latency, not the MFMAs, sets its pace). Each split writes its own fp32 partial tile;
// a separate reduction sums the splits in a fixed order, so the result is
// deterministic. Splits that start past the packed token count write zeros.
#include "common.h"
#include "kernels.h"

namespace tcl {
namespace {

constexpr int BK = 32;            // tokens per chunk
constexpr int TW = 64;            // tile width in i and in j
constexpr int PITCH = TW + 4;     // floats per LDS row
constexpr int NPF = 3;            // chunks in flight per workgroup

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Eight consecutive values of one row as loaded, before conversion (the
// conversion is done when the chunk is parked in LDS, so that it does not
// make the compiler wait for the load right after issuing it).
template <typename T> struct Raw;
template <> struct Raw<float> {
  floatx4 a, b;
  __device__ __forceinline__ void load(__amdgpu_buffer_rsrc_t rs, uint32_t off) {
    a = __builtin_bit_cast(floatx4, __builtin_amdgcn_raw_buffer_load_b128(rs, off, 0, 0));
    b = __builtin_bit_cast(floatx4, __builtin_amdgcn_raw_buffer_load_b128(rs, off + 16, 0, 0));
  }
  __device__ __forceinline__ void zero() { a = b = floatx4{0.f, 0.f, 0.f, 0.f}; }
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
  __device__ __forceinline__ void load(__amdgpu_buffer_rsrc_t rs, uint32_t off) {
    a = __builtin_amdgcn_raw_buffer_load_b128(rs, off, 0, 0);
  }
  __device__ __forceinline__ void zero() { a = u32x4{0u, 0u, 0u, 0u}; }
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
// consecutive columns of one row with 16-byte buffer loads (rows are 16-byte
// aligned: the launcher checks). A row past M reads zero (an out-of-range
// offset). Columns past the operand's width read whatever follows in memory
// (the next row, or zero past the tensor's end): they only feed rows or
// columns of the tile that are never stored. No branch separates the loads.
constexpr uint32_t kOutOfRange = 0x80000000u;  // beyond every resource (sizes < 2^31 bytes)
template <typename T, bool GATHER>
__device__ __forceinline__ void fetch(Raw<T>& raw, __amdgpu_buffer_rsrc_t rs, int64_t ldx, int m0, int M, int c0,
                                      const int* offs, int B, int L, const int* rows) {
  const int tid = threadIdx.x;          // 256 threads: 32 rows x 8 column groups
  const int r = tid >> 3, cg = (tid & 7) * 8;
  const int m = m0 + r;
  int64_t src = m;
  if constexpr (GATHER) {
    if (rows) {
      src = rows[m < M ? m : 0];
    } else if (m < M) {
      int lo = 0, hi = B;
      while (hi - lo > 1) {
        const int mid = (lo + hi) >> 1;
        if (offs[mid] <= m) lo = mid; else hi = mid;
      }
      src = (int64_t)lo * L + (m - offs[lo]);
    }
  }
  const uint32_t off = m < M ? (uint32_t)((src * ldx + c0 + cg) * (int64_t)sizeof(T)) : kOutOfRange;
  raw.load(rs, off);
}

// The same rows and columns element by element, for operands whose rows are
// not 16-byte aligned; columns past ncols read as zero here.
template <typename T, bool GATHER>
__device__ __forceinline__ void fetch_any(Raw<T>& raw, const T* X, int64_t ldx, int ncols, int m0, int M, int c0,
                                          const int* offs, int B, int L) {
  const int tid = threadIdx.x;
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
#pragma unroll
    for (int i = 0; i < 8; ++i)
      if (c0 + cg + i < ncols) raw.one(i, row + i);
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

template <typename TA, typename TB, bool GATHER_B, bool VEC>
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

  // NPF chunks are in flight: when chunk c is parked, chunk c + NPF is
  // fetched into its registers (a fetch past the split's end reads nothing)
  Raw<TA> ra[NPF];
  Raw<TB> rb[NPF];
  const __amdgpu_buffer_rsrc_t Ar =
      raw_rsrc(p.A, VEC ? (uint32_t)((int64_t)p.Mmax * p.lda * (int64_t)sizeof(TA)) : 0u);
  const __amdgpu_buffer_rsrc_t Br = raw_rsrc(
      p.Bm, VEC ? (uint32_t)((GATHER_B ? (int64_t)p.B * p.L : (int64_t)p.Mmax) * p.ldb * (int64_t)sizeof(TB)) : 0u);
  auto fetch_a = [&](Raw<TA>& r, int m0) {
    if constexpr (VEC) fetch<TA, false>(r, Ar, p.lda, m0, m_end, i0, nullptr, 0, 0, nullptr);
    else fetch_any<TA, false>(r, reinterpret_cast<const TA*>(p.A), p.lda, p.NI, m0, m_end, i0, nullptr, 0, 0);
  };
  auto fetch_b = [&](Raw<TB>& r, int m0) {
    if constexpr (VEC) fetch<TB, GATHER_B>(r, Br, p.ldb, m0, m_end, j0, p.offs, p.B, p.L, p.rows);
    else fetch_any<TB, GATHER_B>(r, reinterpret_cast<const TB*>(p.Bm), p.ldb, p.NJ, m0, m_end, j0, p.offs, p.B, p.L);
  };
#pragma unroll
  for (int q = 0; q < NPF; ++q) {
    fetch_a(ra[q], m_begin + q * BK);
    fetch_b(rb[q], m_begin + q * BK);
  }
  for (int m0 = m_begin; m0 < m_end; m0 += NPF * BK) {
#pragma unroll
    for (int q = 0; q < NPF; ++q) {
      // every trip runs all NPF chunks: one past the split's end holds zeros
      // (its fetch read nothing) and adds nothing, and the loop body stays
      // straight-line, so the compiler's waits for the fetches stay exact
      const int mc = m0 + q * BK;
      __syncthreads();
      park(sA, ra[q]);
      park(sB, rb[q]);
      __syncthreads();
      fetch_a(ra[q], mc + NPF * BK);
      fetch_b(rb[q], mc + NPF * BK);
#pragma unroll
      for (int kk = 0; kk < BK / 2; ++kk) {
        const float a = sA[(2 * kk + lg) * PITCH + wi * 32 + li];
        const float b = sB[(2 * kk + lg) * PITCH + wj * 32 + li];
        acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, acc, 0, 0, 0);
      }
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

// The same product on the bf16 matrix cores (v_mfma_f32_32x32x16_bf16), for
// models that compute in bf16: both operands are rounded to bf16 (nearest
// even) as a chunk is parked, and parked transposed, [feature][token], so
// that a lane's eight consecutive tokens of one feature (its MFMA operand
// fragment) are one 16-byte LDS read. A 32-token chunk is two MFMAs per
// wavefront instead of sixteen; fp32 accumulation as above.
constexpr int PT = BK + 8;  // bf16 per transposed LDS row (80 bytes: conflict-free 16-byte reads)

template <typename T>
__device__ __forceinline__ void park_t(uint16_t* s, const Raw<T>& raw) {
  const int tid = threadIdx.x;
  const int r = tid >> 3, cg = (tid & 7) * 8;
  float v[8];
  raw.to_f32(v);
#pragma unroll
  for (int i = 0; i < 8; i += 2) {
    const uint32_t w = f32x2_to_bf16x2(v[i], v[i + 1]);
    s[(cg + i) * PT + r] = (uint16_t)(w & 0xFFFFu);
    s[(cg + i + 1) * PT + r] = (uint16_t)(w >> 16);
  }
}

template <typename TA, typename TB, bool GATHER_B, bool VEC>
__global__ __launch_bounds__(256) void gemm_tn_bf16_kernel(GemmTNArgs p, int nti, int ntj) {
  typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
  __shared__ __attribute__((aligned(16))) uint16_t sA[TW * PT];
  __shared__ __attribute__((aligned(16))) uint16_t sB[TW * PT];
  const int tile = blockIdx.x;
  const int split = blockIdx.y;
  const int ti = tile / ntj, tj = tile % ntj;
  const int i0 = ti * TW, j0 = tj * TW;
  const int M = p.Mdev ? *p.Mdev : p.Mmax;
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

  Raw<TA> ra[NPF];
  Raw<TB> rb[NPF];
  const __amdgpu_buffer_rsrc_t Ar =
      raw_rsrc(p.A, VEC ? (uint32_t)((int64_t)p.Mmax * p.lda * (int64_t)sizeof(TA)) : 0u);
  const __amdgpu_buffer_rsrc_t Br = raw_rsrc(
      p.Bm, VEC ? (uint32_t)((GATHER_B ? (int64_t)p.B * p.L : (int64_t)p.Mmax) * p.ldb * (int64_t)sizeof(TB)) : 0u);
  auto fetch_a = [&](Raw<TA>& r, int m0) {
    if constexpr (VEC) fetch<TA, false>(r, Ar, p.lda, m0, m_end, i0, nullptr, 0, 0, nullptr);
    else fetch_any<TA, false>(r, reinterpret_cast<const TA*>(p.A), p.lda, p.NI, m0, m_end, i0, nullptr, 0, 0);
  };
  auto fetch_b = [&](Raw<TB>& r, int m0) {
    if constexpr (VEC) fetch<TB, GATHER_B>(r, Br, p.ldb, m0, m_end, j0, p.offs, p.B, p.L, p.rows);
    else fetch_any<TB, GATHER_B>(r, reinterpret_cast<const TB*>(p.Bm), p.ldb, p.NJ, m0, m_end, j0, p.offs, p.B, p.L);
  };
#pragma unroll
  for (int q = 0; q < NPF; ++q) {
    fetch_a(ra[q], m_begin + q * BK);
    fetch_b(rb[q], m_begin + q * BK);
  }
  for (int m0 = m_begin; m0 < m_end; m0 += NPF * BK) {
#pragma unroll
    for (int q = 0; q < NPF; ++q) {
      // every trip runs all NPF chunks: one past the split's end holds zeros
      // (its fetch read nothing) and adds nothing, and the loop body stays
      // straight-line, so the compiler's waits for the fetches stay exact
      const int mc = m0 + q * BK;
      __syncthreads();
      park_t(sA, ra[q]);
      park_t(sB, rb[q]);
      __syncthreads();
      fetch_a(ra[q], mc + NPF * BK);
      fetch_b(rb[q], mc + NPF * BK);
      // lane: feature li of its 32-feature block, tokens 16 ks + 8 lg .. +7
#pragma unroll
      for (int ks = 0; ks < BK / 16; ++ks) {
        const bf16x8 a = *reinterpret_cast<const bf16x8*>(&sA[(wi * 32 + li) * PT + 16 * ks + 8 * lg]);
        const bf16x8 b = *reinterpret_cast<const bf16x8*>(&sB[(wj * 32 + li) * PT + 16 * ks + 8 * lg]);
        acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc, 0, 0, 0);
      }
    }
  }

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

namespace {
// the operands' rows can be read as 16-byte units through buffer resources
// of fewer than 2^31 bytes
bool tn_vec(const GemmTNArgs& a, TNKind kind) {
  const int eb = kind == kTN_F32_BF16 ? 2 : 4;
  const int64_t brows = kind == kTN_F32_GatherF32 ? (int64_t)a.B * a.L : (int64_t)a.Mmax;
  auto al16 = [](const void* q) { return reinterpret_cast<uintptr_t>(q) % 16 == 0; };
  return al16(a.A) && al16(a.Bm) && (a.lda * 4) % 16 == 0 && (a.ldb * eb) % 16 == 0 &&
         (int64_t)a.Mmax * a.lda * 4 < (1ll << 31) && brows * a.ldb * eb < (1ll << 31);
}

template <bool BF16, bool VEC>
hipError_t launch_tn(const GemmTNArgs& a, TNKind kind, int splits, hipStream_t s) {
  const int nti = (a.NI + TW - 1) / TW, ntj = (a.NJ + TW - 1) / TW;
  dim3 grid(nti * ntj, splits);
#define TCL_TN(TA, TB, G)                                                                              \
  do {                                                                                                 \
    if constexpr (BF16)                                                                                \
      hipLaunchKernelGGL((gemm_tn_bf16_kernel<TA, TB, G, VEC>), grid, dim3(256), 0, s, a, nti, ntj);     \
    else                                                                                               \
      hipLaunchKernelGGL((gemm_tn_kernel<TA, TB, G, VEC>), grid, dim3(256), 0, s, a, nti, ntj);          \
  } while (0)
  switch (kind) {
    case kTN_F32_F32: TCL_TN(float, float, false); break;
    case kTN_F32_BF16: TCL_TN(float, uint16_t, false); break;
    case kTN_F32_GatherF32: TCL_TN(float, float, true); break;
    default: return hipErrorInvalidValue;
  }
#undef TCL_TN
  return hipGetLastError();
}
}  // namespace

namespace {
__global__ __launch_bounds__(256) void packed_rows_kernel(const int* __restrict__ offs, int B, int L,
                                                          int* __restrict__ rows) {
  const int b = blockIdx.x * 256 + threadIdx.x;
  if (b >= B) return;
  const int base = offs[b], len = offs[b + 1] - base;
  for (int t = 0; t < len; ++t) rows[base + t] = b * L + t;
}
}  // namespace

hipError_t launch_packed_rows(const int* offs, int B, int L, int* rows, hipStream_t s) {
  if (B <= 0) return hipSuccess;
  hipLaunchKernelGGL(packed_rows_kernel, dim3((B + 255) / 256), dim3(256), 0, s, offs, B, L, rows);
  return hipGetLastError();
}

hipError_t launch_gemm_tn(const GemmTNArgs& a, TNKind kind, int splits, hipStream_t s) {
  return tn_vec(a, kind) ? launch_tn<false, true>(a, kind, splits, s) : launch_tn<false, false>(a, kind, splits, s);
}

hipError_t launch_gemm_tn_bf16(const GemmTNArgs& a, TNKind kind, int splits, hipStream_t s) {
  return tn_vec(a, kind) ? launch_tn<true, true>(a, kind, splits, s) : launch_tn<true, false>(a, kind, splits, s);
}

}  // namespace tcl
