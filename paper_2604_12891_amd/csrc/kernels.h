// Host-side launchers of the libtcl kernels (internal to the library).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace tcl {

// ---------------------------------------------------------------- GEMM
// C[M,N] (=|+=) rowscale[r] * (A[M,K] W[N,K]^T) + bias[N], fp32 in and out,
// on the fp32 MFMA units. Rows r >= M (M read from *Mdev when non-null)
// are skipped; A, W are read with bounds checks on K and N.
enum GemmFlags : int {
  kBias = 1,      // + bias[n]
  kResid = 2,     // C += result (residual add, C read before write)
  kRowNorm = 4,   // multiply row r by (mean_k A[r,k]^2 + eps)^-1/2 (RMSNorm)
  kGather = 8,    // A row of packed token r is row b*L + t of the padded input
};

struct GemmArgs {
  const float* A = nullptr;
  int64_t lda = 0;
  const int* offs = nullptr;  // gather: [B+1] token offsets
  int B = 0, L = 0;           // gather: batch and padded length
  const float* W = nullptr;
  int64_t ldw = 0;
  const float* bias = nullptr;
  float* C = nullptr;
  int64_t ldc = 0;
  const int* Mdev = nullptr;  // device row count (null: use Mmax)
  int Mmax = 0;               // upper bound on the row count (grid size)
  int N = 0, K = 0;
  float eps = 0.f;
};

// Tile shapes: kWide = 128x128 (2x2 waves of 64x64), kNarrow = 64x64 for
// small-N projections (x_proj).
enum GemmTile { kWide = 0, kNarrow = 1 };

hipError_t launch_gemm_f32(const GemmArgs& a, int flags, GemmTile tile, hipStream_t s);

// bf16 GEMM: C = A W^T with A fp32 (converted while staged) or bf16, W bf16
// ([N, ldw] row-major, zero-padded in K to a multiple of 8, ldw % 8 == 0),
// C fp32 or bf16, fp32 accumulation. kRowNorm also scales A by gain[k]
// before the conversion (the RMSNorm gain) and needs K % 8 == 0.
struct GemmArgsBF16 {
  const void* A = nullptr;
  int64_t lda = 0;
  const int* offs = nullptr;
  int B = 0, L = 0;
  const uint16_t* W = nullptr;
  int64_t ldw = 0;
  const float* bias = nullptr;
  const float* gain = nullptr;
  void* C = nullptr;
  int64_t ldc = 0;
  const int* Mdev = nullptr;
  int Mmax = 0;
  int N = 0, K = 0;
  float eps = 0.f;
};

enum GemmBF16Kind {
  kInputF32toF32,    // fp32 features (gathered) -> fp32, + bias
  kNormF32toBF16,    // fp32 residual -> RMSNorm (rstd, gain) -> bf16
  kBF16toF32Narrow,  // bf16 -> fp32, 64x64 tiles
  kBF16ResidF32,     // bf16 -> fp32 C += result
  kBF16toF32,        // bf16 -> fp32
  kBF16toF32Bias,    // bf16 -> fp32, + bias
};

hipError_t launch_gemm_bf16(const GemmArgsBF16& a, GemmBF16Kind kind, hipStream_t s);

// ---------------------------------------------------------------- per-program kernels
// offs[b] = sum of valid lengths before b; offs[B] = total packed rows.
// Lengths outside [1, L] count as 0 tokens.
hipError_t launch_offsets(const int* lengths, int B, int L, int* offs, hipStream_t s);

// Activations are stored as fp32 (T = float) or bf16 (T = uint16_t); the
// arithmetic is fp32 either way.

// u = SiLU(conv_b + sum_k w[e,k] x[t-(K-1)+k, e]) within each program.
// E and ldx are multiples of 4 (fp32) or 8 (bf16); pointers 16-byte aligned.
template <typename T>
hipError_t launch_conv_silu(int B, int E, int K, const int* offs, const T* x, int ldx,
                            const float* w, const float* b, T* u, hipStream_t s);

// Selective scan with dt_proj+softplus prologue, D skip and SiLU(z) gate.
// xdbl rows ([dt_r | B | C], R + 2N values) are fp32. out may alias u (each
// element is read then written by the same thread).
template <typename T>
hipError_t launch_scan(int B, int E, int N, int R, const int* offs, const T* u, const float* xdbl,
                       const T* z, int ldz, const float* W_dt, const float* b_dt, const float* A_log,
                       const float* D, T* out, hipStream_t s);

// Final RMSNorm (optional) + masked mean-pool + Linear-ReLU-Linear head.
// W1T is W1 transposed ([d, h]). Programs with invalid lengths get NaN.
hipError_t launch_tail_f32(int B, int L, int d, int h, const int* offs, const int* lengths,
                           const float* H, const float* g_f, int final_norm, float eps,
                           const float* W1T, const float* b1, const float* W2, const float* b2,
                           float* scores, hipStream_t s);

}  // namespace tcl
