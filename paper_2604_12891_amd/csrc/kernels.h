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

// ---------------------------------------------------------------- per-program kernels
// offs[b] = sum of valid lengths before b; offs[B] = total packed rows.
// Lengths outside [1, L] count as 0 tokens.
hipError_t launch_offsets(const int* lengths, int B, int L, int* offs, hipStream_t s);

// u = SiLU(conv_b + sum_k w[e,k] x[t-(K-1)+k, e]) within each program.
hipError_t launch_conv_silu_f32(int B, int E, int K, const int* offs, const float* x, int ldx,
                                const float* w, const float* b, float* u, hipStream_t s);

// Selective scan with dt_proj+softplus prologue, D skip and SiLU(z) gate.
// out may alias u (each element is read then written by the same thread).
hipError_t launch_scan_f32(int B, int E, int N, int R, const int* offs, const float* u,
                           const float* xdbl, const float* z, int ldz, const float* W_dt,
                           const float* b_dt, const float* A_log, const float* D, float* out,
                           hipStream_t s);

// Final RMSNorm (optional) + masked mean-pool + Linear-ReLU-Linear head.
// W1T is W1 transposed ([d, h]). Programs with invalid lengths get NaN.
hipError_t launch_tail_f32(int B, int L, int d, int h, const int* offs, const int* lengths,
                           const float* H, const float* g_f, int final_norm, float eps,
                           const float* W1T, const float* b1, const float* W2, const float* b2,
                           float* scores, hipStream_t s);

}  // namespace tcl
