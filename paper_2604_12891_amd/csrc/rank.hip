// The ranking objectives: LambdaRank (section 5.3, Eq. (6)) on a batch of
// scores against one or two label sets, the teacher-loss gate (Eq. (10)-
// (11)) and the EWC penalty of the distillation objective (section 6,
// Eq. (9)).
//
// LambdaRank, per label set:
//   L = sum over pairs with rel_i > rel_j of
//       |G_i - G_j| |1/D_i - 1/D_j| log2(1 + exp(-sigma (s_i - s_j)))
//   rel = labels min-max normalised over the batch, G = (2^rel - 1) / maxDCG,
//   D_i = log2(1 + r_i) with r_i the 1-based rank of s_i (descending, equal
//   scores in index order), maxDCG = the DCG of the ordering by rel.
// The ranks are counted, not sorted: item i's rank is one plus the number of
// items ahead of it, an O(B^2) pass that is cheap at tuning-round sizes and
// needs no sort. Four launches:
//   count:  a grid of (256 items i) x (j chunks); per item the chunk's
//           items ahead of it by score and, per set, by relevance;
//   prep:   per item its score rank (the chunks' counts summed), and per
//           set its gain 2^rel - 1 and ideal-DCG term (gain over
//           log2(1 + ideal rank));
//   pairs:  a grid of (256 items i) x (j tiles); each thread accumulates
//           its item's loss and gradient over one j tile;
//   finish: sums the j-tile partials in a fixed order (deterministic).
// The chunks and tiles are sized so that a few dozen cover the batch.
// All fp32; maxDCG is summed identically by every block.
#include "common.h"
#include "kernels.h"

namespace tcl {
namespace {

constexpr int kRT = 256;    // threads per block = items per i block = items per j tile
constexpr float kInvLn2 = 1.4426950408889634f;

// Sum over the block; every thread receives the total. The order of the
// additions depends only on the block size, so every block agrees.
__device__ __forceinline__ float block_sum(float v, float* red) {
  v = wave_sum(v);
  const int w = threadIdx.x >> 6;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[w] = v;
  __syncthreads();
  float t = 0.f;
#pragma unroll
  for (int i = 0; i < kRT / 64; ++i) t += red[i];
  return t;
}

__device__ __forceinline__ float block_min(float v, float* red) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fminf(v, __shfl_xor(v, o, 64));
  const int w = threadIdx.x >> 6;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[w] = v;
  __syncthreads();
  float t = red[0];
#pragma unroll
  for (int i = 1; i < kRT / 64; ++i) t = fminf(t, red[i]);
  return t;
}

__device__ __forceinline__ float block_max(float v, float* red) { return -block_min(-v, red); }

// relevance of a label given the set's min and max (all zero when equal)
__device__ __forceinline__ float rel_of(float y, float lo, float inv_range) { return (y - lo) * inv_range; }

// The j range is cut into chunks (counting) and tiles (pairs) sized so that
// a few dozen of them cover the batch: at tuning-round sizes the O(B^2)
// passes then spread over hundreds of workgroups instead of a handful.
__host__ __device__ constexpr int rank_count_chunk(int B) {
  const int c = ((B + 15) / 16 + 63) / 64 * 64;  // <= 16 chunks
  return c < 64 ? 64 : (c > 4096 ? 4096 : c);
}
__host__ __device__ constexpr int rank_pair_tile(int B) {
  const int t = ((B + 63) / 64 + 31) / 32 * 32;  // <= 64 tiles
  return t < 32 ? 32 : (t > 2048 ? 2048 : t);
}

// every block: each set's min and max over the batch
template <int NS>
__device__ __forceinline__ void label_range(int B, const float* const* lab, float* lo, float* ir, float* red) {
#pragma unroll
  for (int k = 0; k < NS; ++k) {
    float mn = INFINITY, mx = -INFINITY;
    for (int j = threadIdx.x; j < B; j += kRT) {
      mn = fminf(mn, lab[k][j]);
      mx = fmaxf(mx, lab[k][j]);
    }
    lo[k] = block_min(mn, red);
    const float hi = block_max(mx, red);
    ir[k] = hi > lo[k] ? 1.0f / (hi - lo[k]) : 0.0f;
  }
}

// grid (i blocks, j chunks of JC): per item i the number of items of the
// chunk ahead of it by score and, per set, by relevance (partial counts
// [chunk][1 + NS][B]); the first chunk's blocks also store rel.
template <int NS>
__global__ __launch_bounds__(kRT) void rank_count_kernel(int B, int JC, const float* __restrict__ s,
                                                         const float* __restrict__ l0,
                                                         const float* __restrict__ l1, float* __restrict__ rel,
                                                         int* __restrict__ cnt) {
  __shared__ float red[kRT / 64];
  extern __shared__ float tj[];  // [1 + NS][JC]: the chunk's scores and relevances
  const float* lab[2] = {l0, l1};
  float lo[NS], ir[NS];
  label_range<NS>(B, lab, lo, ir, red);
  const int i = blockIdx.x * kRT + threadIdx.x;
  const bool ok = i < B;
  const float si = ok ? s[i] : 0.f;
  float ri[NS];
#pragma unroll
  for (int k = 0; k < NS; ++k) ri[k] = ok ? rel_of(lab[k][i], lo[k], ir[k]) : 0.f;
  if (blockIdx.y == 0 && ok) {
#pragma unroll
    for (int k = 0; k < NS; ++k) rel[k * B + i] = ri[k];
  }
  const int j0 = blockIdx.y * JC;
  const int n = min(JC, B - j0);
  for (int jj = threadIdx.x; jj < n; jj += kRT) {
    tj[jj] = s[j0 + jj];
#pragma unroll
    for (int k = 0; k < NS; ++k) tj[(1 + k) * JC + jj] = rel_of(lab[k][j0 + jj], lo[k], ir[k]);
  }
  __syncthreads();
  int ahead = 0, iahead[NS];
#pragma unroll
  for (int k = 0; k < NS; ++k) iahead[k] = 0;
  for (int jj = 0; jj < n; ++jj) {
    const int jg = j0 + jj;
    const float sj = tj[jj];
    ahead += (sj > si || (sj == si && jg < i)) ? 1 : 0;
#pragma unroll
    for (int k = 0; k < NS; ++k) {
      const float rj = tj[(1 + k) * JC + jj];
      iahead[k] += (rj > ri[k] || (rj == ri[k] && jg < i)) ? 1 : 0;
    }
  }
  if (!ok) return;
  int* c = cnt + (int64_t)blockIdx.y * (1 + NS) * B + i;
  c[0] = ahead;
#pragma unroll
  for (int k = 0; k < NS; ++k) c[(int64_t)(1 + k) * B] = iahead[k];
}

// per item: its score rank and, per set, its gain and ideal-DCG term from
// the chunks' counts
template <int NS>
__global__ __launch_bounds__(kRT) void rank_prep_kernel(int B, int chunks, const int* __restrict__ cnt,
                                                        const float* __restrict__ rel, float* __restrict__ gain,
                                                        float* __restrict__ dcg, float* __restrict__ invD) {
  const int i = blockIdx.x * kRT + threadIdx.x;
  if (i >= B) return;
  int ahead = 0, iahead[NS];
#pragma unroll
  for (int k = 0; k < NS; ++k) iahead[k] = 0;
  for (int c = 0; c < chunks; ++c) {
    const int* p = cnt + (int64_t)c * (1 + NS) * B + i;
    ahead += p[0];
#pragma unroll
    for (int k = 0; k < NS; ++k) iahead[k] += p[(int64_t)(1 + k) * B];
  }
  invD[i] = 1.0f / __builtin_amdgcn_logf(2.0f + (float)ahead);  // rank = ahead + 1, D = log2(1 + rank)
#pragma unroll
  for (int k = 0; k < NS; ++k) {
    const float g = __builtin_amdgcn_exp2f(rel[k * B + i]) - 1.0f;
    gain[k * B + i] = g;
    dcg[k * B + i] = g / __builtin_amdgcn_logf(2.0f + (float)iahead[k]);
  }
}

// grid (i blocks, j tiles of JT); part_ds [tiles][B], part_loss [tiles][i blocks][NS]
template <int NS>
__global__ __launch_bounds__(kRT) void rank_pair_kernel(int B, int JT, float sigma, float w0, float w1,
                                                        const float* __restrict__ w1_scale,
                                                        const float* __restrict__ s,
                                                        const float* __restrict__ rel,
                                                        const float* __restrict__ gain,
                                                        const float* __restrict__ dcg,
                                                        const float* __restrict__ invD,
                                                        float* __restrict__ part_ds,
                                                        float* __restrict__ part_loss) {
  __shared__ float red[kRT / 64];
  extern __shared__ float tj[];  // [2 + 2 NS][JT]: scores, 1/D, relevances, gains
  float* ts = tj;
  float* tD = tj + JT;
  float* tr = tj + 2 * JT;            // [NS][JT]
  float* tg = tj + (2 + NS) * JT;     // [NS][JT]
  float imax[NS];
#pragma unroll
  for (int k = 0; k < NS; ++k) {
    float acc = 0.f;
    for (int j = threadIdx.x; j < B; j += kRT) acc += dcg[k * B + j];
    const float mx = block_sum(acc, red);
    imax[k] = mx > 0.f ? 1.0f / mx : 0.f;
  }
  const int j0 = blockIdx.y * JT;
  const int nj = min(JT, B - j0);
  for (int jj = threadIdx.x; jj < nj; jj += kRT) {
    const int j = j0 + jj;
    ts[jj] = s[j];
    tD[jj] = invD[j];
#pragma unroll
    for (int k = 0; k < NS; ++k) {
      tr[k * JT + jj] = rel[k * B + j];
      tg[k * JT + jj] = gain[k * B + j];
    }
  }
  __syncthreads();
  const int i = blockIdx.x * kRT + threadIdx.x;
  const bool ok = i < B;
  const float si = ok ? s[i] : 0.f, Di = ok ? invD[i] : 0.f;
  float ri[NS], gi[NS], loss[NS], grad[NS];
#pragma unroll
  for (int k = 0; k < NS; ++k) {
    ri[k] = ok ? rel[k * B + i] : 0.f;
    gi[k] = ok ? gain[k * B + i] : 0.f;
    loss[k] = 0.f;
    grad[k] = 0.f;
  }
  const int n = ok ? nj : 0;
  for (int jj = 0; jj < n; ++jj) {
    const float x = sigma * (si - ts[jj]);
    const float dD = fabsf(Di - tD[jj]);
    // e = exp(-|x|): sigmoid(-x) and softplus(-x) = log(1 + e^-x) from it
    const float e = exp_fast(-fabsf(x));
    const float r1 = rcp_fast(1.0f + e);
    const float sig_neg = x >= 0.f ? e * r1 : r1;   // 1 / (1 + e^x)
    const float sig_pos = x >= 0.f ? r1 : e * r1;   // 1 / (1 + e^-x)
    const float lp = log1p_unit(e);
    const float sp_neg = fmaxf(-x, 0.f) + lp;      // log(1 + e^-x)
#pragma unroll
    for (int k = 0; k < NS; ++k) {
      const float rj = tr[k * JT + jj];
      const float w = fabsf(gi[k] - tg[k * JT + jj]) * imax[k] * dD;
      if (ri[k] > rj) {
        loss[k] = fmaf(w, sp_neg, loss[k]);
        grad[k] = fmaf(-w, sig_neg, grad[k]);
      } else if (rj > ri[k]) {
        grad[k] = fmaf(w, sig_pos, grad[k]);
      }
    }
  }
  // loss in bits (log2), gradient scaled by sigma / ln 2
  const float c = sigma * kInvLn2;
  if (w1_scale) w1 *= w1_scale[0];
  if (ok) part_ds[(int64_t)blockIdx.y * B + i] = w0 * grad[0] * c + (NS > 1 ? w1 * grad[NS - 1] * c : 0.f);
#pragma unroll
  for (int k = 0; k < NS; ++k) {
    const float t = block_sum(loss[k] * kInvLn2, red);
    if (threadIdx.x == 0) part_loss[((int64_t)blockIdx.y * gridDim.x + blockIdx.x) * NS + k] = t;
  }
}

// ds[i] = sum over j tiles; out: NS == 1: {L}; NS == 2: {w0 L0 + w1 L1, L1, L0}
template <int NS>
__global__ __launch_bounds__(kRT) void rank_finish_kernel(int B, int tiles, int iblocks, float w0, float w1,
                                                          const float* __restrict__ w1_scale,
                                                          const float* __restrict__ part_ds,
                                                          const float* __restrict__ part_loss,
                                                          float* __restrict__ ds, float* __restrict__ out) {
  const int i = blockIdx.x * kRT + threadIdx.x;
  if (i < B && ds) {
    float acc = 0.f;
    for (int t = 0; t < tiles; ++t) acc += part_ds[(int64_t)t * B + i];
    ds[i] = acc;
  }
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    float L[NS];
#pragma unroll
    for (int k = 0; k < NS; ++k) L[k] = 0.f;
    for (int p = 0; p < tiles * iblocks; ++p)
#pragma unroll
      for (int k = 0; k < NS; ++k) L[k] += part_loss[(int64_t)p * NS + k];
    if (NS == 1) {
      out[0] = L[0];
    } else {
      if (w1_scale) w1 *= w1_scale[0];
      out[0] = w0 * L[0] + w1 * L[NS - 1];
      out[1] = L[NS - 1];
      out[2] = L[0];
    }
  }
}

// EWC: grad += lambda F (theta - theta_prev); part[block] = this block's
// share of lambda/2 sum F (theta - theta_prev)^2
constexpr int kEwcBlocks = 256;
__global__ __launch_bounds__(kRT) void ewc_kernel(int64_t n, const float* __restrict__ theta,
                                                  const float* __restrict__ prev,
                                                  const float* __restrict__ fisher, float lam,
                                                  float* __restrict__ grad, float* __restrict__ part) {
  __shared__ float red[kRT / 64];
  float acc = 0.f;
  for (int64_t k = (int64_t)blockIdx.x * kRT + threadIdx.x; k < n; k += (int64_t)kEwcBlocks * kRT) {
    const float d = theta[k] - prev[k];
    const float fd = fisher[k] * d;
    grad[k] = fmaf(lam, fd, grad[k]);
    acc = fmaf(fd, d, acc);
  }
  const float t = block_sum(acc, red);
  if (threadIdx.x == 0) part[blockIdx.x] = 0.5f * lam * t;
}

// loss[3] = the penalty, loss[0] += it
__global__ __launch_bounds__(64) void ewc_finish_kernel(const float* __restrict__ part, float* __restrict__ loss) {
  float acc = 0.f;
  for (int b = threadIdx.x; b < kEwcBlocks; b += 64) acc += part[b];
  acc = wave_sum(acc);
  if (threadIdx.x == 0) {
    loss[3] = acc;
    loss[0] += acc;
  }
}

__global__ void ewc_off_kernel(float* __restrict__ loss) {
  if (threadIdx.x == 0) loss[3] = 0.f;
}

// The teacher-loss gate (Eq. (10)-(11)): phi_j = 1 - (e_j - min e) /
// (max e - min e) over every batch j, one workgroup striding over the n
// losses (a few thousand batches per dataset: latency-bound either way).
// The normalisation runs in fp64 so that each phi_j is the fp32 rounding of
// the exact value; equal losses (max = min) give phi = 1 everywhere.
__global__ __launch_bounds__(kRT) void teacher_gate_kernel(int n, const float* __restrict__ e,
                                                           float* __restrict__ phi) {
  __shared__ float red[kRT / 64];
  float mn = INFINITY, mx = -INFINITY;
  for (int j = threadIdx.x; j < n; j += kRT) {
    mn = fminf(mn, e[j]);
    mx = fmaxf(mx, e[j]);
  }
  const float lo = block_min(mn, red);
  const float hi = block_max(mx, red);
  const double range = (double)hi - (double)lo;
  for (int j = threadIdx.x; j < n; j += kRT)
    phi[j] = range > 0.0 ? (float)(1.0 - ((double)e[j] - (double)lo) / range) : 1.0f;
}

}  // namespace

size_t rank_workspace_floats(int B, int nsets) {
  const size_t iblocks = (size_t)(B + kRT - 1) / kRT;
  const size_t tiles = (size_t)(B + rank_pair_tile(B) - 1) / rank_pair_tile(B);
  const size_t chunks = (size_t)(B + rank_count_chunk(B) - 1) / rank_count_chunk(B);
  // rel, gain, dcg per set; invD; ds; part_ds [tiles][B]; part_loss
  // [tiles][iblocks][nsets]; counts [chunks][1 + nsets][B] (ints)
  return (size_t)3 * nsets * B + B + B + tiles * B + tiles * iblocks * nsets + chunks * (1 + nsets) * B;
}

hipError_t launch_lambdarank(int B, int nsets, const float* s, const float* l0, const float* l1, float sigma,
                             float w0, float w1, float* ws, float* ds, float* out, hipStream_t st,
                             const float* key, const float* w1_scale) {
  if (B <= 0 || (nsets != 1 && nsets != 2) || (nsets == 2 && !l1)) return hipErrorInvalidValue;
  const int iblocks = (B + kRT - 1) / kRT;
  const int JT = rank_pair_tile(B), JC = rank_count_chunk(B);
  const int tiles = (B + JT - 1) / JT, chunks = (B + JC - 1) / JC;
  float* rel = ws;
  float* gain = rel + (size_t)nsets * B;
  float* dcg = gain + (size_t)nsets * B;
  float* invD = dcg + (size_t)nsets * B;
  float* dsw = invD + B;
  float* part_ds = dsw + B;
  float* part_loss = part_ds + (size_t)tiles * B;
  int* cnt = reinterpret_cast<int*>(part_loss + (size_t)tiles * iblocks * nsets);
  float* dsout = ds ? ds : dsw;
  const float* rk = key ? key : s;  // what the score ranks D_i are counted from
  const size_t cnt_lds = (size_t)(1 + nsets) * JC * sizeof(float);
  const size_t pair_lds = (size_t)(2 + 2 * nsets) * JT * sizeof(float);
#define TCL_RANK(NS, L1)                                                                                  \
  do {                                                                                                    \
    hipLaunchKernelGGL(rank_count_kernel<NS>, dim3(iblocks, chunks), dim3(kRT), cnt_lds, st, B, JC, rk, l0, \
                       L1, rel, cnt);                                                                     \
    hipLaunchKernelGGL(rank_prep_kernel<NS>, dim3(iblocks), dim3(kRT), 0, st, B, chunks, cnt, rel, gain,    \
                       dcg, invD);                                                                        \
    hipLaunchKernelGGL(rank_pair_kernel<NS>, dim3(iblocks, tiles), dim3(kRT), pair_lds, st, B, JT, sigma,  \
                       w0, w1, w1_scale, s, rel, gain, dcg, invD, part_ds, part_loss);                    \
    hipLaunchKernelGGL(rank_finish_kernel<NS>, dim3(iblocks), dim3(kRT), 0, st, B, tiles, iblocks, w0, w1, \
                       w1_scale, part_ds, part_loss, dsout, out);                                         \
  } while (0)
  if (nsets == 1) TCL_RANK(1, l0);
  else TCL_RANK(2, l1);
#undef TCL_RANK
  return hipGetLastError();
}

hipError_t launch_teacher_gate(int n, const float* e, float* phi, hipStream_t st) {
  if (n <= 0 || !e || !phi) return hipErrorInvalidValue;
  hipLaunchKernelGGL(teacher_gate_kernel, dim3(1), dim3(kRT), 0, st, n, e, phi);
  return hipGetLastError();
}

int ewc_part_floats() { return kEwcBlocks; }

hipError_t launch_ewc(int64_t n, const float* theta, const float* prev, const float* fisher, float lam,
                      float* grad, float* part, float* loss, hipStream_t st) {
  if (n <= 0) return hipErrorInvalidValue;
  if (lam == 0.f) {  // no penalty: its loss slot reads zero
    hipLaunchKernelGGL(ewc_off_kernel, dim3(1), dim3(64), 0, st, loss);
    return hipGetLastError();
  }
  if (!theta || !prev || !fisher) return hipErrorInvalidValue;
  hipLaunchKernelGGL(ewc_kernel, dim3(kEwcBlocks), dim3(kRT), 0, st, n, theta, prev, fisher, lam, grad, part);
  hipLaunchKernelGGL(ewc_finish_kernel, dim3(1), dim3(64), 0, st, part, loss);
  return hipGetLastError();
}

}  // namespace tcl
