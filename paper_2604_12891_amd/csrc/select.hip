// What consumes the scores: per-segment top-K (the inference phase of
// section 3 keeps the K best candidates of a tuning round) and the RDU
// sampler's selection of programs to label (section 4, Alg. 1, Eq. (1)-(3)).
//
// Top-K: one workgroup of 1,024 threads per segment. Scores map to order-preserving 32-bit
// keys (NaN below everything); a four-pass radix select over 8-bit digits
// finds the K-th largest key; the items above it and the lowest-index items
// equal to it are gathered and bitonic-sorted in LDS by (key descending,
// index ascending).
//
// RDU selection: the greedy loop of Alg. 1, one iteration per selected
// program, on the device (the host only enqueues): a grid pass updates each
// candidate's distance to the labeled set with the last selected program
// (Eq. (1) kept as a running minimum), computes t_s = f d_s + u_s with the
// variance of Eq. (2)-(3) from running sums, and reduces the argmax; a
// one-workgroup pass labels the winner. A candidate whose operator type has
// used its budget can never be labeled, so it is masked out as soon as that
// happens; Alg. 1 drops such candidates one at a time when they come up as
// the argmax, which leaves the same sequence of labeled programs. fp64
// throughout (the normalised predictions, distances, sums and t_s).
#include "common.h"
#include "kernels.h"

namespace tcl {
namespace {

constexpr int kST = 256;  // threads per block

// ---------------------------------------------------------------- top-K
__device__ __forceinline__ uint32_t score_key(float f) {
  if (f != f) return 0u;  // NaN: below every number
  uint32_t u = __float_as_uint(f);
  if ((u << 1) == 0u) u = 0u;  // -0 and +0 are equal scores
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

constexpr int kTK = 1024;  // threads of a top-K workgroup

// block-wide exclusive prefix of a 0/1 flag over the kTK threads (in thread
// order); returns the prefix, *total the block's count
__device__ __forceinline__ int block_prefix(bool flag, int* wsum, int* total) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const uint64_t m = __ballot(flag);
  const int in_wave = __popcll(m & ((1ull << lane) - 1ull));
  __syncthreads();
  if (lane == 0) wsum[w] = __popcll(m);
  __syncthreads();
  int before = 0, all = 0;
#pragma unroll
  for (int i = 0; i < kTK / 64; ++i) {
    before += i < w ? wsum[i] : 0;
    all += wsum[i];
  }
  *total = all;
  return before + in_wave;
}

template <int P>  // P: power of two >= K
__global__ __launch_bounds__(kTK) void topk_kernel(const int* __restrict__ offs, const float* __restrict__ s,
                                                   int K, int* __restrict__ out) {
  __shared__ int hist[kTK / 64][256];  // one histogram per wavefront (scores crowd a few top digits)
  __shared__ int tot[4];
  __shared__ uint64_t cand[P];
  __shared__ int wsum[kTK / 64];
  __shared__ int sdig, sabove, cnt_gt;
  const int g = blockIdx.x;
  const int lo = offs[g];
  const int n = max(offs[g + 1] - lo, 0);
  const int tid = threadIdx.x;
  const int take = min(n, K);

  for (int i = tid; i < P; i += kTK) cand[i] = 0ull;  // padding sorts last
  if (tid == 0) cnt_gt = 0;
  uint32_t kth = 0u;
  int need_eq = take;  // items equal to kth to keep (all, when n <= K)
  if (n > K) {
    uint32_t prefix = 0u, pmask = 0u;
    int krem = K;
    const int wave = tid >> 6;
    for (int shift = 24; shift >= 0; shift -= 8) {
      __syncthreads();
      for (int b = tid; b < (kTK / 64) * 256; b += kTK) (&hist[0][0])[b] = 0;
      __syncthreads();
      for (int i = tid; i < n; i += kTK) {
        const uint32_t key = score_key(s[lo + i]);
        if ((key & pmask) == prefix) atomicAdd(&hist[wave][(key >> shift) & 255], 1);
      }
      __syncthreads();
      // thread t < 256 takes digit 255 - t; an inclusive scan over threads is
      // then the count of keys at or above that digit, and exactly one digit
      // has that count reach krem while the digits above it stay below
      int c = 0, incl = 0;
      if (tid < 256) {
#pragma unroll
        for (int w = 0; w < kTK / 64; ++w) c += hist[w][255 - tid];
        incl = c;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
          const int v = __shfl_up(incl, o, 64);
          if ((tid & 63) >= o) incl += v;
        }
        if ((tid & 63) == 63) tot[tid >> 6] = incl;
      }
      __syncthreads();
      if (tid < 256) {
        for (int w = 0; w < (tid >> 6); ++w) incl += tot[w];
        if (incl >= krem && incl - c < krem) {
          sdig = 255 - tid;
          sabove = incl - c;
        }
      }
      __syncthreads();
      krem -= sabove;
      prefix |= (uint32_t)sdig << shift;
      pmask |= 0xFFu << shift;
    }
    kth = prefix;
    need_eq = krem;
  }
  __syncthreads();
  // gather: every key above kth, then the first need_eq keys equal to it
  int eq_base = 0;
  for (int t0 = 0; t0 < n; t0 += kTK) {
    const int i = t0 + tid;
    const bool ok = i < n;
    const uint32_t key = ok ? score_key(s[lo + i]) : 0u;
    const uint64_t code = ((uint64_t)key << 32) | (uint64_t)(0xFFFFFFFFu - (uint32_t)i);
    const bool gt = ok && n > K && key > kth;
    const bool eq = ok && (n <= K || key == kth);
    if (gt) cand[atomicAdd(&cnt_gt, 1)] = code;
    int tot;
    const int r = block_prefix(eq, wsum, &tot);
    if (eq && eq_base + r < need_eq) cand[(take - need_eq) + eq_base + r] = code;
    eq_base += tot;
  }
  __syncthreads();
  // bitonic sort, descending
  for (int k = 2; k <= P; k <<= 1) {
    for (int j = k >> 1; j > 0; j >>= 1) {
      for (int i = tid; i < P; i += kTK) {
        const int p = i ^ j;
        if (p > i) {
          const uint64_t a = cand[i], b = cand[p];
          const bool desc = (i & k) == 0;
          if (desc ? (a < b) : (a > b)) {
            cand[i] = b;
            cand[p] = a;
          }
        }
      }
      __syncthreads();
    }
  }
  for (int r = tid; r < K; r += kTK)
    out[(int64_t)g * K + r] = r < take ? lo + (int)(0xFFFFFFFFu - (uint32_t)(cand[r] & 0xFFFFFFFFull)) : -1;
}

// ---------------------------------------------------------------- RDU selection
struct RduState {
  double lo, range;  // normalisation of the predictions
  double S1, S2;     // sums of f and f^2 over the labeled set
  int M;             // labeled programs
  int count;         // selected so far
  int last;          // the last selected program (-1: none yet)
  int done;
  int n_select;
  unsigned arrived;  // blocks of the current grid pass that have parked their partial
  int pad_[2];
};

struct Best {
  double t;
  int i;
};

__device__ __forceinline__ bool better(double t, int i, double bt, int bi) {
  return bi < 0 || t > bt || (t == bt && i < bi);
}

__device__ __forceinline__ double fhat(const float* s, int i, const RduState& st) {
  return st.range > 0.0 ? ((double)s[i] - st.lo) / st.range : 0.0;
}

// block argmax of (t, i), lower index on ties; result in thread 0
__device__ Best block_best(double t, int i, double* st, int* si) {
  st[threadIdx.x] = t;
  si[threadIdx.x] = i;
  __syncthreads();
  for (int o = kST / 2; o > 0; o >>= 1) {
    if ((int)threadIdx.x < o) {
      const double t2 = st[threadIdx.x + o];
      const int i2 = si[threadIdx.x + o];
      if (i2 >= 0 && better(t2, i2, st[threadIdx.x], si[threadIdx.x])) {
        st[threadIdx.x] = t2;
        si[threadIdx.x] = i2;
      }
    }
    __syncthreads();
  }
  return Best{st[0], si[0]};
}

// per block: min and max of the scores, and a histogram of operator types
// (types outside [0, n_ops) are counted in opcount[n_ops])
constexpr int kMaxOps = 4096;
__global__ __launch_bounds__(kST) void rdu_stats_kernel(int N, const float* __restrict__ s,
                                                        const int* __restrict__ op, int n_ops,
                                                        float* __restrict__ mm, int* __restrict__ opcount) {
  __shared__ float smin[kST], smax[kST];
  __shared__ int h[kMaxOps + 1];
  for (int o = threadIdx.x; o <= n_ops; o += kST) h[o] = 0;
  __syncthreads();
  float mn = INFINITY, mx = -INFINITY;
  for (int i = blockIdx.x * kST + threadIdx.x; i < N; i += gridDim.x * kST) {
    mn = fminf(mn, s[i]);
    mx = fmaxf(mx, s[i]);
    const int o = op[i];
    atomicAdd(&h[(o >= 0 && o < n_ops) ? o : n_ops], 1);
  }
  __syncthreads();
  for (int o = threadIdx.x; o <= n_ops; o += kST)
    if (h[o]) atomicAdd(&opcount[o], h[o]);
  smin[threadIdx.x] = mn;
  smax[threadIdx.x] = mx;
  __syncthreads();
  for (int o = kST / 2; o > 0; o >>= 1) {
    if ((int)threadIdx.x < o) {
      smin[threadIdx.x] = fminf(smin[threadIdx.x], smin[threadIdx.x + o]);
      smax[threadIdx.x] = fmaxf(smax[threadIdx.x], smax[threadIdx.x + o]);
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    mm[2 * blockIdx.x] = smin[0];
    mm[2 * blockIdx.x + 1] = smax[0];
  }
}

__global__ __launch_bounds__(kST) void rdu_zero_kernel(int n, int* __restrict__ a) {
  for (int i = blockIdx.x * kST + threadIdx.x; i < n; i += gridDim.x * kST) a[i] = 0;
}

// one block: normalisation, budgets, sums over the initial labeled set
__global__ __launch_bounds__(kST) void rdu_setup_kernel(int N, const float* __restrict__ s, int n_ops,
                                                        const int* __restrict__ init, int n_init, int n_select,
                                                        const float* __restrict__ mm, int nmm,
                                                        const int* __restrict__ opcount,
                                                        double* __restrict__ budget, int* __restrict__ sel,
                                                        RduState* __restrict__ state) {
  __shared__ double r1[kST], r2[kST];
  __shared__ int rc[kST];
  __shared__ double slo, srange;
  if (threadIdx.x == 0) {
    float mn = mm[0], mx = mm[1];
    for (int b = 1; b < nmm; ++b) {
      mn = fminf(mn, mm[2 * b]);
      mx = fmaxf(mx, mm[2 * b + 1]);
    }
    slo = (double)mn;
    srange = (double)mx - (double)mn;
  }
  __syncthreads();
  RduState st{};
  st.lo = slo;
  st.range = srange;
  for (int o = threadIdx.x; o < n_ops; o += kST) {
    budget[o] = (double)n_select * (double)opcount[o] / (double)N;
    sel[o] = 0;
  }
  double a1 = 0.0, a2 = 0.0;
  int c = 0;
  for (int j = threadIdx.x; j < n_init; j += kST) {
    const int i = init[j];
    if (i >= 0 && i < N) {
      const double f = fhat(s, i, st);
      a1 += f;
      a2 += f * f;
      ++c;
    }
  }
  r1[threadIdx.x] = a1;
  r2[threadIdx.x] = a2;
  rc[threadIdx.x] = c;
  __syncthreads();
  for (int o = kST / 2; o > 0; o >>= 1) {
    if ((int)threadIdx.x < o) {
      r1[threadIdx.x] += r1[threadIdx.x + o];
      r2[threadIdx.x] += r2[threadIdx.x + o];
      rc[threadIdx.x] += rc[threadIdx.x + o];
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    st.S1 = r1[0];
    st.S2 = r2[0];
    st.M = rc[0];
    st.count = 0;
    st.last = -1;
    st.n_select = n_select;
    st.done = (n_select <= 0 || rc[0] == 0) ? 1 : 0;
    *state = st;
  }
}

// The initial labeled set's normalised predictions, sorted ascending (at
// most kSortInit of them; larger sets use rdu_dinit_kernel's direct pass).
constexpr int kSortInit = 8192;
__global__ __launch_bounds__(1024) void rdu_sort_init_kernel(int N, const float* __restrict__ s,
                                                             const int* __restrict__ init, int n_init,
                                                             const RduState* __restrict__ state,
                                                             double* __restrict__ sorted, int* __restrict__ n_valid) {
  __shared__ double v[kSortInit];
  const RduState st = *state;
  int P = 1;
  while (P < n_init) P <<= 1;
  for (int j = threadIdx.x; j < P; j += 1024) {
    const int i = j < n_init ? init[j] : -1;
    v[j] = (i >= 0 && i < N && s[i] == s[i]) ? fhat(s, i, st) : INFINITY;  // invalid entries sort last
  }
  __syncthreads();
  for (int k = 2; k <= P; k <<= 1) {
    for (int jj = k >> 1; jj > 0; jj >>= 1) {
      for (int i = threadIdx.x; i < P; i += 1024) {
        const int p = i ^ jj;
        if (p > i) {
          const double a = v[i], b = v[p];
          const bool up = (i & k) == 0;
          if (up ? (a > b) : (a < b)) {
            v[i] = b;
            v[p] = a;
          }
        }
      }
      __syncthreads();
    }
  }
  __shared__ int cnt;
  if (threadIdx.x == 0) cnt = 0;
  __syncthreads();
  for (int j = threadIdx.x; j < n_init; j += 1024) {
    sorted[j] = v[j];
    if (v[j] != INFINITY) atomicAdd(&cnt, 1);
  }
  __syncthreads();
  if (threadIdx.x == 0) *n_valid = cnt;
}

// d[i] = min over the initial set of |f_i - f_j|: the nearest value on each
// side of f_i in the sorted set (a binary search) gives the same minimum
__global__ __launch_bounds__(kST) void rdu_dinit_sorted_kernel(int N, const float* __restrict__ s,
                                                               const double* __restrict__ sorted,
                                                               const int* __restrict__ n_valid,
                                                               const RduState* __restrict__ state,
                                                               double* __restrict__ d) {
  const RduState st = *state;
  const int m = *n_valid;
  for (int i = blockIdx.x * kST + threadIdx.x; i < N; i += gridDim.x * kST) {
    if (s[i] != s[i] || m == 0) {
      d[i] = s[i] != s[i] ? -1.0 : INFINITY;
      continue;
    }
    const double fi = fhat(s, i, st);
    int lo = 0, hi = m;  // first index with sorted[idx] >= fi
    while (lo < hi) {
      const int mid = (lo + hi) >> 1;
      if (sorted[mid] < fi) lo = mid + 1; else hi = mid;
    }
    double best = INFINITY;
    if (lo < m) best = fmin(best, fabs(fi - sorted[lo]));
    if (lo > 0) best = fmin(best, fabs(fi - sorted[lo - 1]));
    d[i] = best;
  }
}

// d[i] = min over the initial labeled set of |f_i - f_j|
__global__ __launch_bounds__(kST) void rdu_dinit_kernel(int N, const float* __restrict__ s,
                                                        const int* __restrict__ init, int n_init,
                                                        const RduState* __restrict__ state,
                                                        double* __restrict__ d) {
  __shared__ double tf[kST];
  const RduState st = *state;
  const int i = blockIdx.x * kST + threadIdx.x;
  const double fi = i < N ? fhat(s, i, st) : 0.0;
  double best = INFINITY;
  for (int j0 = 0; j0 < n_init; j0 += kST) {
    __syncthreads();
    const int j = j0 + threadIdx.x;
    const int idx = j < n_init ? init[j] : -1;
    tf[threadIdx.x] = (idx >= 0 && idx < N) ? fhat(s, idx, st) : NAN;
    __syncthreads();
    const int n = min(kST, n_init - j0);
    for (int jj = 0; jj < n; ++jj) {
      const double fj = tf[jj];
      if (fj == fj) best = fmin(best, fabs(fi - fj));
    }
  }
  if (i < N) d[i] = s[i] == s[i] ? best : -1.0;  // an unscored (NaN) program is no candidate
}

// the initial labeled programs are not candidates
__global__ __launch_bounds__(kST) void rdu_mark_kernel(int N, const int* __restrict__ init, int n_init,
                                                       double* __restrict__ d) {
  const int j = blockIdx.x * kST + threadIdx.x;
  if (j < n_init) {
    const int i = init[j];
    if (i >= 0 && i < N) d[i] = -1.0;
  }
}

// one iteration, grid pass: distances, masks, t_s, block argmax; the last
// block to finish reduces the blocks' partials and labels the winner.
// Candidates go four per thread per round, their loads issued together.
constexpr int kRduUnroll = 4;
__global__ __launch_bounds__(kST) void rdu_score_kernel(int N, const float* __restrict__ s,
                                                        const int* __restrict__ op, int n_ops,
                                                        const double* __restrict__ budget,
                                                        int* __restrict__ sel, RduState* __restrict__ state,
                                                        double* __restrict__ d, Best* __restrict__ part,
                                                        int* __restrict__ out) {
  __shared__ double bt[kST];
  __shared__ int bi[kST];
  __shared__ int am_last;
  const RduState st = *state;
  if (st.done) return;
  const double fl = st.last >= 0 ? fhat(s, st.last, st) : 0.0;
  const double inv = 1.0 / (double)(st.M + 1);
  double best_t = 0.0;
  int best_i = -1;
  constexpr int U = kRduUnroll;
  for (int i0 = blockIdx.x * kST * U + threadIdx.x; i0 < N; i0 += gridDim.x * kST * U) {
    double dv[U];
    int ov[U];
    float sv[U];
#pragma unroll
    for (int k = 0; k < U; ++k) {
      const int i = i0 + k * kST;
      const bool ok = i < N;
      dv[k] = ok ? d[i] : -1.0;
      ov[k] = ok ? op[i] : -1;
      sv[k] = ok ? s[i] : 0.f;
    }
#pragma unroll
    for (int k = 0; k < U; ++k) {
      const int i = i0 + k * kST;
      double di = dv[k];
      if (di < 0.0) continue;  // labeled, past the end, or its operator's budget is used up
      const int o = ov[k];
      if (o < 0 || o >= n_ops || (double)sel[o] >= budget[o]) {
        d[i] = -1.0;
        continue;
      }
      const double fi = st.range > 0.0 ? ((double)sv[k] - st.lo) / st.range : 0.0;
      if (st.last >= 0) {
        const double dn = fabs(fi - fl);  // Eq. (1) as a running minimum
        if (dn < di) {
          di = dn;
          d[i] = dn;
        }
      }
      const double mu = (fi + st.S1) * inv;                 // Eq. (2)
      const double u = (fi * fi + st.S2) * inv - mu * mu;   // Eq. (3), from the running sums
      const double t = fi * di + u;
      if (better(t, i, best_t, best_i)) {
        best_t = t;
        best_i = i;
      }
    }
  }
  const Best b = block_best(best_t, best_i, bt, bi);
  if (threadIdx.x == 0) {
    part[blockIdx.x] = b;
    __threadfence();  // the partial is visible before the arrival is counted
    am_last = atomicAdd(&state->arrived, 1u) == gridDim.x - 1;
  }
  __syncthreads();
  if (!am_last) return;

  // the last block: every partial is in; reduce them and label the winner
  __threadfence();
  double t = 0.0;
  int i = -1;
  for (int q = threadIdx.x; q < (int)gridDim.x; q += kST) {
    const Best pq = part[q];
    if (pq.i >= 0 && better(pq.t, pq.i, t, i)) {
      t = pq.t;
      i = pq.i;
    }
  }
  const Best w = block_best(t, i, bt, bi);
  if (threadIdx.x == 0) {
    RduState ns = st;
    ns.arrived = 0;
    if (w.i < 0) {
      ns.done = 1;
    } else {
      const double f = fhat(s, w.i, st);
      out[ns.count] = w.i;
      ns.count += 1;
      ns.M += 1;
      ns.S1 += f;
      ns.S2 += f * f;
      ns.last = w.i;
      sel[op[w.i]] += 1;
      d[w.i] = -1.0;
      if (ns.count >= ns.n_select) ns.done = 1;
    }
    *state = ns;
  }
}

__global__ __launch_bounds__(kST) void rdu_finish_kernel(int n_select, const RduState* __restrict__ state,
                                                         int* __restrict__ out, int* __restrict__ count) {
  const int c = state->count;
  for (int i = threadIdx.x; i < n_select; i += kST)
    if (i >= c) out[i] = -1;
  if (threadIdx.x == 0) *count = c;
}

constexpr int kRduGrid = 1024;  // blocks of the grid passes (grid-stride)

size_t al256(size_t x) { return (x + 255) & ~size_t(255); }

// ---------------------------------------------------------------- Top-k score (Eq. (12))
// One workgroup per segment: the lowest latency of the segment and the
// lowest among its k best-ranked candidates (indices from topk_kernel), each
// times the segment's weight. fp32 latencies and weights multiply exactly in
// fp64. An empty segment contributes (0, 0).
__global__ __launch_bounds__(kST) void topk_score_seg_kernel(const int* __restrict__ offs, int k,
                                                             const int* __restrict__ top,
                                                             const float* __restrict__ lat,
                                                             const float* __restrict__ w,
                                                             double* __restrict__ part) {
  __shared__ float sA[kST / 64], sB[kST / 64];
  const int g = blockIdx.x, tid = threadIdx.x;
  const int lo = offs[g], hi = offs[g + 1];
  float mAll = __builtin_inff(), mTop = __builtin_inff();
  for (int i = lo + tid; i < hi; i += kST) mAll = fminf(mAll, lat[i]);
  for (int j = tid; j < k; j += kST) {
    const int i = top[(int64_t)g * k + j];
    if (i >= 0) mTop = fminf(mTop, lat[i]);
  }
  for (int o = 32; o > 0; o >>= 1) {
    mAll = fminf(mAll, __shfl_xor(mAll, o));
    mTop = fminf(mTop, __shfl_xor(mTop, o));
  }
  if ((tid & 63) == 0) {
    sA[tid >> 6] = mAll;
    sB[tid >> 6] = mTop;
  }
  __syncthreads();
  if (tid == 0) {
    float a = sA[0], b = sB[0];
    for (int v = 1; v < kST / 64; ++v) {
      a = fminf(a, sA[v]);
      b = fminf(b, sB[v]);
    }
    const bool empty = hi <= lo;
    part[2 * g] = empty ? 0.0 : (double)w[g] * (double)a;
    part[2 * g + 1] = empty ? 0.0 : (double)w[g] * (double)b;
  }
}

// One workgroup: both sums over the segments in a fixed order (a strided
// serial pass per thread, then a fixed tree), so the result is deterministic.
__global__ __launch_bounds__(1024) void topk_score_sum_kernel(int n_seg, const double* __restrict__ part,
                                                              double* __restrict__ out) {
  __shared__ double sN[1024], sD[1024];
  const int tid = threadIdx.x;
  double n = 0.0, d = 0.0;
  for (int g = tid; g < n_seg; g += 1024) {
    n += part[2 * g];
    d += part[2 * g + 1];
  }
  sN[tid] = n;
  sD[tid] = d;
  __syncthreads();
  for (int o = 512; o > 0; o >>= 1) {
    if (tid < o) {
      sN[tid] += sN[tid + o];
      sD[tid] += sD[tid + o];
    }
    __syncthreads();
  }
  if (tid == 0) {
    out[0] = sN[0] / sD[0];
    out[1] = sN[0];
    out[2] = sD[0];
  }
}

}  // namespace

size_t topk_score_workspace_bytes(int n_seg, int k) {
  return al256((size_t)n_seg * k * 4) + al256((size_t)n_seg * 2 * 8);
}

hipError_t launch_topk_score(int n_seg, const int* offs, const float* s, const float* lat, const float* w,
                             int k, double* out, void* ws, hipStream_t st) {
  if (n_seg <= 0 || k < 1 || k > 1024) return hipErrorInvalidValue;
  int* top = static_cast<int*>(ws);
  double* part = reinterpret_cast<double*>(static_cast<char*>(ws) + al256((size_t)n_seg * k * 4));
  hipError_t e = launch_topk(n_seg, offs, s, k, top, st);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(topk_score_seg_kernel, dim3(n_seg), dim3(kST), 0, st, offs, k, top, lat, w, part);
  hipLaunchKernelGGL(topk_score_sum_kernel, dim3(1), dim3(1024), 0, st, n_seg, part, out);
  return hipGetLastError();
}

hipError_t launch_topk(int n_seg, const int* offs, const float* s, int K, int* out, hipStream_t st) {
  if (n_seg <= 0 || K < 1 || K > 1024) return hipErrorInvalidValue;
#define TCL_TOPK(PP) hipLaunchKernelGGL((topk_kernel<PP>), dim3(n_seg), dim3(kTK), 0, st, offs, s, K, out)
  if (K <= 64) TCL_TOPK(64);
  else if (K <= 256) TCL_TOPK(256);
  else TCL_TOPK(1024);
#undef TCL_TOPK
  return hipGetLastError();
}

size_t rdu_workspace_bytes(int N, int n_ops) {
  const int grid = std::min((N + kST - 1) / kST, kRduGrid);
  return al256(sizeof(RduState)) + al256((size_t)N * 8) + al256((size_t)n_ops * 8) +
         al256((size_t)(n_ops + 1) * 4) * 2 + al256((size_t)grid * 2 * 4) + al256((size_t)grid * sizeof(Best)) +
         al256((size_t)kSortInit * 8) + 256;
}

hipError_t launch_rdu_select(int N, const float* s, const int* op, int n_ops, const int* init, int n_init,
                             int n_select, int* out, int* count, void* ws, hipStream_t st) {
  if (N <= 0 || n_ops <= 0 || n_ops > kMaxOps || n_init < 0 || n_select < 0) return hipErrorInvalidValue;
  const int grid = std::min((N + kST - 1) / kST, kRduGrid);
  char* p = static_cast<char*>(ws);
  RduState* state = reinterpret_cast<RduState*>(p);
  p += al256(sizeof(RduState));
  double* d = reinterpret_cast<double*>(p);
  p += al256((size_t)N * 8);
  double* budget = reinterpret_cast<double*>(p);
  p += al256((size_t)n_ops * 8);
  int* opcount = reinterpret_cast<int*>(p);
  p += al256((size_t)(n_ops + 1) * 4);
  int* sel = reinterpret_cast<int*>(p);
  p += al256((size_t)(n_ops + 1) * 4);
  float* mm = reinterpret_cast<float*>(p);
  p += al256((size_t)grid * 2 * 4);
  Best* part = reinterpret_cast<Best*>(p);
  p += al256((size_t)grid * sizeof(Best));
  double* sorted = reinterpret_cast<double*>(p);
  p += al256((size_t)kSortInit * 8);
  int* n_valid = reinterpret_cast<int*>(p);

  hipLaunchKernelGGL(rdu_zero_kernel, dim3(std::max(1, std::min((n_ops + kST) / kST, 64))), dim3(kST), 0, st,
                     n_ops + 1, opcount);
  hipLaunchKernelGGL(rdu_stats_kernel, dim3(grid), dim3(kST), 0, st, N, s, op, n_ops, mm, opcount);
  hipLaunchKernelGGL(rdu_setup_kernel, dim3(1), dim3(kST), 0, st, N, s, n_ops, init, n_init, n_select, mm, grid,
                     opcount, budget, sel, state);
  if (n_init <= kSortInit) {
    hipLaunchKernelGGL(rdu_sort_init_kernel, dim3(1), dim3(1024), 0, st, N, s, init, n_init, state, sorted, n_valid);
    hipLaunchKernelGGL(rdu_dinit_sorted_kernel, dim3(grid), dim3(kST), 0, st, N, s, sorted, n_valid, state, d);
  } else {
    hipLaunchKernelGGL(rdu_dinit_kernel, dim3((N + kST - 1) / kST), dim3(kST), 0, st, N, s, init, n_init, state, d);
  }
  if (n_init > 0)
    hipLaunchKernelGGL(rdu_mark_kernel, dim3((n_init + kST - 1) / kST), dim3(kST), 0, st, N, init, n_init, d);
  const int sgrid = std::min((N + kST * kRduUnroll - 1) / (kST * kRduUnroll), kRduGrid);
  for (int it = 0; it < n_select; ++it)
    hipLaunchKernelGGL(rdu_score_kernel, dim3(sgrid), dim3(kST), 0, st, N, s, op, n_ops, budget, sel, state, d,
                       part, out);
  hipLaunchKernelGGL(rdu_finish_kernel, dim3(1), dim3(kST), 0, st, n_select, state, out, count);
  return hipGetLastError();
}

}  // namespace tcl
