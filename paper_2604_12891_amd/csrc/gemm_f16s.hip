// fp32 GEMMs on the fp16 matrix cores with two-part operands: C = rowscale *
// (A W^T) + bias, A and W fp32, with fp32-level accuracy. The fp32 model's
// in_proj (with the RMSNorm prologue) and its gathered input Linear run here.
//
// Two-part fp16 operands. After an exact power-of-two scale that puts it in
// fp16's range, each fp32 value x is held as x = h + 2^-11 l + r with
// h = fp16(x) and l = fp16(2^11 (x - h)): x - h is exact in fp32 and at most
// 2^-11 |x|, and rounding it to l's 11 bits leaves |r| <= 2^-22 |x| (for
// |x| >= 2^-3; smaller scaled values lose bits of l in fp16's subnormal range,
// an absolute error below 2^-36). Of the four products of two such values
// three are kept, h_a h_w + 2^-11 (h_a l_w + l_a h_w), in two accumulators
// (the large products, and the two small ones together):
// fp16 x fp16 products are exact in fp32 and the MFMA accumulates in fp32.
// The dropped 2^-22 l_a l_w and the two operands' r add at most 3 * 2^-22 |a w|
// to each product, 12 units of fp32 rounding (2^-24), against the K units that
// bound an fp32 dot product itself. An fp16 MFMA runs at the bf16 rate, so the
// three products cost half the six of the three-part bf16 split, with the
// operands in two parts instead of three (two thirds of the registers, LDS
// bytes and fragment reads).
//
// Scales: each row of A by 2^eA, taken from the row's RMS (RMSNorm prologue:
// scaled values below 2 * 16 * 2^8 for K <= 256) or from its largest value
// (below 2^15); W by 2^10 when its parts are derived (the model routes a
// matrix here only if every |w| < 32, so the scaled W stays below 2^15). The
// epilogue multiplies by 2^-(eA + 10) (exact) and by the RMSNorm factor.
//
// Row panels of 128 rows, 4 wavefronts of 32 rows, each holding its rows'
// two parts over the whole K (up to 256) as MFMA fragments in registers; W's
// two parts stream through a double-buffered LDS stage 32 columns at a time
// (one barrier per block; the next block loaded in two halves and staged
// halfway through and at the end of the current block's MFMAs). A workgroup
// takes 68 KB of LDS and at most 256 registers per lane, so two share a CU:
// up to 512 panels run at once (61,715 token rows are 483 panels, one round),
// and on each SIMD one workgroup's wavefront issues while the other's waits.
// Fragment k-order (A and W alike): k-step s, lane half g holds k = 16 s +
// 8 g .. +7.
#include <algorithm>
#include <type_traits>

#include "common.h"
#include "kernels.h"

namespace tcl {
namespace {

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kWaves = 4;
constexpr int kNT = kWaves * 64;
constexpr int kBM = kWaves * 32;
constexpr uint32_t kBufferFlags = 0x00020000;  // 32-bit data format, raw (stride 0)
constexpr uint32_t kOutOfRange = 0x80000000u;  // beyond every resource used here
constexpr float kLowInv = 1.0f / kF16LowScale;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, bytes, kBufferFlags);
}

// 2^e as a float, e in [-126, 127]
__device__ __forceinline__ float pow2f(int e) { return __uint_as_float((uint32_t)(e + 127) << 23); }

// floor(log2(x)) for a positive normal float (the exponent field); -127 for 0
__device__ __forceinline__ int exponent_of(float x) { return (int)((__float_as_uint(x) >> 23) & 0xFF) - 127; }

// 8 scaled fp32 values -> their two fp16 parts (FLAT: the low part unscaled)
template <bool FLAT = false>
__device__ __forceinline__ void split8_f16(const float* x, f16x8& h, f16x8& l) {
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const _Float16 hj = (_Float16)x[j];
    h[j] = hj;
    l[j] = FLAT ? (_Float16)(x[j] - (float)hj) : (_Float16)((x[j] - (float)hj) * kF16LowScale);
  }
}

template <int KS, int FL>
__global__ __launch_bounds__(kNT, 2) void gemm_f16s_kernel(GemmArgs p, const uint16_t* Wh, int ldwh) {
  constexpr int RU = 2 * KS;                             // 16-byte units (8 k) of a W row
  constexpr int RUP = RU <= 8 ? 8 : RU <= 16 ? 16 : 32;  // a staged row: a power of two
  constexpr int SWZ = (RUP < 16 ? RUP : 16) - 1;         // unit swizzle of a staged row
  constexpr int PARTU = 32 * RUP;                        // units of one part of one buffer
  constexpr int BUFU = 2 * PARTU;                        // units of one buffer (a column block)
  constexpr int NI = BUFU / kNT;                         // loads per lane per block
  constexpr bool kNorm = (FL & kRowNorm) != 0;
  // vector memory operations a block issues after its successor's W loads:
  // at least the epilogue's 16 stores (vector memory operations complete in
  // order, so waiting until at most that many are outstanding waits for the
  // loads; a bias load among them only makes the wait stricter)
  constexpr int kAfterLoads = 16;
  static_assert((FL & kResid) == 0, "no residual epilogue");
  static_assert(RU <= 32 && NI * kNT == BUFU, "K up to 256");

  __shared__ __attribute__((aligned(16))) uint16_t sW[2 * BUFU * 8];
  __shared__ float sF[kWaves][32];
  __shared__ int sSrc[kBM];

  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63;
  const int li = lane & 31, lg = lane >> 5;
  const int M = p.Mdev ? *p.Mdev : p.Mmax;
  const int row0 = blockIdx.x * kBM;
  if (row0 >= M) return;

  for (int r = tid; r < kBM; r += kNT) {
    const int grow = row0 + r;
    int src = grow < M ? grow : -1;
    if constexpr ((FL & kGather) != 0) {
      if (src >= 0) {
        int lo = 0, hi = p.B;
        while (hi - lo > 1) {
          const int mid = (lo + hi) >> 1;
          if (p.offs[mid] <= grow) lo = mid; else hi = mid;
        }
        src = lo * p.L + (grow - p.offs[lo]);
        if (p.tpos) p.tpos[grow] = (uint8_t)min(grow - p.offs[lo], 255);
      }
    }
    sSrc[r] = src;
  }

  const __amdgpu_buffer_rsrc_t wres = make_rsrc(Wh, (uint32_t)__builtin_amdgcn_readfirstlane(2 * p.N * ldwh * 2));
  // this workgroup's column blocks [sb, se): all of them, or one of
  // gridDim.y ranges when a small batch leaves too few panels for the GPU
  const int nblk = (p.N + 31) / 32;
  const int sb = (int)(blockIdx.y * nblk / gridDim.y), se = (int)((blockIdx.y + 1) * nblk / gridDim.y);

  // W goes from memory straight into LDS (buffer_load ... lds: lane l of a
  // load writes the 16 bytes at the load's base + 16 l, whatever unit it
  // reads). Staged layout: [part][row 32][RUP units], unit u of row r at
  // position u ^ (r & SWZ), so that a fragment read (32 rows, one unit each,
  // per half-wavefront) touches every bank once. A unit with no data (k past
  // ldwh: A is zero there; rows past N: columns never stored) loads W's
  // first unit instead.
  using lds_ptr = __attribute__((address_space(3))) void*;
  auto wdma = [&](int n0, int buf) {
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int f = (wave * NI + i) * 64 + lane;  // staged position this lane writes
      const int part = f / PARTU, row = (f / RUP) % 32, u = (f % RUP) ^ (row & SWZ);
      const int n = n0 + row, k = 8 * u;
      const bool ok = u < RU && n < p.N && k < ldwh;
      const uint32_t off = ok ? (uint32_t)(((part * p.N + n) * ldwh + k) * 2) : 0u;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(wres, (lds_ptr)&sW[(buf * BUFU + (wave * NI + i) * 64) * 8], 16,
                                               off, 0, 0, 0);
    }
  };
  // a wavefront's wait for its own W loads: at most `after` vector memory
  // operations (issued after them) still outstanding
  auto wait_vm = [](auto after) {
    constexpr int n = decltype(after)::value;
    __builtin_amdgcn_s_waitcnt((n & 15) | (7 << 4) | (15 << 8) | ((n >> 4) << 14));
  };
  __syncthreads();   // sSrc
  wdma(sb * 32, 0);  // in flight during the prologue (after the barrier, which would wait for it)

  // prologue: row li of this wavefront's 32, lane half lg's 8 k of every
  // k-step, scaled by a power of two and split into its two fp16 parts
  f16x8 ah[KS], al[KS];
  {
    const int src = sSrc[wave * 32 + li];
    const float* arow = p.A + (src >= 0 ? (int64_t)src * p.lda : 0);
    float x[KS][8];
    float ss = 0.f, mx = 0.f;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      const int k = 16 * s + 8 * lg;
      const bool ok0 = src >= 0 && k < p.K, ok1 = src >= 0 && k + 4 < p.K;
      floatx4 v0 = *reinterpret_cast<const floatx4*>(arow + (ok0 ? k : 0));
      floatx4 v1 = *reinterpret_cast<const floatx4*>(arow + (ok1 ? k + 4 : 0));
      if (!ok0) v0 = floatx4{0.f, 0.f, 0.f, 0.f};
      if (!ok1) v1 = floatx4{0.f, 0.f, 0.f, 0.f};
      x[s][0] = v0.x; x[s][1] = v0.y; x[s][2] = v0.z; x[s][3] = v0.w;
      x[s][4] = v1.x; x[s][5] = v1.y; x[s][6] = v1.z; x[s][7] = v1.w;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        if constexpr (kNorm) ss = fmaf(x[s][j], x[s][j], ss);
        else mx = fmaxf(mx, fabsf(x[s][j]));
      }
    }
    int eA;
    float f;
    if constexpr (kNorm) {
      ss += __shfl_xor(ss, 32, 64);  // the other half of the row
      const float ms = ss / (float)p.K;
      // the scaled row's RMS in [2^8, 2^9): every value below 2^8 * 2 sqrt(K)
      eA = ms > 0.f ? min(8 - exponent_of(sqrtf(ms)), 100) : 0;
      f = pow2f(-(eA + kF16WeightExp)) * (1.0f / sqrtf(ms + p.eps));
    } else {
      mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
      // the scaled row's largest value in [2^14, 2^15)
      eA = mx > 0.f ? min(14 - exponent_of(mx), 100) : 0;
      f = pow2f(-(eA + kF16WeightExp));
    }
    const float sc = pow2f(eA);
#pragma unroll
    for (int s = 0; s < KS; ++s) {
#pragma unroll
      for (int j = 0; j < 8; ++j) x[s][j] *= sc;
      split8_f16(x[s], ah[s], al[s]);
    }
    if (lg == 0) sF[wave][li] = f;
  }

  const uint32_t panel_bytes = (uint32_t)(min(kBM, M - row0) * p.ldc * 4);
  const __amdgpu_buffer_rsrc_t cres = make_rsrc(p.C + (int64_t)row0 * p.ldc, panel_bytes);

  for (int s = sb; s < se; ++s) {
    const int buf = (s - sb) & 1, n0 = s * 32;
    // block s in LDS: this wavefront's loads of it are done (only the
    // previous block's stores and bias load came after them), then every
    // wavefront's; every wavefront is past block s-1, so the other buffer
    // is free for block s+1
    if (s == sb) wait_vm(std::integral_constant<int, 0>{});
    else wait_vm(std::integral_constant<int, kAfterLoads>{});
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
    if (s + 1 < se) wdma(n0 + 32, buf ^ 1);
    __builtin_amdgcn_sched_barrier(0);

    floatx16 am, ax;
#pragma unroll
    for (int r = 0; r < 16; ++r) am[r] = ax[r] = 0.f;
    const uint16_t* wb = &sW[(buf * BUFU + li * RUP) * 8];
    const int wsw = lg ^ (li & SWZ);  // unit 2 ks + lg of row li sits at 2 ks ^ wsw
    auto wfrag = [&](int part, int ks) {
      return __builtin_bit_cast(f16x8, *reinterpret_cast<const u32x4*>(wb + (part * PARTU + ((2 * ks) ^ wsw)) * 8));
    };
    // W fragments one k-step ahead of their MFMAs (the other workgroup's
    // wavefront on the SIMD covers the rest of the LDS latency)
    f16x8 q[2][2];
    q[0][0] = wfrag(0, 0);
    q[0][1] = wfrag(1, 0);
    __builtin_amdgcn_sched_group_barrier(0x0100, 2, 0);
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      if (ks + 1 < KS) {
        q[(ks + 1) & 1][0] = wfrag(0, ks + 1);
        q[(ks + 1) & 1][1] = wfrag(1, ks + 1);
      }
      const f16x8* w = q[ks & 1];
      // the small products' chain between the two MFMAs of the large one's
      ax = __builtin_amdgcn_mfma_f32_32x32x16_f16(ah[ks], w[1], ax, 0, 0, 0);
      am = __builtin_amdgcn_mfma_f32_32x32x16_f16(ah[ks], w[0], am, 0, 0, 0);
      ax = __builtin_amdgcn_mfma_f32_32x32x16_f16(al[ks], w[0], ax, 0, 0, 0);
      if (ks + 1 < KS) __builtin_amdgcn_sched_group_barrier(0x0100, 2, 0);
      __builtin_amdgcn_sched_group_barrier(0x0008, 3, 0);
    }

    // epilogue: lane l holds column l % 32 and rows 8*(r/4) + 4*(l/32) + (r%4)
    const int col = n0 + li;
    const bool cok = col < p.N;
    const float bias = ((FL & kBias) != 0) ? p.bias[cok ? col : 0] : 0.f;
    // the block's rows: row-major with leading dimension ldc, or (kXBlk) in
    // its channel block (64 floats a row) or in the packed rest
    __amdgpu_buffer_rsrc_t bres = cres;
    int64_t bld = p.ldc;
    int bcol = col;
    if constexpr ((FL & kXBlk) != 0) {
      const int rows = min(kBM, M - row0);
      if (n0 < p.xblk_cols) {
        bres = make_rsrc(p.C + ((int64_t)(n0 / 64) * p.xblk_rows + row0) * 64, (uint32_t)(rows * 64 * 4));
        bld = 64;
        bcol = col % 64;
      } else {
        const int nz = p.N - p.xblk_cols;
        bres = make_rsrc(p.C + (int64_t)p.xblk_cols * p.xblk_rows + (int64_t)row0 * nz, (uint32_t)(rows * nz * 4));
        bld = nz;
        bcol = col - p.xblk_cols;
      }
    }
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int rl = 8 * (r >> 2) + 4 * lg + (r & 3);
      float v = fmaf(ax[r], kLowInv, am[r]) * sF[wave][rl] + bias;
      if (p.relu) v = fmaxf(v, 0.f);
      // rows past M fall outside the resource
      const uint32_t off = cok ? (uint32_t)(((wave * 32 + rl) * bld + bcol) * 4) : kOutOfRange;
      __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, v), bres, off, 0, 0);
    }
  }
}

// ---------------------------------------------------------------- columns in registers (out_proj)
// 128-row panels (32 rows per wavefront) whose accumulators for up to 128
// columns stay in registers while K (up to 512) is walked in chunks of 128:
// out_proj with its residual epilogue. N <= 256 columns are split over two
// (or, for small batches, four) workgroups per panel, and two workgroups
// share a CU (one, holding all 256 columns, left the MFMAs idle while its
// single wavefront per SIMD waited for A: 8-12% slower). With the
// accumulators taking most registers there is no room for a second set, so
// the low parts are unscaled (l = fp16(x - h), for A and for W:
// split2_f16_flat) and all three part products go into one accumulator;
// x - h stays in fp16's normal range for every value above 2^-17 of the
// chunk's largest (after its scale), and W's scale puts every weight above
// 2^-13 there. A row's values are not all known when its first chunk
// is split, so the row scale runs: chunk c is scaled by 2^e with e the
// smallest of (14 - the exponent of each chunk's largest value so far), and
// when e drops the accumulators already holding earlier chunks are
// multiplied by the power of two between the old and the new scale (exact).
// Column blocks go in pairs whose MFMAs alternate between the two blocks'
// accumulators (no MFMA waits for the one before it), one barrier per pair,
// W staged through a ring of four one-block LDS buffers: the next pair's
// first block staged a quarter of the way through the pair's k-steps, its
// second at three quarters.
template <int KCH, int NB, int FL>
__global__ __launch_bounds__(kNT, 2) void gemm_f16acc_kernel(GemmArgs p, const uint16_t* Wh, int ldwh) {
  constexpr int NS = 8;              // 16-k MFMA steps per chunk of 128
  constexpr int RU = 16;             // 16-byte units (8 k) of a W row of a chunk
  constexpr int RP = RU + 1;         // staged row pitch in units (conflict-free fragment reads)
  constexpr int PARTU = 32 * RP;     // units of one part of one block buffer
  constexpr int BUFU = 2 * PARTU;    // units of one block buffer
  constexpr int NQ = BUFU / 64;      // 64-unit loads per block (17), spread over the wavefronts
  static_assert(NB % 2 == 0 && NB >= 2, "column blocks go in pairs");
  static_assert((FL & (kRowNorm | kGather)) == 0, "plain, bias and residual GEMMs only");

  __shared__ __attribute__((aligned(16))) uint16_t sW[4 * BUFU * 8];

  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63;
  const int li = lane & 31, lg = lane >> 5;
  const int M = p.Mdev ? *p.Mdev : p.Mmax;
  // the columns split over CS workgroups per panel (NB blocks of 32 each).
  // Workgroups go to the 8 XCDs round-robin: the CS workgroups of a panel
  // take consecutive slots on one XCD, so the panel's A is read from HBM
  // once and then hits that XCD's L2
  const int CS = ((p.N + 31) / 32 + NB - 1) / NB;
  const int xcd = blockIdx.x & 7, j = blockIdx.x >> 3;
  const int row0 = ((j / CS) * 8 + xcd) * kBM;
  if (row0 >= M) return;
  const int cb = (j % CS) * NB * 32;

  const __amdgpu_buffer_rsrc_t wres = make_rsrc(Wh, (uint32_t)__builtin_amdgcn_readfirstlane(2 * p.N * ldwh * 2));
  // W's blocks go from memory straight into a ring of four LDS buffers
  // (buffer_load ... lds: lane l of a load writes the 16 bytes at the load's
  // base + 16 l), rows at a pitch of 17 units so that a fragment read
  // touches every bank once; the pad unit and a unit with no data (k past
  // ldwh: A is zero there; rows past N: columns never stored) load W's first
  // unit instead.
  using lds_ptr = __attribute__((address_space(3))) void*;
  auto wdma = [&](int n0, int k0, int buf) {
#pragma unroll
    for (int i = 0; i < (NQ + kWaves - 1) / kWaves; ++i) {
      const int q = i * kWaves + wave;  // this wavefront's i-th load of the block (uniform)
      if (q < NQ) {
        const int f = q * 64 + lane;
        const int part = f / PARTU, row = (f / RP) % 32, u = f % RP;
        const int n = n0 + row, k = k0 + 8 * u;
        const bool ok = u < RU && n < p.N && k < ldwh;
        const uint32_t off = ok ? (uint32_t)(((part * p.N + n) * ldwh + k) * 2) : 0u;
        __builtin_amdgcn_raw_ptr_buffer_load_lds(wres, (lds_ptr)&sW[(buf * BUFU + q * 64) * 8], 16, off, 0, 0, 0);
      }
    }
  };
  wdma(cb, 0, 0);
  wdma(cb + 32, 0, 1);

  const int grow = row0 + wave * 32 + li;
  const bool rok = grow < M;
  const float* arow = p.A + (rok ? (int64_t)grow * p.lda : 0);

  floatx16 acc[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[nb][r] = 0.f;
  int erun = 100;  // this lane's row's running scale exponent

#pragma unroll
  for (int c = 0; c < KCH; ++c) {
    // keep the next chunk's loads of A below this point: hoisted, they would
    // hold a second chunk in registers
    __builtin_amdgcn_sched_barrier(0);
    f16x8 ah[NS], al[NS];
    {
      float x[NS][8];
      float mx = 0.f;
#pragma unroll
      for (int s = 0; s < NS; ++s) {
        const int k = c * 128 + 16 * s + 8 * lg;
        const bool ok0 = rok && k < p.K, ok1 = rok && k + 4 < p.K;
        floatx4 v0 = *reinterpret_cast<const floatx4*>(arow + (ok0 ? k : 0));
        floatx4 v1 = *reinterpret_cast<const floatx4*>(arow + (ok1 ? k + 4 : 0));
        if (!ok0) v0 = floatx4{0.f, 0.f, 0.f, 0.f};
        if (!ok1) v1 = floatx4{0.f, 0.f, 0.f, 0.f};
        x[s][0] = v0.x; x[s][1] = v0.y; x[s][2] = v0.z; x[s][3] = v0.w;
        x[s][4] = v1.x; x[s][5] = v1.y; x[s][6] = v1.z; x[s][7] = v1.w;
#pragma unroll
        for (int j = 0; j < 8; ++j) mx = fmaxf(mx, fabsf(x[s][j]));
      }
      mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
      // 14 - exponent puts the chunk's largest value in [2^14, 2^15) (at least
      // -113 for finite values); rows of values below 2^-86 are scaled by 2^100
      const int ec = mx > 0.f ? min(14 - exponent_of(mx), 100) : 100;
      const int enew = min(erun, ec);
      if (c > 0) {
        // accumulator entry r of this lane is row 8 (r / 4) + 4 lg + r % 4,
        // whose scale exponents are held by lane (that row) of the wavefront
        const int dlt = enew - erun;  // <= 0
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int rl = 8 * (r >> 2) + 4 * lg + (r & 3);
          const float f = pow2f(max(__shfl(dlt, rl, 64), -126));
#pragma unroll
          for (int nb = 0; nb < NB; ++nb) acc[nb][r] *= f;
        }
      }
      erun = enew;
      const float sc = pow2f(erun);
#pragma unroll
      for (int s = 0; s < NS; ++s) {
#pragma unroll
        for (int j = 0; j < 8; ++j) x[s][j] *= sc;
        split8_f16<true>(x[s], ah[s], al[s]);
      }
    }
#pragma unroll
    for (int pp = 0; pp < NB / 2; ++pp) {
      const int g = c * NB + 2 * pp;  // global index of the pair's first block
      // this pair in LDS: this wavefront's loads of it are done (no vector
      // memory operation is outstanding here but them: the chunk's A loads
      // were waited for), then every wavefront's; every wavefront is past the
      // previous pair, whose buffers take the next pair
      __builtin_amdgcn_s_waitcnt((7 << 4) | (15 << 8));  // vmcnt(0)
      __builtin_amdgcn_s_barrier();
      const bool more = pp + 1 < NB / 2 || c + 1 < KCH;
      const int ncol = cb + (pp + 1 < NB / 2 ? (2 * pp + 2) * 32 : 0);
      const int nk = pp + 1 < NB / 2 ? c * 128 : (c + 1) * 128;
      if (more) {
        wdma(ncol, nk, (g + 2) & 3);
        wdma(ncol + 32, nk, (g + 3) & 3);
      }

      const uint16_t* wb0 = &sW[((g & 3) * BUFU + li * RP + lg) * 8];
      const uint16_t* wb1 = &sW[(((g + 1) & 3) * BUFU + li * RP + lg) * 8];
      auto wfrag = [&](const uint16_t* wb, int part, int ks) {
        return __builtin_bit_cast(f16x8, *reinterpret_cast<const u32x4*>(wb + (part * PARTU + 2 * ks) * 8));
      };
      f16x8 q[2][4];
      q[0][0] = wfrag(wb0, 0, 0);
      q[0][1] = wfrag(wb0, 1, 0);
      q[0][2] = wfrag(wb1, 0, 0);
      q[0][3] = wfrag(wb1, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x0100, 4, 0);
      floatx16& x0 = acc[2 * pp];
      floatx16& x1 = acc[2 * pp + 1];
#pragma unroll
      for (int ks = 0; ks < NS; ++ks) {
        if (ks + 1 < NS) {
          q[(ks + 1) & 1][0] = wfrag(wb0, 0, ks + 1);
          q[(ks + 1) & 1][1] = wfrag(wb0, 1, ks + 1);
          q[(ks + 1) & 1][2] = wfrag(wb1, 0, ks + 1);
          q[(ks + 1) & 1][3] = wfrag(wb1, 1, ks + 1);
        }
        const f16x8* w = q[ks & 1];
        // the small part products first, the large last
        x0 = __builtin_amdgcn_mfma_f32_32x32x16_f16(al[ks], w[0], x0, 0, 0, 0);
        x1 = __builtin_amdgcn_mfma_f32_32x32x16_f16(al[ks], w[2], x1, 0, 0, 0);
        x0 = __builtin_amdgcn_mfma_f32_32x32x16_f16(ah[ks], w[1], x0, 0, 0, 0);
        x1 = __builtin_amdgcn_mfma_f32_32x32x16_f16(ah[ks], w[3], x1, 0, 0, 0);
        x0 = __builtin_amdgcn_mfma_f32_32x32x16_f16(ah[ks], w[0], x0, 0, 0, 0);
        x1 = __builtin_amdgcn_mfma_f32_32x32x16_f16(ah[ks], w[2], x1, 0, 0, 0);
        if (ks + 1 < NS) __builtin_amdgcn_sched_group_barrier(0x0100, 4, 0);
        __builtin_amdgcn_sched_group_barrier(0x0008, 6, 0);
      }
    }
  }

  // epilogue: lane l holds column nb*32 + l % 32 and rows 8*(r/4) + 4*(l/32) + (r%4)
  const uint32_t panel_bytes = (uint32_t)(min(kBM, M - row0) * p.ldc * 4);
  const __amdgpu_buffer_rsrc_t cres = make_rsrc(p.C + (int64_t)row0 * p.ldc, panel_bytes);
  const __amdgpu_buffer_rsrc_t rres =
      make_rsrc((p.R ? p.R : p.C) + (int64_t)row0 * p.ldc, (FL & kResid) != 0 ? panel_bytes : 0);
  float fr[16];
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const int rl = 8 * (r >> 2) + 4 * lg + (r & 3);
    fr[r] = pow2f(-(__shfl(erun, rl, 64) + kF16WeightExp));
  }
  // every column block's residuals are loaded before the first store: the
  // residual is read in place (R = C), so the compiler keeps loads after
  // earlier stores, and each block's loads would otherwise wait for the
  // previous block's stores to complete
  float res[NB][16];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    const int col = cb + nb * 32 + li;
    const bool cok = col < p.N;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int rl = 8 * (r >> 2) + 4 * lg + (r & 3);
      const uint32_t off = cok ? (uint32_t)(((wave * 32 + rl) * p.ldc + col) * 4) : kOutOfRange;
      res[nb][r] = ((FL & kResid) != 0)
                       ? __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rres, off, 0, 0))
                       : 0.f;
    }
  }
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    const int col = cb + nb * 32 + li;
    const bool cok = col < p.N;
    const float bias = ((FL & kBias) != 0) ? p.bias[cok ? col : 0] : 0.f;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int rl = 8 * (r >> 2) + 4 * lg + (r & 3);
      float v = fmaf(acc[nb][r], fr[r], bias + res[nb][r]);
      if (p.relu) v = fmaxf(v, 0.f);
      const uint32_t off = cok ? (uint32_t)(((wave * 32 + rl) * p.ldc + col) * 4) : kOutOfRange;
      __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, v), cres, off, 0, 0);
    }
  }
}

template <int FL>
hipError_t launch_f16s(const GemmArgs& a, const uint16_t* Wh, int ldwh, hipStream_t s) {
  const int grid = (a.Mmax + kBM - 1) / kBM;
  if (grid <= 0) return hipSuccess;
  // two workgroups per CU: with fewer than two panels per CU the columns are
  // also split, up to 8 ways (each workgroup repeats its panel's prologue)
  const int nblk = (a.N + 31) / 32;
  const int cs = std::max(1, std::min({8, nblk, 512 / grid}));
  const dim3 g(grid, cs);
#define TCL_F16S(KS)                                                                        \
  hipLaunchKernelGGL((gemm_f16s_kernel<KS, FL>), g, dim3(kNT), 0, s, a, Wh, ldwh); \
  break
  switch ((a.K + 15) / 16) {
    case 4: TCL_F16S(4);
    case 8: TCL_F16S(8);
    case 11: TCL_F16S(11);
    case 12: TCL_F16S(12);
    case 16: TCL_F16S(16);
    default: return hipErrorInvalidValue;
  }
#undef TCL_F16S
  return hipGetLastError();
}

// W -> its two fp16 parts after the 2^10 scale, [2][N][ldw], the padding k >= K zero
__global__ __launch_bounds__(256) void split_weights_f16_kernel(const float* __restrict__ W, int N, int K,
                                                                int ldw, uint16_t* __restrict__ out, int flat) {
  const int64_t n_all = (int64_t)N * ldw;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n_all; i += (int64_t)gridDim.x * 256) {
    const int n = (int)(i / ldw), k = (int)(i % ldw);
    const float v = k < K ? W[(int64_t)n * K + k] : 0.f;
    uint16_t h, l;
    if (flat)
      split2_f16_flat(v, h, l);
    else
      split2_f16_scaled(v, h, l);
    out[i] = h;
    out[n_all + i] = l;
  }
}

}  // namespace

template <int FL>
hipError_t launch_f16acc(const GemmArgs& a, const uint16_t* Wh, int ldwh, hipStream_t s) {
  const int grid = (a.Mmax + kBM - 1) / kBM;
  if (grid <= 0) return hipSuccess;
  const int nb = (a.N + 31) / 32;
  // at most 128 columns per workgroup (two workgroups per CU); a batch with
  // fewer panels than two per CU splits 256 columns over 4 workgroups per
  // panel instead of 2 (each repeats its panel's A chunks, from L2)
  const bool small = 512 / grid >= 4;
#define TCL_F16ACC(KCH, NB, CS) \
  hipLaunchKernelGGL((gemm_f16acc_kernel<KCH, NB, FL>), dim3(8 * (CS) * ((grid + 7) / 8)), dim3(kNT), 0, s, a, Wh, ldwh)
#define TCL_F16ACC_K(KCH)                       \
  if (nb <= 2) TCL_F16ACC(KCH, 2, 1);           \
  else if (nb <= 4) TCL_F16ACC(KCH, 2, 2);      \
  else if (small) TCL_F16ACC(KCH, 2, 4);        \
  else TCL_F16ACC(KCH, 4, 2);
  switch ((a.K + 127) / 128) {
    case 1: TCL_F16ACC_K(1); break;
    case 2: TCL_F16ACC_K(2); break;
    case 3: TCL_F16ACC_K(3); break;
    case 4: TCL_F16ACC_K(4); break;
    default: return hipErrorInvalidValue;
  }
#undef TCL_F16ACC_K
#undef TCL_F16ACC
  return hipGetLastError();
}

bool gemm_f16s_supports(const GemmArgs& a, int flags) {
  const int ks = (a.K + 15) / 16;
  const bool kfit = ks == 4 || ks == 8 || ks == 11 || ks == 12 || ks == 16;
  const bool fl = flags == kRowNorm || flags == (kBias | kGather) || flags == kBias || flags == 0 ||
                  (flags == (kRowNorm | kXBlk) && a.xblk_cols > 0 && a.xblk_cols % 64 == 0 &&
                   a.xblk_cols < a.N && a.xblk_rows >= a.Mmax && (int64_t)kBM * 64 * 4 < (1ll << 31) &&
                   (int64_t)kBM * (a.N - a.xblk_cols) * 4 < (1ll << 31) && reinterpret_cast<uintptr_t>(a.C) % 16 == 0);
  return kfit && fl && a.K % 4 == 0 && a.lda % 4 == 0 && reinterpret_cast<uintptr_t>(a.A) % 16 == 0 &&
         // byte offsets of the buffer resources stay below 2^31
         (int64_t)2 * a.N * ((a.K + 7) & ~7) * 2 < (1ll << 31) && (int64_t)kBM * a.ldc * 4 < (1ll << 31);
}

hipError_t launch_gemm_f16s(const GemmArgs& a, const uint16_t* Wh, int ldwh, int flags, hipStream_t s) {
  if (!gemm_f16s_supports(a, flags) || ldwh < a.K || ldwh % 8) return hipErrorInvalidValue;
  switch (flags) {
    case 0: return launch_f16s<0>(a, Wh, ldwh, s);
    case kBias: return launch_f16s<kBias>(a, Wh, ldwh, s);
    case kRowNorm: return launch_f16s<kRowNorm>(a, Wh, ldwh, s);
    case kRowNorm | kXBlk: return launch_f16s<kRowNorm | kXBlk>(a, Wh, ldwh, s);
    case kBias | kGather: return launch_f16s<kBias | kGather>(a, Wh, ldwh, s);
    default: return hipErrorInvalidValue;
  }
}

bool gemm_f16acc_supports(const GemmArgs& a, int flags) {
  const bool fl = flags == 0 || flags == kBias || flags == kResid;
  return fl && a.K % 4 == 0 && a.K <= 512 && a.N >= 1 && a.N <= 256 && a.lda % 4 == 0 &&
         reinterpret_cast<uintptr_t>(a.A) % 16 == 0 && (int64_t)2 * a.N * ((a.K + 7) & ~7) * 2 < (1ll << 31) &&
         (int64_t)kBM * a.ldc * 4 < (1ll << 31);
}

hipError_t launch_gemm_f16acc(const GemmArgs& a, const uint16_t* Wh, int ldwh, int flags, hipStream_t s) {
  if (!gemm_f16acc_supports(a, flags) || ldwh < a.K || ldwh % 8) return hipErrorInvalidValue;
  switch (flags) {
    case 0: return launch_f16acc<0>(a, Wh, ldwh, s);
    case kBias: return launch_f16acc<kBias>(a, Wh, ldwh, s);
    case kResid: return launch_f16acc<kResid>(a, Wh, ldwh, s);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_split_weights_f16(const float* W, int N, int K, int ldw, uint16_t* out, hipStream_t s,
                                    bool flat) {
  if (N <= 0 || K <= 0 || ldw < K) return hipErrorInvalidValue;
  const int64_t n_all = (int64_t)N * ldw;
  const int grid = (int)std::min<int64_t>((n_all + 255) / 256, 4096);
  hipLaunchKernelGGL(split_weights_f16_kernel, dim3(grid), dim3(256), 0, s, W, N, K, ldw, out, (int)flat);
  return hipGetLastError();
}

}  // namespace tcl
