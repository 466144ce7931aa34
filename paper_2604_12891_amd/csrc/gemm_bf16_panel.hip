// Row-panel bf16 GEMM for short K (K <= 256): C[M, N] = A W^T, fp32
// accumulation on v_mfma_f32_32x32x16_bf16.
//
// The tiled kernel re-reads every A row once per column tile (8 times for a
// 1024-wide output) and, with an fp32 A, converts and normalises it again
// each time; at ~1M rows those L2 re-reads, not the MFMAs or HBM, set its
// speed. Here a workgroup owns a panel of 256 rows and all N columns:
//
//  * prologue: each of the 4 wavefronts loads its 64 rows of A once
//    (coalesced, through a small LDS stage), applies the RMSNorm gain and
//    sum of squares when asked, rounds to bf16 and keeps the rows as MFMA
//    A-fragments in registers (2 row blocks x K/16 k-steps x 8 bf16);
//  * main loop: 32 columns of W at a time go through a double-buffered LDS
//    stage shared by the 4 wavefronts (one barrier per step; the next
//    step's W is loaded into registers while the MFMAs run); the W
//    fragments are read from LDS two k-steps ahead of their MFMAs;
//  * epilogue per group of steps: the accumulators go through a
//    per-wavefront LDS stage and are stored (and residuals loaded) along
//    rows as 16-byte segments. An fp32 C is staged as fp32 and gets its row
//    scale, bias and residual on the way out; a bf16 C is scaled and
//    rounded in the accumulator layout and staged as bf16, which halves the
//    stage so that three 128-row workgroups fit in a CU's LDS.
//
// A is read from memory exactly once and W once per panel. K-order of
// the fragments: k-step s covers k = 16s .. 16s+15, lane half g supplying
// 16s + 8g .. +7, for A and W alike.
#include "common.h"
#include "kernels.h"

namespace tcl {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int kWaves = 4;

__device__ __forceinline__ uint32_t pack2(float a, float b) { return f32x2_to_bf16x2(a, b); }

// LDS traffic of one wavefront is ordered by the hardware; this keeps the
// compiler from moving a lane's LDS reads above another lane's writes.
__device__ __forceinline__ void wave_lds_order() { __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront"); }

constexpr int cmax(int a, int b) { return a > b ? a : b; }

// Raw buffer resources: accesses at offsets >= num_records read zero and
// drop stores, so bounds become data (an out-of-range offset) instead of
// branches, and the compiler can count outstanding memory operations exactly.
constexpr uint32_t kBufferFlags = 0x00020000;  // 32-bit data format, raw (stride 0)
constexpr uint32_t kOutOfRange = 0x80000000u;  // beyond every resource used here
constexpr int kStoreNT = 2;  // cache-policy bits of a buffer store: non-temporal

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, bytes, kBufferFlags);
}

// MB 32-row MFMA blocks per wavefront: its rows of A stay in registers
// (MB * K / 2 VGPRs), so MB = 2 runs two wavefronts per SIMD, MB = 1 three
template <typename TA, typename TC, int KC, int MB, int FL>
__global__ __launch_bounds__(kWaves * 64, MB == 1 ? 3 : 2) void gemm_bf16_panel_kernel(GemmArgsBF16 p) {
  constexpr int RW = MB * 32;           // rows per wavefront
  constexpr int BM = kWaves * RW;       // rows per workgroup
  constexpr int NS = KC * 4;            // MFMA k-steps
  constexpr int WP = KC * 64 + 8;       // bf16 pitch of a staged W row
  constexpr int WU = KC * 8;            // 16-byte units per staged W row
  constexpr int NW = 32 * WU / (kWaves * 64);  // W units per thread per step
  static_assert(NW * kWaves * 64 == 32 * WU, "W stage must divide evenly");
  constexpr bool kF32A = sizeof(TA) == 4;
  constexpr bool kNorm = (FL & kRowNorm) != 0;
  constexpr bool kF32C = sizeof(TC) == 4;
  static_assert(!kNorm || kF32A, "RMSNorm prologue needs the fp32 residual stream");
  constexpr int PK = kF32A ? 32 : 64;   // k per prologue piece (128 bytes of an A row)
  constexpr int KPIECES = KC * 64 / PK;
  // bf16 rows of one 32-column step are 64 bytes, half a 128-byte line; with
  // one row block per wavefront (registers to spare) two steps are stored
  // together, as whole lines
  constexpr int SPS = (!kF32C && MB == 1) ? 2 : 1;  // steps per store
  constexpr int CW = 32 * SPS;          // columns per store
  // the output stage holds fp32 values for an fp32 C and the finished bf16
  // values for a bf16 C (half the LDS: three workgroups then fit on a CU)
  constexpr int CP = kF32C ? CW + 4 : CW + 8;  // pitch in elements (conflict-free both ways)
  constexpr int APITCH = PK + 8;        // bf16 pitch of the A stage (80 or 144 B: conflict-free fragment reads)
  constexpr int kStageA = 32 * APITCH * 2;
  constexpr int kStageC = RW * CP * (kF32C ? 4 : 2);
  constexpr bool kGath = (FL & kGather) != 0;

  __shared__ __attribute__((aligned(16))) uint16_t sW[2][32 * WP];
  __shared__ __attribute__((aligned(16))) unsigned char sX[kWaves][cmax(kStageA, kStageC)];
  __shared__ __attribute__((aligned(16))) float sR[kWaves][RW];
  __shared__ int sSrc[kGath ? BM : 1];
  __shared__ __attribute__((aligned(16))) float sG[kNorm ? KC * 64 : 4];

  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63;
  const int li = lane & 31, lg = lane >> 5;
  const int M = p.Mdev ? *p.Mdev : p.Mmax;
  const int row0 = blockIdx.x * BM;
  if (row0 >= M) return;
  const int Kw = (p.K + 7) & ~7;  // W is zero-padded to here

  // source row of each panel row: the packed-token gather, else the row
  // itself (-1 past M)
  if constexpr (kGath) {
    for (int r = tid; r < BM; r += kWaves * 64) {
      const int grow = row0 + r;
      int src = -1;
      if (grow < M) {
        int lo = 0, hi = p.B;
        while (hi - lo > 1) {
          const int mid = (lo + hi) >> 1;
          if (p.offs[mid] <= grow) lo = mid; else hi = mid;
        }
        src = lo * p.L + (grow - p.offs[lo]);
      }
      sSrc[r] = src;
    }
  }
  if constexpr (kNorm) {
    for (int k = tid; k < KC * 64; k += kWaves * 64) sG[k] = k < p.K ? p.gain[k] : 0.f;
  }

  // W stage loads: unit i of this thread is row n = u / WU, k = 8 (u % WU);
  // rows n >= N and units past Kw read zero through the resource (an
  // out-of-range offset), so staging is a plain copy of the loaded units
  const __amdgpu_buffer_rsrc_t wres = make_rsrc(p.W, (uint32_t)(p.N * p.ldw * 2));
  u32x4 rw[NW];
  const int nsteps = (p.N + 31) / 32;
  auto gload_w = [&](int n0) {
#pragma unroll
    for (int i = 0; i < NW; ++i) {
      const int u = tid + i * kWaves * 64;
      const int n = n0 + u / WU, k = 8 * (u % WU);
      rw[i] = __builtin_amdgcn_raw_buffer_load_b128(wres, k < Kw ? (uint32_t)((n * p.ldw + k) * 2) : kOutOfRange,
                                                    0, 0);
    }
  };
  auto stage_w = [&](int buf) {
#pragma unroll
    for (int i = 0; i < NW; ++i) {
      const int u = tid + i * kWaves * 64;
      *reinterpret_cast<u32x4*>(&sW[buf][(u / WU) * WP + 8 * (u % WU)]) = rw[i];
    }
  };
  gload_w(0);  // in flight during the prologue
  __syncthreads();  // sSrc, sG

  // ---- prologue: this wavefront's 64 rows of A -> bf16 fragments, in pieces
  // of 32 rows x PK k (4 KB: PK = 32 fp32 or 64 bf16), software-pipelined:
  // the next piece's global loads are issued before the current one is
  // converted, staged and read back as fragments. Unit j of this lane is row
  // (lane + 64 j) / 8 of the block and 16-byte unit lane % 8 of the piece.
  bf16x8 af[MB][NS];
  uint16_t* stA = reinterpret_cast<uint16_t*>(sX[wave]);
  const int au = lane % 8;
  int srcs[MB][4];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int r = wave * RW + mb * 32 + (lane + 64 * j) / 8;
      srcs[mb][j] = kGath ? sSrc[r] : (row0 + r < M ? row0 + r : -1);
    }
  u32x4 va[4], vn[4];  // raw 16-byte units (fp32 x4 or bf16 x8)
  auto gload_a = [&](int piece, u32x4* v) {
    const int mb = piece / KPIECES;
    const int k = (piece % KPIECES) * PK + au * (16 / (int)sizeof(TA));
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int src = srcs[mb][j];
      // clamped in-bounds address; out-of-range units are zeroed when staged
      v[j] = *reinterpret_cast<const u32x4*>(reinterpret_cast<const TA*>(p.A) +
                                             (src >= 0 && k < p.K ? (int64_t)src * p.lda + k : 0));
    }
  };
  float ss[MB][4];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int j = 0; j < 4; ++j) ss[mb][j] = 0.f;
  gload_a(0, va);
#pragma unroll
  for (int piece = 0; piece < MB * KPIECES; ++piece) {
    const int mb = piece / KPIECES, k0 = (piece % KPIECES) * PK;
    const bool kin = k0 + au * (16 / (int)sizeof(TA)) < p.K;
    if (piece + 1 < MB * KPIECES) gload_a(piece + 1, vn);
    // keep the scheduler from hoisting every piece's loads to the top
    // (that would hold the whole panel of A in registers at once)
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int r = (lane + 64 * j) / 8;
      const u32x4 x = (kin && srcs[mb][j] >= 0) ? va[j] : u32x4{0u, 0u, 0u, 0u};
      if constexpr (kF32A) {
        floatx4 v = __builtin_bit_cast(floatx4, x);
        if constexpr (kNorm) {
          const int k = k0 + 4 * au;
          const floatx4 g = *reinterpret_cast<const floatx4*>(&sG[k]);
          ss[mb][j] += v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
          // materialise the running sum here: otherwise the compiler sinks
          // these FMAs to the final reduction and keeps every piece of A live
          asm volatile("" : "+v"(ss[mb][j]));
          v *= g;
        }
        *reinterpret_cast<u32x2*>(&stA[r * APITCH + 4 * au]) = u32x2{pack2(v.x, v.y), pack2(v.z, v.w)};
      } else {
        *reinterpret_cast<u32x4*>(&stA[r * APITCH + 8 * au]) = x;
      }
    }
    wave_lds_order();
#pragma unroll
    for (int c = 0; c < PK / 16; ++c)
      af[mb][k0 / 16 + c] =
          __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(&stA[li * APITCH + 16 * c + 8 * lg]));
    wave_lds_order();
#pragma unroll
    for (int j = 0; j < 4; ++j) va[j] = vn[j];
  }
  if constexpr (kNorm) {
    // the 8 lanes of a row hold its partial sums: reduce, then 1/rms
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        float v = ss[mb][j];
#pragma unroll
        for (int o = 1; o < 8; o <<= 1) v += __shfl_xor(v, o, 64);
        if (au == 0) sR[wave][mb * 32 + (lane + 64 * j) / 8] = 1.0f / sqrtf(v / (float)p.K + p.eps);
      }
  }

  // ---- main loop over 32-column steps
  float* stC = reinterpret_cast<float*>(sX[wave]);
  uint16_t* stB = reinterpret_cast<uint16_t*>(sX[wave]);
  // this panel's rows of C (and of the residual source R, same pitch)
  const uint32_t panel_bytes = (uint32_t)(min(BM, M - row0) * p.ldc * (int)sizeof(TC));
  const __amdgpu_buffer_rsrc_t cres =
      make_rsrc(reinterpret_cast<const TC*>(p.C) + (int64_t)row0 * p.ldc, panel_bytes);
  const __amdgpu_buffer_rsrc_t rres = make_rsrc(
      (p.R ? p.R : reinterpret_cast<const float*>(p.C)) + ((FL & kResid) != 0 ? (int64_t)row0 * p.ldc : 0),
      (FL & kResid) != 0 ? panel_bytes : 0);
  // Steps run in groups of SPS with one epilogue per group, and the next
  // step's W is loaded on every step but the very last: every path from a
  // W load to its staging then holds the same memory operations, so the
  // compiler's wait for it is exact. (With a conditional epilogue the
  // counts of the two paths merge to the smaller one, and a wavefront would
  // wait for its own just-issued C stores before staging W.) When nsteps is
  // odd the last group's extra step stages rows >= N, which read as zero.
  const int ngroups = (nsteps + SPS - 1) / SPS;
  for (int grp = 0; grp < ngroups; ++grp) {
    floatx16 acc[SPS][MB];
#pragma unroll
    for (int h = 0; h < SPS; ++h) {
      const int s = grp * SPS + h, buf = s & 1;
      stage_w(buf);
      __syncthreads();  // W step s visible; every wavefront is past step s-1's reads of this buffer's pair
      if (s + 1 < ngroups * SPS) gload_w((s + 1) * 32);

#pragma unroll
      for (int mb = 0; mb < MB; ++mb)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[h][mb][r] = 0.f;
      // W fragments in a ring of 4, read three k-steps ahead so that LDS
      // latency overlaps the MFMAs in between; the scheduling groups pin the
      // order (three reads, then per k-step: its MB MFMAs, one read)
      auto wfrag = [&](int ks) {
        return __builtin_bit_cast(bf16x8,
                                  *reinterpret_cast<const u32x4*>(&sW[buf][li * WP + 16 * ks + 8 * lg]));
      };
      constexpr int AHEAD = NS < 3 ? NS : 3;
      bf16x8 bq[4];
#pragma unroll
      for (int ks = 0; ks < AHEAD; ++ks) bq[ks] = wfrag(ks);
      __builtin_amdgcn_sched_group_barrier(0x0100, AHEAD, 0);
#pragma unroll
      for (int ks = 0; ks < NS; ++ks) {
#pragma unroll
        for (int mb = 0; mb < MB; ++mb)
          acc[h][mb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[mb][ks], bq[ks & 3], acc[h][mb], 0, 0, 0);
        __builtin_amdgcn_sched_group_barrier(0x0008, MB, 0);
        if (ks + AHEAD < NS) {
          bq[(ks + AHEAD) & 3] = wfrag(ks + AHEAD);
          __builtin_amdgcn_sched_group_barrier(0x0100, 1, 0);
        }
      }
    }

    // epilogue of the group: accumulator layout (lane l: column l % 32,
    // rows 8*(r/4) + 4*(l/32) + (r%4)) -> row-major stage -> each lane
    // finishes 8 consecutive columns of its rows with 16-byte stores. fp32
    // C: staged as fp32, then row scale, bias, residual; bf16 C (no bias,
    // no residual): row scale and rounding in the accumulator layout,
    // staged as bf16
    if constexpr (kF32C) {
#pragma unroll
      for (int h = 0; h < SPS; ++h)
#pragma unroll
        for (int mb = 0; mb < MB; ++mb)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int row = mb * 32 + 8 * (r >> 2) + 4 * lg + (r & 3);
            stC[row * CP + 32 * h + li] = acc[h][mb][r];
          }
    } else {
      static_assert(kF32C || (FL & (kBias | kResid)) == 0, "bf16 C takes neither bias nor residual");
#pragma unroll
      for (int mb = 0; mb < MB; ++mb)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int row = mb * 32 + 8 * q + 4 * lg;  // rows row .. row + 3 of this lane
          floatx4 sc = floatx4{1.f, 1.f, 1.f, 1.f};
          if constexpr (kNorm) sc = *reinterpret_cast<const floatx4*>(&sR[wave][row]);
#pragma unroll
          for (int h = 0; h < SPS; ++h)
#pragma unroll
            for (int i = 0; i < 4; i += 2) {
              const uint32_t w = pack2(acc[h][mb][4 * q + i] * sc[i], acc[h][mb][4 * q + i + 1] * sc[i + 1]);
              stB[(row + i) * CP + 32 * h + li] = (uint16_t)(w & 0xFFFFu);
              stB[(row + i + 1) * CP + 32 * h + li] = (uint16_t)(w >> 16);
            }
        }
    }
    wave_lds_order();
    constexpr int LPR = CW / 8;          // lanes per row
    constexpr int RPI = 64 / LPR;        // rows per store instruction
    const int u = lane % LPR;  // 8-column unit of this lane (the same for all its rows)
    const int c0 = grp * CW + 8 * u;
    const bool ok0 = c0 < p.N, ok1 = c0 + 4 < p.N;  // N % 4 == 0: halves are all in or all out
    floatx4 b0 = floatx4{0.f, 0.f, 0.f, 0.f}, b1 = b0;
    if constexpr ((FL & kBias) != 0) {
      const floatx4 x0 = *reinterpret_cast<const floatx4*>(p.bias + (ok0 ? c0 : 0));
      const floatx4 x1 = *reinterpret_cast<const floatx4*>(p.bias + (ok1 ? c0 + 4 : 0));
      if (ok0) b0 = x0;
      if (ok1) b1 = x1;
    }
#pragma unroll
    for (int i = 0; i < RW / RPI; ++i) {
      const int rl = lane / LPR + RPI * i;
      const int prow = wave * RW + rl;  // row within the panel; rows past M fall outside cres
      const uint32_t off = (uint32_t)(prow * p.ldc + c0) * (uint32_t)sizeof(TC);
      if constexpr (!kF32C) {
        // N % 8 == 0 for bf16 C: a unit is all in or all out; stored
        // non-temporal (a streamed output, re-read only by the next kernel)
        const u32x4 w = *reinterpret_cast<const u32x4*>(&stB[rl * CP + 8 * u]);
        __builtin_amdgcn_raw_buffer_store_b128(w, cres, ok0 ? off : kOutOfRange, 0, kStoreNT);
        continue;
      }
      floatx4 v0 = *reinterpret_cast<const floatx4*>(&stC[rl * CP + 8 * u]);
      floatx4 v1 = *reinterpret_cast<const floatx4*>(&stC[rl * CP + 8 * u + 4]);
      if constexpr (kNorm) {
        const float sc = sR[wave][rl];
        v0 *= sc;
        v1 *= sc;
      }
      v0 += b0;
      v1 += b1;
      {
        const uint32_t o0 = ok0 ? off : kOutOfRange, o1 = ok1 ? off + 16 : kOutOfRange;
        if constexpr ((FL & kResid) != 0) {
          v0 += __builtin_bit_cast(floatx4, __builtin_amdgcn_raw_buffer_load_b128(rres, o0, 0, 0));
          v1 += __builtin_bit_cast(floatx4, __builtin_amdgcn_raw_buffer_load_b128(rres, o1, 0, 0));
        }
        __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, v0), cres, o0, 0, 0);
        __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, v1), cres, o1, 0, 0);
      }
    }
    wave_lds_order();
  }
}

template <typename TA, typename TC, int MB, int FL>
hipError_t launch_kc(const GemmArgsBF16& a, hipStream_t s) {
  constexpr int BM = kWaves * MB * 32;
  const int grid = (a.Mmax + BM - 1) / BM;
  if (grid <= 0) return hipSuccess;
  const int kc = (a.K + 63) / 64;
  switch (kc) {
    case 1: hipLaunchKernelGGL((gemm_bf16_panel_kernel<TA, TC, 1, MB, FL>), dim3(grid), dim3(kWaves * 64), 0, s, a); break;
    case 2: hipLaunchKernelGGL((gemm_bf16_panel_kernel<TA, TC, 2, MB, FL>), dim3(grid), dim3(kWaves * 64), 0, s, a); break;
    case 3: hipLaunchKernelGGL((gemm_bf16_panel_kernel<TA, TC, 3, MB, FL>), dim3(grid), dim3(kWaves * 64), 0, s, a); break;
    case 4: hipLaunchKernelGGL((gemm_bf16_panel_kernel<TA, TC, 4, MB, FL>), dim3(grid), dim3(kWaves * 64), 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <typename TA, typename TC, int FL>
hipError_t launch_mb(const GemmArgsBF16& a, int rows_per_wave, hipStream_t s) {
  return rows_per_wave == 32 ? launch_kc<TA, TC, 1, FL>(a, s) : launch_kc<TA, TC, 2, FL>(a, s);
}

}  // namespace

bool gemm_bf16_panel_fits(const GemmArgsBF16& a, bool bf16_out) {
  // 16-byte row segments of C need a 16-byte-aligned row pitch
  const int64_t pitch_bytes = a.ldc * (bf16_out ? 2 : 4);
  auto al16 = [](const void* q) { return reinterpret_cast<uintptr_t>(q) % 16 == 0; };
  return a.K >= 1 && a.K <= 256 && pitch_bytes % 16 == 0 && al16(a.C) && (a.R == nullptr || al16(a.R)) &&
         (a.bias == nullptr || al16(a.bias)) && (!bf16_out || a.N % 8 == 0) &&
         // byte offsets of the buffer resources stay below 2^31
         (int64_t)kWaves * 64 * pitch_bytes < (1ll << 31) && (int64_t)(a.N + 64) * a.ldw * 2 < (1ll << 31);
}

hipError_t launch_gemm_bf16_panel(const GemmArgsBF16& a, GemmBF16Kind kind, int rows_per_wave, hipStream_t s) {
  if (rows_per_wave != 32 && rows_per_wave != 64) return hipErrorInvalidValue;
  switch (kind) {
    case kInputF32toF32: return launch_mb<float, float, kBias | kGather>(a, rows_per_wave, s);
    case kNormF32toBF16: return launch_mb<float, uint16_t, kRowNorm>(a, rows_per_wave, s);
    case kBF16ResidF32: return launch_mb<uint16_t, float, kResid>(a, rows_per_wave, s);
    case kBF16toF32: return launch_mb<uint16_t, float, 0>(a, rows_per_wave, s);
    case kBF16toF32Bias: return launch_mb<uint16_t, float, kBias>(a, rows_per_wave, s);
    case kBF16toBF16: return launch_mb<uint16_t, uint16_t, 0>(a, rows_per_wave, s);
    case kF32toF32:
    case kF32ResidF32: return hipErrorInvalidValue;  // tiles only
  }
  return hipErrorInvalidValue;
}

}  // namespace tcl
