// Progressive KB + AC forward of the CKD framework (section 6, Fig. 6,
// Eq. (7)): the frozen knowledge base (KB) and the active column (AC) run
// layer by layer on the same packed tokens, and every AC layer after the
// first adds alpha_i * U_i ReLU(V_i h^KB_{i-1} + c_i) of the KB's input to
// the same layer before its own activation.
//
// Per layer: the AC's own layer, then the adapter on the KB's input to the
// layer accumulated into the AC's output (alpha folded into U's rows at
// create; ReLU after the sum for hidden Linear layers; one fused pass per
// row for narrow adapters, two GEMMs otherwise), then the KB's own layer. The encoder and Mamba
// blocks run on packed token rows; both columns are pooled and the decoder
// Linear layers run as GEMMs over the B pooled rows. The KB's last layer is
// not computed: no AC layer reads its output.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstring>

#include "common.h"
#include "model.h"

using namespace tcl;

struct tcl_lateral {
  tcl_model* kb = nullptr;
  tcl_model* ac = nullptr;
  int a = 0;
  size_t n_params = 0;
  void* dev = nullptr;
  struct Lat {
    int n_in = 0, n_out = 0;
    float *V = nullptr, *c = nullptr, *U = nullptr;  // U with alpha folded into its rows
  };
  std::vector<Lat> lats;
};

namespace {

// (n_in, n_out) of every layer in forward order: encoder Linear layers,
// Mamba blocks, decoder Linear layers.
std::vector<std::pair<int, int>> layer_widths(const tcl_config& c) {
  const BlobLayout bl = blob_layout(c);
  std::vector<std::pair<int, int>> w;
  for (int i = 0; i < bl.n_enc; ++i) w.push_back({bl.enc_dims[i], bl.enc_dims[i + 1]});
  for (int l = 0; l < c.n_layers; ++l) w.push_back({c.d_model, c.d_model});
  w.push_back({c.d_model, c.head_hidden});
  if (c.dec_hidden2 > 0) {
    w.push_back({c.head_hidden, c.dec_hidden2});
    w.push_back({c.dec_hidden2, 1});
  } else {
    w.push_back({c.head_hidden, 1});
  }
  return w;
}

size_t lateral_count(const tcl_config& c, int a) {
  const auto w = layer_widths(c);
  size_t n = 0;
  for (size_t j = 1; j < w.size(); ++j) n += (size_t)a * w[j].first + a + (size_t)w[j].second * a + w[j].second;
  return n;
}

bool same_architecture(const tcl_config& x, const tcl_config& y) {
  return x.F == y.F && x.d_model == y.d_model && x.d_inner == y.d_inner && x.d_state == y.d_state &&
         x.d_conv == y.d_conv && x.dt_rank == y.dt_rank && x.n_layers == y.n_layers &&
         x.head_hidden == y.head_hidden && x.final_norm == y.final_norm && x.norm_eps == y.norm_eps &&
         x.dtype == y.dtype && x.enc_hidden[0] == y.enc_hidden[0] && x.enc_hidden[1] == y.enc_hidden[1] &&
         x.dec_hidden2 == y.dec_hidden2;
}

struct ProgPlan {
  size_t offs, tpos, feats, Hkb, Hac, xz, u, xdbl, T, ekb[2], eac[2], Pkb, Pac, rkb[2], rac[2], scr, total;
};

ProgPlan prog_plan(const tcl_config& c, int a, int64_t B, int64_t L) {
  ProgPlan p{};
  const int64_t rows = B * L;
  const int XW = c.dt_rank + 2 * c.d_state;
  const int dec_w = std::max(c.head_hidden, c.dec_hidden2);
  size_t o = 0;
  auto take = [&](size_t bytes) {
    const size_t at = o;
    o = align256(o + bytes);
    return at;
  };
  p.offs = take((size_t)(B + 1) * 4);
  p.tpos = take((size_t)rows);
  p.feats = take(c.F % 4 ? (size_t)rows * ((c.F + 3) & ~3) * 4 : 0);
  p.Hkb = take((size_t)rows * c.d_model * 4);
  p.Hac = take((size_t)rows * c.d_model * 4);
  p.xz = take((size_t)rows * 2 * c.d_inner * 4);
  p.u = take((size_t)rows * c.d_inner * 4);
  p.xdbl = take((size_t)rows * XW * 4);
  p.T = take((size_t)rows * a * 4);
  for (int i = 0; i < 2; ++i) {
    p.ekb[i] = take((size_t)rows * std::max(c.enc_hidden[i], 0) * 4);
    p.eac[i] = take((size_t)rows * std::max(c.enc_hidden[i], 0) * 4);
    p.rkb[i] = take((size_t)B * dec_w * 4);
    p.rac[i] = take((size_t)B * dec_w * 4);
  }
  p.Pkb = take((size_t)B * c.d_model * 4);
  p.Pac = take((size_t)B * c.d_model * 4);
  p.scr = take((size_t)B * 4);
  p.total = o;
  return p;
}

// A plain fp32 GEMM C = act(A W^T + bias (+ C)) over `rows` rows (device
// count *Mdev when given).
GemmArgs plain(const float* A, int lda, const float* W, const float* bias, float* C, int ldc, int N, int K,
               const int* Mdev, int Mmax, bool relu) {
  GemmArgs g;
  g.A = A; g.lda = lda; g.W = W; g.ldw = K; g.bias = bias; g.C = C; g.ldc = ldc;
  g.Mdev = Mdev; g.Mmax = Mmax; g.N = N; g.K = K; g.relu = relu;
  return g;
}

// A narrow adapter in one pass over the rows: one wavefront per row (two
// rows in flight), lane l holding inputs l + 64p and outputs l + 64p; V, c
// and U' stay in registers. Per row the A inner sums are reduce-scattered
// across the wavefront (lane bit 5 by a half-wave swap, bit 4 by a row swap,
// then DPP / swizzle steps; each step halves the values a lane carries until
// one is left, then plain pair sums), so lane l ends with the total of sum
// k = l >> (6 - log2 A); the A totals are then read back as wave-uniform
// values. Every output is C + sum_k U'[j][k] ReLU(t_k + c_k), ReLU'd when
// `act`. Nothing of size [rows, A] is stored.
template <int N>
__device__ __forceinline__ void swap32(float* w) {
  // bit 5: lanes 0-31 keep w[i], lanes 32-63 keep w[N/2 + i], each summed over the lane pair
#pragma unroll
  for (int i = 0; i < N / 2; ++i) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(w[i]), __float_as_uint(w[N / 2 + i]), false, false);
    w[i] = __uint_as_float(r[0]) + __uint_as_float(r[1]);
  }
}
template <int N>
__device__ __forceinline__ void swap16(float* w) {
  // bit 4: rows 0, 2 keep w[i], rows 1, 3 keep w[N/2 + i]
#pragma unroll
  for (int i = 0; i < N / 2; ++i) {
    const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(w[i]), __float_as_uint(w[N / 2 + i]), false, false);
    w[i] = __uint_as_float(r[0]) + __uint_as_float(r[1]);
  }
}
__device__ __forceinline__ float ror8(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x128, 0xF, 0xF, false));  // xor 8 in a row
}
__device__ __forceinline__ float xor4(float v) { return __int_as_float(__builtin_amdgcn_ds_swizzle(__float_as_int(v), 0x101F)); }
__device__ __forceinline__ float xor2(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x4E, 0xF, 0xF, false));
}
__device__ __forceinline__ float xor1(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0xB1, 0xF, 0xF, false));
}

// A in {4, 8, 16}: returns lane l's total of value l >> (6 - log2 A).
template <int A>
__device__ __forceinline__ float reduce_scatter(float* w, int lane) {
  swap32<A>(w);
  swap16<A / 2>(w);
  float z;
  if constexpr (A == 4) {
    z = w[0] + ror8(w[0]);
    z += xor4(z);
  } else {
    const bool b3 = (lane & 8) != 0;
    float y[A / 8];
#pragma unroll
    for (int i = 0; i < A / 8; ++i) {
      const float mine = b3 ? w[A / 8 + i] : w[i], other = b3 ? w[i] : w[A / 8 + i];
      y[i] = mine + ror8(other);
    }
    if constexpr (A == 8) {
      z = y[0] + xor4(y[0]);
    } else {
      const bool b2 = (lane & 4) != 0;
      const float mine = b2 ? y[1] : y[0], other = b2 ? y[0] : y[1];
      z = mine + xor4(other);
    }
  }
  z += xor2(z);
  return z + xor1(z);
}

template <int PI, int PO, int A>
__global__ __launch_bounds__(256) void adapter_kernel(int Mmax, const int* __restrict__ Mdev,
                                                      const float* __restrict__ X, int n_in,
                                                      const float* __restrict__ V, const float* __restrict__ cb,
                                                      const float* __restrict__ U, int n_out, float* __restrict__ C,
                                                      int ldc, int act) {
  constexpr int LA = A == 4 ? 2 : A == 8 ? 3 : 4;
  const int M = Mdev ? *Mdev : Mmax;
  const int lane = threadIdx.x & 63;
  const int wave = blockIdx.x * 4 + (threadIdx.x >> 6), nwaves = gridDim.x * 4;
  float v[A][PI], u[PO][A], c[A];
#pragma unroll
  for (int k = 0; k < A; ++k) {
    c[k] = cb[k];
#pragma unroll
    for (int p = 0; p < PI; ++p) {
      const int i = lane + 64 * p;
      v[k][p] = i < n_in ? V[k * n_in + i] : 0.f;
    }
  }
#pragma unroll
  for (int p = 0; p < PO; ++p) {
    const int j = lane + 64 * p;
#pragma unroll
    for (int k = 0; k < A; ++k) u[p][k] = j < n_out ? U[j * A + k] : 0.f;
  }
  for (int r0 = 2 * wave; r0 < M; r0 += 2 * nwaves) {
    // two rows; past the end the second repeats the first and is not stored
    const int rows[2] = {r0, min(r0 + 1, M - 1)};
    float x[2][PI], y[2][PO];
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const float* xr = X + (int64_t)rows[q] * n_in;
      const float* cr = C + (int64_t)rows[q] * ldc;
#pragma unroll
      for (int p = 0; p < PI; ++p) x[q][p] = xr[min(lane + 64 * p, n_in - 1)];  // V is zero past n_in
#pragma unroll
      for (int p = 0; p < PO; ++p) y[q][p] = cr[min(lane + 64 * p, n_out - 1)];
    }
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      float w[A];
#pragma unroll
      for (int k = 0; k < A; ++k) {
        float acc = 0.f;
#pragma unroll
        for (int p = 0; p < PI; ++p) acc = fmaf(v[k][p], x[q][p], acc);
        w[k] = acc;
      }
      const float z = reduce_scatter<A>(w, lane);
      float t[A];
#pragma unroll
      for (int k = 0; k < A; ++k)
        t[k] = fmaxf(__int_as_float(__builtin_amdgcn_readlane(__float_as_int(z), k << (6 - LA))) + c[k], 0.f);
      if (q == 1 && r0 + 1 >= M) break;
      float* cr = C + (int64_t)rows[q] * ldc;
#pragma unroll
      for (int p = 0; p < PO; ++p) {
        const int j = lane + 64 * p;
        float o = y[q][p];
#pragma unroll
        for (int k = 0; k < A; ++k) o = fmaf(u[p][k], t[k], o);
        if (act) o = fmaxf(o, 0.f);
        if (j < n_out) cr[j] = o;
      }
    }
  }
}

int lanes_per(int n) { return n <= 64 ? 1 : n <= 128 ? 2 : n <= 256 ? 4 : 0; }

// The fused adapter kernel for n_in, n_out <= 256 and a in {4, 8, 16};
// hipErrorNotSupported otherwise (the caller then uses two GEMMs).
hipError_t launch_adapter(int Mmax, const int* Mdev, const float* X, int n_in, const float* V, const float* c,
                          const float* U, int n_out, int a, float* C, int ldc, bool act, hipStream_t s) {
  const int pi = lanes_per(n_in), po = lanes_per(n_out);
  if (!pi || !po || (a != 4 && a != 8 && a != 16)) return hipErrorNotSupported;
  if (Mmax <= 0) return hipSuccess;
  const int grid = std::min((Mmax + 3) / 4, 4096);
#define TCL_ADP(PI_, PO_, A_)                                                                                \
  hipLaunchKernelGGL((adapter_kernel<PI_, PO_, A_>), dim3(grid), dim3(256), 0, s, Mmax, Mdev, X, n_in, V, c, U, \
                     n_out, C, ldc, act ? 1 : 0)
#define TCL_ADP_A(PI_, PO_)               \
  switch (a) {                            \
    case 4: TCL_ADP(PI_, PO_, 4); break;  \
    case 8: TCL_ADP(PI_, PO_, 8); break;  \
    default: TCL_ADP(PI_, PO_, 16); break; \
  }
  switch (pi * 10 + po) {
    case 11: TCL_ADP_A(1, 1); break;
    case 12: TCL_ADP_A(1, 2); break;
    case 14: TCL_ADP_A(1, 4); break;
    case 21: TCL_ADP_A(2, 1); break;
    case 22: TCL_ADP_A(2, 2); break;
    case 24: TCL_ADP_A(2, 4); break;
    case 41: TCL_ADP_A(4, 1); break;
    case 42: TCL_ADP_A(4, 2); break;
    default: TCL_ADP_A(4, 4); break;
  }
#undef TCL_ADP_A
#undef TCL_ADP
  return hipGetLastError();
}

// Adapter j: C = act(C + U' ReLU(X_kb V^T + c)) -- one fused pass for narrow
// adapters, else T = ReLU(X_kb V^T + c) by one GEMM and the accumulation by
// a second (residual epilogue).
tcl_status lateral(tcl_lateral* lt, Timing& T, int j, const float* X_kb, float* Tbuf, float* C, int ldc,
                   const int* Mdev, int Mmax, bool act, hipStream_t s) {
  const auto& A = lt->lats[j];
  if (lanes_per(A.n_in) && lanes_per(A.n_out) && (lt->a == 4 || lt->a == 8 || lt->a == 16)) {
    TCL_LAUNCH(T, "lat:adapter", launch_adapter(Mmax, Mdev, X_kb, A.n_in, A.V, A.c, A.U, A.n_out, lt->a, C, ldc,
                                                act, s));
    return TCL_OK;
  }
  const GemmArgs gv = plain(X_kb, A.n_in, A.V, A.c, Tbuf, lt->a, lt->a, A.n_in, Mdev, Mmax, true);
  TCL_LAUNCH(T, "lat:gemm_V", launch_gemm_f32(gv, kBias, -1, s));
  const GemmArgs gu = plain(Tbuf, lt->a, A.U, nullptr, C, ldc, A.n_out, lt->a, Mdev, Mmax, act);
  TCL_LAUNCH(T, "lat:gemm_U", launch_gemm_f32(gu, kResid, -1, s));
  return TCL_OK;
}

#define TCL_TRY(x)                   \
  do {                               \
    tcl_status st_ = (x);            \
    if (st_ != TCL_OK) return st_;   \
  } while (0)

tcl_status run_progressive(tcl_lateral* lt, int B, int L, const float* d_feats, const int* d_lengths,
                           float* d_scores, char* ws, hipStream_t s) {
  tcl_model* kb = lt->kb;
  tcl_model* ac = lt->ac;
  const tcl_config& c = kb->cfg;
  const ProgPlan p = prog_plan(c, lt->a, B, L);
  auto F32 = [&](size_t off) { return reinterpret_cast<float*>(ws + off); };
  int* offs = reinterpret_cast<int*>(ws + p.offs);
  Timing& T = ac->timing;
  const int Mmax = B * L;
  const int* Mdev = offs + B;
  const BlobLayout bl = blob_layout(c);
  const int n_enc = bl.n_enc, d = c.d_model, h = c.head_hidden, h2 = c.dec_hidden2;

  TCL_LAUNCH(T, "offsets", launch_offsets(d_lengths, B, L, offs, s));
  uint8_t* tpos = reinterpret_cast<uint8_t*>(ws + p.tpos);
  const bool fuse = kb->split && ac->split;
  if (fuse) TCL_LAUNCH(T, "token_pos", launch_token_pos(offs, B, tpos, s));
  const float* feats = d_feats;
  const int ldf = (c.F + 3) & ~3;
  if (ldf != c.F) {
    TCL_LAUNCH(T, "pad_features", launch_pad_rows(d_feats, (int64_t)B * L, c.F, ldf, F32(p.feats), s));
    feats = F32(p.feats);
  }
  float* Hkb = F32(p.Hkb);
  float* Hac = F32(p.Hac);
  float* Tb = F32(p.T);
  int j = 0;  // next adapter

  // encoder
  const float* kb_in = feats;
  const float* ac_in = feats;
  for (int i = 0; i < n_enc; ++i) {
    const bool last = i == n_enc - 1;
    float* kb_out = last ? Hkb : F32(p.ekb[i]);
    float* ac_out = last ? Hac : F32(p.eac[i]);
    if (i == 0) {
      TCL_TRY(enqueue_encoder_layer_f32(ac, T, "ac:", i, B, L, offs, ac_in, ac_out, !last, s));
    } else {
      TCL_TRY(enqueue_encoder_layer_f32(ac, T, "ac:", i, B, L, offs, ac_in, ac_out, false, s));
      TCL_TRY(lateral(lt, T, j++, kb_in, Tb, ac_out, bl.enc_dims[i + 1], Mdev, Mmax, !last, s));
    }
    TCL_TRY(enqueue_encoder_layer_f32(kb, T, "kb:", i, B, L, offs, kb_in, kb_out, !last, s));
    kb_in = kb_out;
    ac_in = ac_out;
  }
  // Mamba blocks: the adapter reads the KB's block input before the KB's block runs
  float* xz = F32(p.xz);
  float* u = F32(p.u);
  float* xdbl = F32(p.xdbl);
  for (int l = 0; l < c.n_layers; ++l) {
    TCL_TRY(enqueue_block_f32(ac, T, "ac:", l, B, L, offs, fuse ? tpos : nullptr, Hac, xz, u, xdbl, s));
    TCL_TRY(lateral(lt, T, j++, Hkb, Tb, Hac, d, Mdev, Mmax, false, s));
    TCL_TRY(enqueue_block_f32(kb, T, "kb:", l, B, L, offs, fuse ? tpos : nullptr, Hkb, xz, u, xdbl, s));
  }
  // final norm and pool of both columns (the tail's own head output is not used)
  float* Pkb = F32(p.Pkb);
  float* Pac = F32(p.Pac);
  TCL_LAUNCH(T, "kb:pool", launch_tail_f32(B, L, d, h, offs, d_lengths, Hkb, kb->g_f, c.final_norm, c.norm_eps,
                                           kb->W1T, kb->b1, kb->W2, kb->b2, F32(p.scr), s, Pkb));
  TCL_LAUNCH(T, "ac:pool", launch_tail_f32(B, L, d, h, offs, d_lengths, Hac, ac->g_f, c.final_norm, c.norm_eps,
                                           ac->W1T, ac->b1, ac->W2, ac->b2, F32(p.scr), s, Pac));
  // decoder over the B pooled rows
  struct DL {
    int n_in, n_out;
    const float *Wk, *bk, *Wa, *ba;
  };
  std::vector<DL> dec = {{d, h, kb->W1, kb->b1, ac->W1, ac->b1}};
  if (h2 > 0) {
    dec.push_back({h, h2, kb->W2, kb->b2, ac->W2, ac->b2});
    dec.push_back({h2, 1, kb->W3, kb->b3, ac->W3, ac->b3});
  } else {
    dec.push_back({h, 1, kb->W2, kb->b2, ac->W2, ac->b2});
  }
  const float* xk = Pkb;
  const float* xa = Pac;
  for (size_t k = 0; k < dec.size(); ++k) {
    const bool last = k + 1 == dec.size();
    const DL& D = dec[k];
    float* ya = last ? d_scores : F32(p.rac[k % 2]);
    const int ldo = last ? 1 : D.n_out;
    const GemmArgs ga = plain(xa, D.n_in, D.Wa, D.ba, ya, ldo, D.n_out, D.n_in, nullptr, B, false);
    TCL_LAUNCH(T, "ac:gemm_decoder", launch_gemm_f32(ga, kBias, -1, s));
    TCL_TRY(lateral(lt, T, j++, xk, Tb, ya, ldo, nullptr, B, !last, s));
    if (!last) {
      // the KB's hidden decoder layer (its input feeds the next adapter)
      float* yk = F32(p.rkb[k % 2]);
      const GemmArgs gk = plain(xk, D.n_in, D.Wk, D.bk, yk, D.n_out, D.n_out, D.n_in, nullptr, B, true);
      TCL_LAUNCH(T, "kb:gemm_decoder", launch_gemm_f32(gk, kBias, -1, s));
      xk = yk;
      xa = ya;
    }
  }
  TCL_LAUNCH(T, "mask_scores", launch_mask_scores(B, L, d_lengths, d_scores, s));
  return TCL_OK;
}

}  // namespace

TCL_API size_t tcl_lateral_param_count(const tcl_config* cfg, int32_t adapter) {
  if (!cfg || adapter <= 0 || cfg->n_layers < 0) return 0;
  return lateral_count(*cfg, adapter);
}

TCL_API tcl_status tcl_lateral_create(tcl_model* kb, tcl_model* ac, int32_t adapter, const float* h_params,
                                      size_t n_params, tcl_lateral** out) {
  if (!out) return fail(TCL_ERR_INVALID_ARG, "out is NULL");
  *out = nullptr;
  if (!kb || !ac || kb == ac) return fail(TCL_ERR_INVALID_ARG, "two distinct models (KB, AC) are required");
  if (!same_architecture(kb->cfg, ac->cfg))
    return fail(TCL_ERR_INVALID_ARG, "the KB and the AC must share one architecture");
  const tcl_config& c = kb->cfg;
  if (c.dtype != TCL_F32) return fail(TCL_ERR_UNSUPPORTED, "the progressive forward needs fp32 models");
  if (c.dec_hidden2 % 4) return fail(TCL_ERR_UNSUPPORTED, "dec_hidden2 must be a multiple of 4");
  if (adapter < 4 || adapter > 512 || adapter % 4)
    return fail(TCL_ERR_UNSUPPORTED, "adapter width must be a multiple of 4 in [4, 512] (got %d)", adapter);
  if (!h_params) return fail(TCL_ERR_INVALID_ARG, "h_params is NULL");
  const size_t need = lateral_count(c, adapter);
  if (n_params != need)
    return fail(TCL_ERR_INVALID_ARG, "lateral blob has %zu values, needs %zu", n_params, need);
  tcl_lateral* lt = new tcl_lateral();
  lt->kb = kb;
  lt->ac = ac;
  lt->a = adapter;
  lt->n_params = n_params;
  // device layout: per adapter V [a, n_in], c [a], U' [n_out, a] with
  // U'[r] = alpha[r] U[r] (fp32 products, formed here once)
  const auto w = layer_widths(c);
  std::vector<float> host;
  std::vector<size_t> offV, offc, offU;
  size_t src = 0;
  auto put = [&](const float* p, size_t n) {
    const size_t at = host.size();
    host.insert(host.end(), p, p + n);
    host.resize((host.size() + 63) & ~size_t(63));  // 256-byte alignment
    return at;
  };
  for (size_t j = 1; j < w.size(); ++j) {
    const int n_in = w[j].first, n_out = w[j].second, a = adapter;
    const float* V = h_params + src;
    const float* cb = V + (size_t)a * n_in;
    const float* U = cb + a;
    const float* al = U + (size_t)n_out * a;
    src += (size_t)a * n_in + a + (size_t)n_out * a + n_out;
    std::vector<float> Uf((size_t)n_out * a);
    for (int r = 0; r < n_out; ++r)
      for (int k = 0; k < a; ++k) Uf[(size_t)r * a + k] = al[r] * U[(size_t)r * a + k];
    offV.push_back(put(V, (size_t)a * n_in));
    offc.push_back(put(cb, a));
    offU.push_back(put(Uf.data(), Uf.size()));
  }
  if (hipMalloc(&lt->dev, std::max<size_t>(host.size(), 64) * 4) != hipSuccess) {
    delete lt;
    return fail(TCL_ERR_OOM, "hipMalloc of the lateral adapters failed");
  }
  if (hipMemcpy(lt->dev, host.data(), host.size() * 4, hipMemcpyHostToDevice) != hipSuccess) {
    (void)hipFree(lt->dev);
    delete lt;
    return fail(TCL_ERR_HIP, "upload of the lateral adapters failed");
  }
  float* base = static_cast<float*>(lt->dev);
  for (size_t j = 1; j < w.size(); ++j) {
    tcl_lateral::Lat L;
    L.n_in = w[j].first;
    L.n_out = w[j].second;
    L.V = base + offV[j - 1];
    L.c = base + offc[j - 1];
    L.U = base + offU[j - 1];
    lt->lats.push_back(L);
  }
  *out = lt;
  return TCL_OK;
}

TCL_API tcl_status tcl_lateral_destroy(tcl_lateral* lt) {
  if (!lt) return TCL_OK;
  if (lt->dev) (void)hipFree(lt->dev);
  delete lt;
  return TCL_OK;
}

TCL_API size_t tcl_progressive_workspace_bytes(const tcl_lateral* lt, int32_t B, int32_t L) {
  if (!lt || B <= 0 || L <= 0) return 0;
  return prog_plan(lt->kb->cfg, lt->a, B, L).total;
}

TCL_API tcl_status tcl_progressive_score(tcl_lateral* lt, int32_t B, int32_t L, const float* d_feats,
                                         const int32_t* d_lengths, float* d_scores, void* d_ws, size_t ws_bytes,
                                         void* stream) {
  if (!lt) return fail(TCL_ERR_INVALID_ARG, "lateral handle is NULL");
  if (B <= 0 || L <= 0) return fail(TCL_ERR_INVALID_ARG, "B and L must be positive (B=%d L=%d)", B, L);
  if ((int64_t)B * L > (int64_t)1 << 30)
    return fail(TCL_ERR_UNSUPPORTED, "B*L = %lld exceeds 2^30 tokens", (long long)B * L);
  if (!d_feats || !d_lengths || !d_scores || !d_ws) return fail(TCL_ERR_INVALID_ARG, "NULL device pointer");
  if (reinterpret_cast<uintptr_t>(d_feats) % 16 || reinterpret_cast<uintptr_t>(d_ws) % 256)
    return fail(TCL_ERR_INVALID_ARG, "d_feats must be 16-byte and d_workspace 256-byte aligned");
  const size_t need = prog_plan(lt->kb->cfg, lt->a, B, L).total;
  if (ws_bytes < need) return fail(TCL_ERR_WORKSPACE, "workspace has %zu bytes, needs %zu", ws_bytes, need);
  return run_progressive(lt, B, L, d_feats, d_lengths, d_scores, static_cast<char*>(d_ws),
                         static_cast<hipStream_t>(stream));
}
