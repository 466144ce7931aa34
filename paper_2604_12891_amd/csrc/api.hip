// Host runtime of libtcl: argument checking, model state, workspace
// planning and the launch sequence of the scoring pass. Every launch is
// stream-ordered on the caller's stream; nothing here synchronises except
// create / set / get, which move parameters between host and device.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <string>
#include <vector>

#include "../../include/tcl.h"
#include "kernels.h"

using namespace tcl;

namespace {

thread_local std::string g_err;

tcl_status fail(tcl_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_err = buf;
  return st;
}

#define TCL_HIP(call)                                                                     \
  do {                                                                                     \
    hipError_t e_ = (call);                                                                \
    if (e_ != hipSuccess) return fail(TCL_ERR_HIP, "%s: %s", #call, hipGetErrorString(e_)); \
  } while (0)

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

// Launch CALL (a hipError_t expression); with timing enabled, bracket it by
// events on stream `s` under category NAME.
#define TCL_LAUNCH(M, NAME, CALL)                                                 \
  do {                                                                           \
    hipEvent_t ea_ = nullptr, eb_ = nullptr;                                     \
    if ((M)->timing.on) {                                                        \
      TCL_HIP((M)->timing.event(&ea_));                                          \
      TCL_HIP(hipEventRecord(ea_, s));                                           \
    }                                                                            \
    TCL_HIP(CALL);                                                               \
    if ((M)->timing.on) {                                                        \
      TCL_HIP((M)->timing.event(&eb_));                                          \
      TCL_HIP(hipEventRecord(eb_, s));                                           \
      (M)->timing.pending.push_back({(M)->timing.category(NAME), ea_, eb_});     \
    }                                                                            \
  } while (0)

// Offsets of each tensor in the canonical blob.
struct BlobLayout {
  size_t W0, b0, g_f, W1, b1, W2, b2, total;
  struct L {
    size_t g, W_in, conv_w, conv_b, W_x, W_dt, b_dt, A_log, D, W_out;
  };
  std::vector<L> layers;
};

BlobLayout blob_layout(const tcl_config& c) {
  BlobLayout bl;
  const size_t d = c.d_model, E = c.d_inner, N = c.d_state, K = c.d_conv, R = c.dt_rank;
  const size_t F = c.F, h = c.head_hidden;
  size_t o = 0;
  bl.W0 = o; o += d * F;
  bl.b0 = o; o += d;
  for (int l = 0; l < c.n_layers; ++l) {
    BlobLayout::L L;
    L.g = o; o += d;
    L.W_in = o; o += 2 * E * d;
    L.conv_w = o; o += E * K;
    L.conv_b = o; o += E;
    L.W_x = o; o += (R + 2 * N) * E;
    L.W_dt = o; o += E * R;
    L.b_dt = o; o += E;
    L.A_log = o; o += E * N;
    L.D = o; o += E;
    L.W_out = o; o += d * E;
    bl.layers.push_back(L);
  }
  bl.g_f = o; o += d;
  bl.W1 = o; o += h * d;
  bl.b1 = o; o += h;
  bl.W2 = o; o += h;
  bl.b2 = o; o += 1;
  bl.total = o;
  return bl;
}

tcl_status check_config(const tcl_config* c) {
  if (!c) return fail(TCL_ERR_INVALID_ARG, "config is NULL");
  if (c->F <= 0 || c->d_model <= 0 || c->d_inner <= 0 || c->d_state <= 0 || c->d_conv <= 0 ||
      c->dt_rank <= 0 || c->n_layers <= 0 || c->head_hidden <= 0 || !(c->norm_eps > 0.f))
    return fail(TCL_ERR_INVALID_ARG, "config has a non-positive field");
  if (c->dtype != TCL_F32 && c->dtype != TCL_BF16)
    return fail(TCL_ERR_INVALID_ARG, "unknown dtype %d", c->dtype);
  if (c->F % 4) return fail(TCL_ERR_UNSUPPORTED, "F must be a multiple of 4 (got %d)", c->F);
  if (c->d_model != 64 && c->d_model != 128 && c->d_model != 256)
    return fail(TCL_ERR_UNSUPPORTED, "d_model must be 64, 128 or 256 (got %d)", c->d_model);
  if (c->d_inner % 64 || c->d_inner > 2048)
    return fail(TCL_ERR_UNSUPPORTED, "d_inner must be a multiple of 64, <= 2048 (got %d)", c->d_inner);
  if (c->d_state != 16) return fail(TCL_ERR_UNSUPPORTED, "d_state must be 16 (got %d)", c->d_state);
  if (c->d_conv > 4) return fail(TCL_ERR_UNSUPPORTED, "d_conv must be <= 4 (got %d)", c->d_conv);
  if (c->dt_rank % 4 || c->dt_rank > 32)
    return fail(TCL_ERR_UNSUPPORTED, "dt_rank must be a multiple of 4, <= 32 (got %d)", c->dt_rank);
  if (c->head_hidden % 64 || c->head_hidden > 256)
    return fail(TCL_ERR_UNSUPPORTED, "head_hidden must be a multiple of 64, <= 256 (got %d)",
                c->head_hidden);
  if (c->n_layers > 16) return fail(TCL_ERR_UNSUPPORTED, "n_layers must be <= 16");
  return TCL_OK;
}

}  // namespace

// Device-side state of a model. All derived weights live in one allocation.
struct tcl_model {
  tcl_config cfg{};
  int device = 0;
  std::vector<float> master;  // canonical fp32 blob
  void* dev = nullptr;
  size_t dev_bytes = 0;
  struct Layer {
    float *W_in, *conv_w, *conv_b, *W_x, *W_dt, *b_dt, *A_log, *D, *W_out;
    float* g;                                    // RMSNorm gain (bf16 path applies it to A)
    uint16_t *W_in_h, *W_x_h, *W_out_h;          // bf16 copies (bf16 models only)
  };
  float *W0 = nullptr, *b0 = nullptr, *g_f = nullptr, *W1T = nullptr, *b1 = nullptr,
        *W2 = nullptr, *b2 = nullptr;
  uint16_t* W0_h = nullptr;  // bf16 [d, ldw0_h], K zero-padded to a multiple of 8
  int ldw0_h = 0;
  std::vector<Layer> layers;

  // Per-kernel event timing (tcl_timing_*).
  struct Timing {
    bool on = false;
    std::vector<std::string> names;
    std::vector<double> total_ms;
    std::vector<int64_t> count;
    struct Pending {
      int cat;
      hipEvent_t a, b;
    };
    std::vector<Pending> pending;
    std::vector<hipEvent_t> pool;
    int category(const char* n) {
      for (size_t i = 0; i < names.size(); ++i)
        if (names[i] == n) return (int)i;
      names.emplace_back(n);
      total_ms.push_back(0.0);
      count.push_back(0);
      return (int)names.size() - 1;
    }
    hipError_t event(hipEvent_t* e) {
      if (!pool.empty()) {
        *e = pool.back();
        pool.pop_back();
        return hipSuccess;
      }
      return hipEventCreate(e);
    }
    hipError_t flush() {
      for (auto& p : pending) {
        hipError_t err = hipEventSynchronize(p.b);
        if (err != hipSuccess) return err;
        float ms = 0.f;
        err = hipEventElapsedTime(&ms, p.a, p.b);
        if (err != hipSuccess) return err;
        total_ms[p.cat] += ms;
        count[p.cat] += 1;
        pool.push_back(p.a);
        pool.push_back(p.b);
      }
      pending.clear();
      return hipSuccess;
    }
    void release() {
      (void)flush();
      for (auto e : pool) (void)hipEventDestroy(e);
      pool.clear();
    }
  } timing;
};

namespace {

uint16_t host_bf16(float f) {
  uint32_t u;
  std::memcpy(&u, &f, 4);
  if ((u & 0x7FFFFFFFu) > 0x7F800000u) return (uint16_t)((u >> 16) | 0x40u);  // quiet NaN
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

float round_bf16(float f) {
  const uint32_t u = (uint32_t)host_bf16(f) << 16;
  float r;
  std::memcpy(&r, &u, 4);
  return r;
}

// Derive the kernel layouts from the master blob and upload them:
//  - fp32 models: W_in gets the pre-norm gain folded in, RMSNorm(h; g) W_in^T
//    = rstd(h) * h (W_in diag(g))^T, so the in_proj GEMM only needs rstd.
//  - bf16 models: every weight is rounded to bf16 (nearest-even) first; the
//    projections are stored as bf16 (W0 zero-padded in K to a multiple of 8)
//    and the gain is applied to the activations, not folded into W_in.
//  - W1 is stored transposed for coalesced reads in the head.
tcl_status upload(tcl_model* m) {
  const tcl_config& c = m->cfg;
  const bool bf = c.dtype == TCL_BF16;
  const BlobLayout bl = blob_layout(c);
  std::vector<float> work(m->master);
  if (bf)
    for (auto& v : work) v = round_bf16(v);
  const float* P = work.data();
  const size_t d = c.d_model, E = c.d_inner, N = c.d_state, K = c.d_conv, R = c.dt_rank;
  const size_t F = c.F, h = c.head_hidden;
  const size_t ldw0h = (F + 7) & ~size_t(7);

  std::vector<uint8_t> host;
  auto put = [&](size_t bytes) {
    const size_t off = host.size();
    host.resize(align256(off + bytes), 0);
    return off;
  };
  auto f32 = [&](size_t off) { return reinterpret_cast<float*>(host.data() + off); };
  auto b16 = [&](size_t off) { return reinterpret_cast<uint16_t*>(host.data() + off); };
  auto copy = [&](size_t src, size_t n) {
    const size_t o = put(n * 4);
    std::memcpy(host.data() + o, P + src, n * 4);
    return o;
  };
  auto copy_h = [&](size_t src, size_t rows, size_t cols, size_t ld) {
    const size_t o = put(rows * ld * 2);
    for (size_t r = 0; r < rows; ++r)
      for (size_t k = 0; k < cols; ++k) b16(o)[r * ld + k] = host_bf16(P[src + r * cols + k]);
    return o;
  };

  const size_t oW0 = copy(bl.W0, d * F), ob0 = copy(bl.b0, d);
  const size_t oW0h = bf ? copy_h(bl.W0, d, F, ldw0h) : 0;
  struct LO { size_t W_in, conv_w, conv_b, W_x, W_dt, b_dt, A_log, D, W_out, g, W_in_h, W_x_h, W_out_h; };
  std::vector<LO> lo;
  for (int l = 0; l < c.n_layers; ++l) {
    const auto& L = bl.layers[l];
    LO o{};
    o.W_in = put(2 * E * d * 4);
    for (size_t j = 0; j < 2 * E; ++j)
      for (size_t k = 0; k < d; ++k)
        f32(o.W_in)[j * d + k] = (float)((double)P[L.W_in + j * d + k] * (double)P[L.g + k]);
    o.conv_w = copy(L.conv_w, E * K);
    o.conv_b = copy(L.conv_b, E);
    o.W_x = copy(L.W_x, (R + 2 * N) * E);
    o.W_dt = copy(L.W_dt, E * R);
    o.b_dt = copy(L.b_dt, E);
    o.A_log = copy(L.A_log, E * N);
    o.D = copy(L.D, E);
    o.W_out = copy(L.W_out, d * E);
    o.g = copy(L.g, d);
    if (bf) {
      o.W_in_h = copy_h(L.W_in, 2 * E, d, d);
      o.W_x_h = copy_h(L.W_x, R + 2 * N, E, E);
      o.W_out_h = copy_h(L.W_out, d, E, E);
    }
    lo.push_back(o);
  }
  const size_t og = copy(bl.g_f, d);
  const size_t oW1T = put(d * h * 4);
  for (size_t j = 0; j < h; ++j)
    for (size_t k = 0; k < d; ++k) f32(oW1T)[k * h + j] = P[bl.W1 + j * d + k];
  const size_t ob1 = copy(bl.b1, h), oW2 = copy(bl.W2, h), ob2 = copy(bl.b2, 1);

  const size_t bytes = host.size();
  if (m->dev && m->dev_bytes != bytes) {
    (void)hipFree(m->dev);
    m->dev = nullptr;
  }
  if (!m->dev) {
    if (hipMalloc(&m->dev, bytes) != hipSuccess) {
      m->dev = nullptr;
      return fail(TCL_ERR_OOM, "hipMalloc of %zu bytes for the weights failed", bytes);
    }
    m->dev_bytes = bytes;
  }
  TCL_HIP(hipMemcpy(m->dev, host.data(), bytes, hipMemcpyHostToDevice));
  uint8_t* base = static_cast<uint8_t*>(m->dev);
  auto F32 = [&](size_t off) { return reinterpret_cast<float*>(base + off); };
  auto B16 = [&](size_t off) { return reinterpret_cast<uint16_t*>(base + off); };
  m->W0 = F32(oW0);
  m->b0 = F32(ob0);
  m->W0_h = bf ? B16(oW0h) : nullptr;
  m->ldw0_h = (int)ldw0h;
  m->layers.clear();
  for (int l = 0; l < c.n_layers; ++l) {
    tcl_model::Layer L{};
    L.W_in = F32(lo[l].W_in);
    L.conv_w = F32(lo[l].conv_w);
    L.conv_b = F32(lo[l].conv_b);
    L.W_x = F32(lo[l].W_x);
    L.W_dt = F32(lo[l].W_dt);
    L.b_dt = F32(lo[l].b_dt);
    L.A_log = F32(lo[l].A_log);
    L.D = F32(lo[l].D);
    L.W_out = F32(lo[l].W_out);
    L.g = F32(lo[l].g);
    if (bf) {
      L.W_in_h = B16(lo[l].W_in_h);
      L.W_x_h = B16(lo[l].W_x_h);
      L.W_out_h = B16(lo[l].W_out_h);
    }
    m->layers.push_back(L);
  }
  m->g_f = F32(og);
  m->W1T = F32(oW1T);
  m->b1 = F32(ob1);
  m->W2 = F32(oW2);
  m->b2 = F32(ob2);
  return TCL_OK;
}

// Workspace plan of one scoring call (byte offsets, 256-aligned).
struct ScorePlan {
  size_t offs, H, xz, u, xdbl, total;
};

ScorePlan score_plan(const tcl_config& c, int64_t B, int64_t L) {
  ScorePlan p;
  const int64_t rows = B * L;
  const int64_t XW = c.dt_rank + 2 * c.d_state;
  const size_t act = c.dtype == TCL_BF16 ? 2 : 4;  // bytes per stored activation
  size_t o = 0;
  p.offs = o; o = align256(o + (size_t)(B + 1) * 4);
  p.H = o; o = align256(o + (size_t)rows * c.d_model * 4);
  p.xz = o; o = align256(o + (size_t)rows * 2 * c.d_inner * act);
  p.u = o; o = align256(o + (size_t)rows * c.d_inner * act);
  p.xdbl = o; o = align256(o + (size_t)rows * XW * 4);
  p.total = o;
  return p;
}

}  // namespace

TCL_API size_t tcl_param_count(const tcl_config* cfg) {
  if (!cfg || cfg->n_layers < 0) return 0;
  return blob_layout(*cfg).total;
}

TCL_API const char* tcl_last_error(void) { return g_err.c_str(); }

TCL_API tcl_status tcl_cost_model_create(const tcl_config* cfg, const float* h_params,
                                         size_t n_params, tcl_model** out) {
  if (!out) return fail(TCL_ERR_INVALID_ARG, "out is NULL");
  *out = nullptr;
  tcl_status st = check_config(cfg);
  if (st != TCL_OK) return st;
  if (!h_params) return fail(TCL_ERR_INVALID_ARG, "h_params is NULL");
  const size_t need = tcl_param_count(cfg);
  if (n_params != need)
    return fail(TCL_ERR_INVALID_ARG, "parameter blob has %zu values, config needs %zu", n_params, need);
  tcl_model* m = new tcl_model();
  m->cfg = *cfg;
  if (hipGetDevice(&m->device) != hipSuccess) {
    delete m;
    return fail(TCL_ERR_HIP, "hipGetDevice failed");
  }
  m->master.assign(h_params, h_params + n_params);
  st = upload(m);
  if (st != TCL_OK) {
    if (m->dev) (void)hipFree(m->dev);
    delete m;
    return st;
  }
  *out = m;
  return TCL_OK;
}

TCL_API tcl_status tcl_cost_model_destroy(tcl_model* m) {
  if (!m) return TCL_OK;
  m->timing.release();
  if (m->dev) (void)hipFree(m->dev);
  delete m;
  return TCL_OK;
}

TCL_API tcl_status tcl_get_params(const tcl_model* m, float* h_out, size_t n) {
  if (!m || !h_out) return fail(TCL_ERR_INVALID_ARG, "NULL argument");
  if (n != m->master.size())
    return fail(TCL_ERR_INVALID_ARG, "buffer has %zu values, model has %zu", n, m->master.size());
  std::memcpy(h_out, m->master.data(), n * 4);
  return TCL_OK;
}

TCL_API tcl_status tcl_set_params(tcl_model* m, const float* h_params, size_t n) {
  if (!m || !h_params) return fail(TCL_ERR_INVALID_ARG, "NULL argument");
  if (n != m->master.size())
    return fail(TCL_ERR_INVALID_ARG, "blob has %zu values, model has %zu", n, m->master.size());
  m->master.assign(h_params, h_params + n);
  return upload(m);
}

TCL_API size_t tcl_score_workspace_bytes(const tcl_model* m, int32_t B, int32_t L) {
  if (!m || B <= 0 || L <= 0) return 0;
  return score_plan(m->cfg, B, L).total;
}

TCL_API tcl_status tcl_score(tcl_model* m, int32_t B, int32_t L, const float* d_feats,
                             const int32_t* d_lengths, float* d_scores, void* d_ws, size_t ws_bytes,
                             void* stream) {
  if (!m) return fail(TCL_ERR_INVALID_ARG, "model is NULL");
  if (B <= 0 || L <= 0) return fail(TCL_ERR_INVALID_ARG, "B and L must be positive (B=%d L=%d)", B, L);
  if ((int64_t)B * L > (int64_t)1 << 30)
    return fail(TCL_ERR_UNSUPPORTED, "B*L = %lld exceeds 2^30 tokens", (long long)B * L);
  if (!d_feats || !d_lengths || !d_scores || !d_ws)
    return fail(TCL_ERR_INVALID_ARG, "NULL device pointer");
  if (reinterpret_cast<uintptr_t>(d_feats) % 16 || reinterpret_cast<uintptr_t>(d_ws) % 256)
    return fail(TCL_ERR_INVALID_ARG, "d_feats must be 16-byte and d_workspace 256-byte aligned");
  const tcl_config& c = m->cfg;
  const ScorePlan p = score_plan(c, B, L);
  if (ws_bytes < p.total)
    return fail(TCL_ERR_WORKSPACE, "workspace has %zu bytes, needs %zu", ws_bytes, p.total);
  hipStream_t s = static_cast<hipStream_t>(stream);
  char* ws = static_cast<char*>(d_ws);
  int* offs = reinterpret_cast<int*>(ws + p.offs);
  float* H = reinterpret_cast<float*>(ws + p.H);
  float* xdbl = reinterpret_cast<float*>(ws + p.xdbl);
  const int d = c.d_model, E = c.d_inner, N = c.d_state, R = c.dt_rank, XW = R + 2 * N;
  const int Mmax = B * L;

  TCL_LAUNCH(m, "offsets", launch_offsets(d_lengths, B, L, offs, s));
  if (c.dtype == TCL_F32) {
    float* xz = reinterpret_cast<float*>(ws + p.xz);
    float* u = reinterpret_cast<float*>(ws + p.u);
    GemmArgs g;
    g.A = d_feats; g.lda = c.F; g.offs = offs; g.B = B; g.L = L;
    g.W = m->W0; g.ldw = c.F; g.bias = m->b0; g.C = H; g.ldc = d;
    g.Mdev = offs + B; g.Mmax = Mmax; g.N = d; g.K = c.F;
    TCL_LAUNCH(m, "gemm_input", launch_gemm_f32(g, kBias | kGather, kWide, s));

    for (int l = 0; l < c.n_layers; ++l) {
      const auto& W = m->layers[l];
      GemmArgs gi;
      gi.A = H; gi.lda = d; gi.W = W.W_in; gi.ldw = d; gi.C = xz; gi.ldc = 2 * E;
      gi.Mdev = offs + B; gi.Mmax = Mmax; gi.N = 2 * E; gi.K = d; gi.eps = c.norm_eps;
      TCL_LAUNCH(m, "gemm_in_proj", launch_gemm_f32(gi, kRowNorm, kWide, s));

      TCL_LAUNCH(m, "conv_silu", launch_conv_silu<float>(B, E, c.d_conv, offs, xz, 2 * E, W.conv_w,
                                                         W.conv_b, u, s));
      GemmArgs gx;
      gx.A = u; gx.lda = E; gx.W = W.W_x; gx.ldw = E; gx.C = xdbl; gx.ldc = XW;
      gx.Mdev = offs + B; gx.Mmax = Mmax; gx.N = XW; gx.K = E;
      TCL_LAUNCH(m, "gemm_x_proj", launch_gemm_f32(gx, 0, kNarrow, s));

      TCL_LAUNCH(m, "scan", launch_scan<float>(B, E, N, R, offs, u, xdbl, xz + E, 2 * E, W.W_dt,
                                               W.b_dt, W.A_log, W.D, u, s));
      GemmArgs go;
      go.A = u; go.lda = E; go.W = W.W_out; go.ldw = E; go.C = H; go.ldc = d;
      go.Mdev = offs + B; go.Mmax = Mmax; go.N = d; go.K = E;
      TCL_LAUNCH(m, "gemm_out_proj", launch_gemm_f32(go, kResid, kWide, s));
    }
  } else {
    uint16_t* xz = reinterpret_cast<uint16_t*>(ws + p.xz);
    uint16_t* u = reinterpret_cast<uint16_t*>(ws + p.u);
    GemmArgsBF16 g;
    g.A = d_feats; g.lda = c.F; g.offs = offs; g.B = B; g.L = L;
    g.W = m->W0_h; g.ldw = m->ldw0_h; g.bias = m->b0; g.C = H; g.ldc = d;
    g.Mdev = offs + B; g.Mmax = Mmax; g.N = d; g.K = c.F;
    TCL_LAUNCH(m, "gemm_input", launch_gemm_bf16(g, kInputF32toF32, s));

    for (int l = 0; l < c.n_layers; ++l) {
      const auto& W = m->layers[l];
      GemmArgsBF16 gi;
      gi.A = H; gi.lda = d; gi.W = W.W_in_h; gi.ldw = d; gi.gain = W.g; gi.C = xz; gi.ldc = 2 * E;
      gi.Mdev = offs + B; gi.Mmax = Mmax; gi.N = 2 * E; gi.K = d; gi.eps = c.norm_eps;
      TCL_LAUNCH(m, "gemm_in_proj", launch_gemm_bf16(gi, kNormF32toBF16, s));

      TCL_LAUNCH(m, "conv_silu", launch_conv_silu<uint16_t>(B, E, c.d_conv, offs, xz, 2 * E,
                                                            W.conv_w, W.conv_b, u, s));
      GemmArgsBF16 gx;
      gx.A = u; gx.lda = E; gx.W = W.W_x_h; gx.ldw = E; gx.C = xdbl; gx.ldc = XW;
      gx.Mdev = offs + B; gx.Mmax = Mmax; gx.N = XW; gx.K = E;
      TCL_LAUNCH(m, "gemm_x_proj", launch_gemm_bf16(gx, kBF16toF32Narrow, s));

      TCL_LAUNCH(m, "scan", launch_scan<uint16_t>(B, E, N, R, offs, u, xdbl, xz + E, 2 * E, W.W_dt,
                                                  W.b_dt, W.A_log, W.D, u, s));
      GemmArgsBF16 go;
      go.A = u; go.lda = E; go.W = W.W_out_h; go.ldw = E; go.C = H; go.ldc = d;
      go.Mdev = offs + B; go.Mmax = Mmax; go.N = d; go.K = E;
      TCL_LAUNCH(m, "gemm_out_proj", launch_gemm_bf16(go, kBF16ResidF32, s));
    }
  }

  TCL_LAUNCH(m, "tail", launch_tail_f32(B, L, d, c.head_hidden, offs, d_lengths, H, m->g_f,
                                        c.final_norm, c.norm_eps, m->W1T, m->b1, m->W2, m->b2,
                                        d_scores, s));
  return TCL_OK;
}

// ------------------------------------------------------------------ timing

TCL_API tcl_status tcl_timing_enable(tcl_model* m, int32_t enable) {
  if (!m) return fail(TCL_ERR_INVALID_ARG, "model is NULL");
  m->timing.on = enable != 0;
  return TCL_OK;
}

TCL_API int32_t tcl_timing_count(const tcl_model* m) {
  return m ? (int32_t)m->timing.names.size() : 0;
}

TCL_API tcl_status tcl_timing_get(tcl_model* m, int32_t idx, const char** name, double* total_ms,
                                  int64_t* launches) {
  if (!m) return fail(TCL_ERR_INVALID_ARG, "model is NULL");
  TCL_HIP(m->timing.flush());
  if (idx < 0 || idx >= (int32_t)m->timing.names.size())
    return fail(TCL_ERR_INVALID_ARG, "timing index %d out of range", idx);
  if (name) *name = m->timing.names[idx].c_str();
  if (total_ms) *total_ms = m->timing.total_ms[idx];
  if (launches) *launches = m->timing.count[idx];
  return TCL_OK;
}

TCL_API tcl_status tcl_timing_reset(tcl_model* m) {
  if (!m) return fail(TCL_ERR_INVALID_ARG, "model is NULL");
  TCL_HIP(m->timing.flush());
  for (auto& t : m->timing.total_ms) t = 0.0;
  for (auto& c : m->timing.count) c = 0;
  return TCL_OK;
}

// ------------------------------------------------------------------ kernel-level entry points

TCL_API tcl_status tcl_test_gemm_f32(int32_t M, int32_t N, int32_t K, const float* d_A,
                                     const float* d_W, const float* d_bias, float* d_C,
                                     void* stream) {
  if (M <= 0 || N <= 0 || K <= 0 || K % 4) return fail(TCL_ERR_INVALID_ARG, "bad M/N/K");
  if (!d_A || !d_W || !d_C) return fail(TCL_ERR_INVALID_ARG, "NULL device pointer");
  if (reinterpret_cast<uintptr_t>(d_A) % 16 || reinterpret_cast<uintptr_t>(d_W) % 16)
    return fail(TCL_ERR_INVALID_ARG, "A and W must be 16-byte aligned");
  GemmArgs g;
  g.A = d_A; g.lda = K; g.W = d_W; g.ldw = K; g.bias = d_bias; g.C = d_C; g.ldc = N;
  g.Mmax = M; g.N = N; g.K = K;
  TCL_HIP(launch_gemm_f32(g, d_bias ? kBias : 0, N <= 64 ? kNarrow : kWide,
                          static_cast<hipStream_t>(stream)));
  return TCL_OK;
}

TCL_API tcl_status tcl_test_conv_silu_f32(int32_t B, int32_t E, int32_t K, const int32_t* d_offs,
                                          const float* d_x, int32_t ldx, const float* d_w,
                                          const float* d_b, float* d_u, void* stream) {
  if (B <= 0 || E <= 0 || K < 1 || K > 4 || ldx < E) return fail(TCL_ERR_INVALID_ARG, "bad sizes");
  if (E % 4 || ldx % 4) return fail(TCL_ERR_INVALID_ARG, "E and ldx must be multiples of 4");
  if (!d_offs || !d_x || !d_w || !d_b || !d_u) return fail(TCL_ERR_INVALID_ARG, "NULL device pointer");
  TCL_HIP(launch_conv_silu<float>(B, E, K, d_offs, d_x, ldx, d_w, d_b, d_u,
                                  static_cast<hipStream_t>(stream)));
  return TCL_OK;
}

TCL_API tcl_status tcl_test_scan_f32(int32_t B, int32_t E, int32_t N, int32_t R,
                                     const int32_t* d_offs, const float* d_u, const float* d_xdbl,
                                     const float* d_z, int32_t ldz, const float* d_W_dt,
                                     const float* d_b_dt, const float* d_A_log, const float* d_D,
                                     float* d_out, void* stream) {
  if (B <= 0 || E <= 0 || ldz < E) return fail(TCL_ERR_INVALID_ARG, "bad sizes");
  if (N != 16) return fail(TCL_ERR_UNSUPPORTED, "d_state must be 16");
  if (R % 4 || R <= 0 || R > 32) return fail(TCL_ERR_UNSUPPORTED, "dt_rank must be 4..32, step 4");
  if (!d_offs || !d_u || !d_xdbl || !d_z || !d_W_dt || !d_b_dt || !d_A_log || !d_D || !d_out)
    return fail(TCL_ERR_INVALID_ARG, "NULL device pointer");
  TCL_HIP(launch_scan<float>(B, E, N, R, d_offs, d_u, d_xdbl, d_z, ldz, d_W_dt, d_b_dt, d_A_log,
                             d_D, d_out, static_cast<hipStream_t>(stream)));
  return TCL_OK;
}

TCL_API tcl_status tcl_test_gemm_bf16(int32_t M, int32_t N, int32_t K, const uint16_t* d_A,
                                      const uint16_t* d_W, const float* d_bias, float* d_C,
                                      void* stream) {
  if (M <= 0 || N <= 0 || K <= 0 || K % 8) return fail(TCL_ERR_INVALID_ARG, "bad M/N/K");
  if (!d_A || !d_W || !d_C) return fail(TCL_ERR_INVALID_ARG, "NULL device pointer");
  if (reinterpret_cast<uintptr_t>(d_A) % 16 || reinterpret_cast<uintptr_t>(d_W) % 16)
    return fail(TCL_ERR_INVALID_ARG, "A and W must be 16-byte aligned");
  GemmArgsBF16 g;
  g.A = d_A; g.lda = K; g.W = d_W; g.ldw = K; g.bias = d_bias; g.C = d_C; g.ldc = N;
  g.Mmax = M; g.N = N; g.K = K;
  TCL_HIP(launch_gemm_bf16(g, d_bias ? kBF16toF32Bias : kBF16toF32, static_cast<hipStream_t>(stream)));
  return TCL_OK;
}
