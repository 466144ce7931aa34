// Host runtime of libtcl: argument checking, model state, weight layouts,
// workspace planning and the launch sequence of the scoring pass. Every
// launch is stream-ordered on the caller's stream; nothing here synchronises
// except create / set / get, which move parameters between host and device.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstring>
#include <mutex>

#include "model.h"

using namespace tcl;

namespace tcl {

namespace {
thread_local std::string g_err;
}

tcl_status fail(tcl_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_err = buf;
  return st;
}

const char* last_error() { return g_err.c_str(); }

int Timing::category(const char* n) {
  for (size_t i = 0; i < names.size(); ++i)
    if (names[i] == n) return (int)i;
  names.emplace_back(n);
  total_ms.push_back(0.0);
  count.push_back(0);
  return (int)names.size() - 1;
}

hipError_t Timing::event(hipEvent_t* e) {
  if (!pool.empty()) {
    *e = pool.back();
    pool.pop_back();
    return hipSuccess;
  }
  return hipEventCreate(e);
}

hipError_t Timing::flush() {
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

void Timing::release() {
  (void)flush();
  for (auto e : pool) (void)hipEventDestroy(e);
  pool.clear();
}

BlobLayout blob_layout(const tcl_config& c) {
  BlobLayout bl;
  const size_t d = c.d_model, E = c.d_inner, N = c.d_state, K = c.d_conv, R = c.dt_rank;
  const size_t F = c.F, h = c.head_hidden;
  size_t o = 0;
  bl.enc_dims[0] = (int)F;
  bl.n_enc = 1;
  for (int i = 0; i < 2 && c.enc_hidden[i] > 0; ++i) bl.enc_dims[bl.n_enc++] = c.enc_hidden[i];
  bl.enc_dims[bl.n_enc] = (int)d;
  for (int i = 0; i < bl.n_enc; ++i) {
    bl.We[i] = o; o += (size_t)bl.enc_dims[i + 1] * bl.enc_dims[i];
    bl.be[i] = o; o += bl.enc_dims[i + 1];
  }
  bl.W0 = bl.We[0];
  bl.b0 = bl.be[0];
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
  const size_t h2 = c.dec_hidden2 > 0 ? c.dec_hidden2 : 0;
  bl.g_f = o; o += d;
  bl.W1 = o; o += h * d;
  bl.b1 = o; o += h;
  if (h2) {
    bl.W2 = o; o += h2 * h;
    bl.b2 = o; o += h2;
    bl.W3 = o; o += h2;
    bl.b3 = o; o += 1;
  } else {
    bl.W2 = o; o += h;
    bl.b2 = o; o += 1;
  }
  bl.total = o;
  return bl;
}

ScorePlan score_plan(const tcl_config& c, int64_t B, int64_t L) {
  ScorePlan p;
  const int64_t rows = B * L;
  const int64_t XW = c.dt_rank + 2 * c.d_state;
  const size_t act = c.dtype == TCL_BF16 ? 2 : 4;  // bytes per stored activation
  size_t o = 0;
  p.offs = o; o = align256(o + (size_t)(B + 1) * 4);
  p.ord = o; o = align256(o + (size_t)B * 4);
  p.tpos = o; o = align256(o + (size_t)rows);
  p.H = o; o = align256(o + (size_t)rows * c.d_model * 4);
  p.xz = o; o = align256(o + (size_t)rows * 2 * c.d_inner * act);
  p.u = o; o = align256(o + (size_t)rows * c.d_inner * act);
  p.xdbl = o; o = align256(o + (size_t)rows * XW * 4);
  // F not a multiple of 4: the features are copied with rows padded to 4
  p.feats = o; if (c.F % 4) o = align256(o + (size_t)rows * ((c.F + 3) & ~3) * 4);
  p.enc1 = o; if (c.enc_hidden[0] > 0) o = align256(o + (size_t)rows * c.enc_hidden[0] * 4);
  p.enc2 = o; if (c.enc_hidden[1] > 0) o = align256(o + (size_t)rows * c.enc_hidden[1] * 4);
  p.total = o;
  return p;
}

tcl_status derive_weights(tcl_model* m, hipStream_t s) {
  TCL_HIP(launch_derive(m->master, m->jobs, m->njobs, m->derive_total, m->dev,
                        m->cfg.dtype == TCL_BF16 ? 1 : 0, s));
  return TCL_OK;
}

hipError_t model_gemm(const tcl_model* m, const GemmArgs& a, const uint16_t* Ws, int ldws, int flags,
                      hipStream_t s) {
  // the split path where it has a kernel for the shape, the fp32 MFMA path otherwise
  if (m->split && Ws && gemm_split_variant(a, flags) > 0) return launch_gemm_split(a, Ws, ldws, flags, -1, s);
  return launch_gemm_f32(a, flags, -1, s);
}

tcl_status enqueue_encoder_layer_f32(tcl_model* m, Timing& T, const std::string& tag, int i, int B, int L,
                                     const int* offs, const float* A, float* C, bool act, hipStream_t s,
                                     uint8_t* tpos_out, bool* tpos_written) {
  if (tpos_written) *tpos_written = false;
  const tcl_config& c = m->cfg;
  const BlobLayout bl = blob_layout(c);
  const int in = i == 0 ? m->ldw0 : bl.enc_dims[i], out = bl.enc_dims[i + 1];
  GemmArgs g;
  g.A = A; g.lda = in; g.C = C; g.ldc = out; g.Mdev = offs + B; g.Mmax = B * L; g.N = out; g.K = in;
  g.relu = act;
  if (i == 0) {
    // the gathered input Linear (rows b*L + t of the padded input)
    g.offs = offs; g.B = B; g.L = L; g.W = m->W0; g.ldw = m->ldw0; g.bias = m->b0;
    // on the split path the row lookup of the gather also yields the token positions
    const bool on_h2 = m->W0_h2 && m->W0_h2_ok && gemm_f16s_supports(g, kBias | kGather);
    const bool on_split = on_h2 || (m->split && m->W0_s && gemm_split_variant(g, kBias | kGather) > 0);
    if (on_split && tpos_out) {
      g.tpos = tpos_out;
      if (tpos_written) *tpos_written = true;
    }
    if (on_h2)
      TCL_LAUNCH(T, (tag + "gemm_input").c_str(), launch_gemm_f16s(g, m->W0_h2, m->ldw0_h, kBias | kGather, s));
    else
      TCL_LAUNCH(T, (tag + "gemm_input").c_str(), model_gemm(m, g, m->W0_s, m->ldw0_h, kBias | kGather, s));
  } else {
    g.W = m->We[i]; g.ldw = in; g.bias = m->be[i];
    if (m->We_h2[i] && m->We_h2_ok[i] && gemm_f16s_supports(g, kBias))
      TCL_LAUNCH(T, (tag + "gemm_encoder").c_str(), launch_gemm_f16s(g, m->We_h2[i], (in + 7) & ~7, kBias, s));
    else
      TCL_LAUNCH(T, (tag + "gemm_encoder").c_str(), model_gemm(m, g, m->We_s[i], (in + 7) & ~7, kBias, s));
  }
  return TCL_OK;
}

tcl_status enqueue_block_f32(tcl_model* m, Timing& T, const std::string& tag, int l, int B, int L,
                             const int* offs, const uint8_t* tpos, float* H, float* xz, float* u, float* xdbl,
                             hipStream_t s, const int* ord) {
  const tcl_config& c = m->cfg;
  const int d = c.d_model, E = c.d_inner, N = c.d_state, R = c.dt_rank, XW = R + 2 * N;
  const int Mmax = B * L;
  const int chunks = scan_chunks_for(B, E, L);
  const auto& W = m->layers[l];
  GemmArgs gi;
  gi.A = H; gi.lda = d; gi.W = W.W_in_fold; gi.ldw = d; gi.C = xz; gi.ldc = 2 * E;
  gi.Mdev = offs + B; gi.Mmax = Mmax; gi.N = 2 * E; gi.K = d; gi.eps = c.norm_eps;
  GemmArgs gx;
  gx.A = u; gx.lda = E; gx.W = W.W_x; gx.ldw = E; gx.C = xdbl; gx.ldc = XW;
  gx.Mdev = offs + B; gx.Mmax = Mmax; gx.N = XW; gx.K = E;
  ConvIn cv;
  cv.x = xz; cv.ldx = 2 * E; cv.w = W.conv_w; cv.b = W.conv_b; cv.tpos = tpos; cv.u = u;
  const bool f16_in = W.W_in_h2 && W.in_h2_ok && gemm_f16s_supports(gi, kRowNorm);
  const bool fused = m->split && W.W_x_s && gemm_split_conv_supports(gx, cv, c.d_conv);
  // with both on the split path, in_proj writes x channel-blocked ([E / 64]
  // blocks of [Mmax][64]) and z after it ([Mmax][E]), so that the conv reads
  // each chunk's rows contiguously
  GemmArgs gib = gi;
  gib.xblk_rows = Mmax; gib.xblk_cols = E;
  ConvIn cvb = cv;
  cvb.xblk_rows = Mmax;
  const bool blk = f16_in && fused && gemm_f16s_supports(gib, kRowNorm | kXBlk) &&
                   gemm_split_conv_supports(gx, cvb, c.d_conv);
  const float* z = blk ? xz + (int64_t)Mmax * E : xz + E;
  const int ldz = blk ? E : 2 * E;
  if (blk)
    TCL_LAUNCH(T, (tag + "gemm_in_proj").c_str(),
               launch_gemm_f16s(gib, W.W_in_h2, (d + 7) & ~7, kRowNorm | kXBlk, s));
  else if (f16_in)
    TCL_LAUNCH(T, (tag + "gemm_in_proj").c_str(), launch_gemm_f16s(gi, W.W_in_h2, (d + 7) & ~7, kRowNorm, s));
  else
    TCL_LAUNCH(T, (tag + "gemm_in_proj").c_str(), model_gemm(m, gi, W.W_in_s, d, kRowNorm, s));
  if (fused) {
    // the conv + SiLU computed in front of x_proj, u stored on the way
    TCL_LAUNCH(T, (tag + "gemm_x_proj_conv").c_str(), launch_gemm_split_conv(gx, blk ? cvb : cv, W.W_x_s, E, s));
  } else {
    TCL_LAUNCH(T, (tag + "conv_silu").c_str(),
               launch_conv_silu<float>(B, E, c.d_conv, offs, xz, 2 * E, W.conv_w, W.conv_b, u, s));
    TCL_LAUNCH(T, (tag + "gemm_x_proj").c_str(), model_gemm(m, gx, W.W_x_s, E, 0, s));
  }
  if (chunks > 0)
    TCL_LAUNCH(T, (tag + "scan_chunked").c_str(),
               launch_scan_chunked<float>(B, E, N, R, chunks, offs, u, xdbl, z, ldz, W.W_dt, W.b_dt,
                                          W.A_log, W.D, u, s));
  else
    TCL_LAUNCH(T, (tag + "scan").c_str(), launch_scan<float>(B, E, N, R, offs, u, xdbl, z, ldz, W.W_dt,
                                                             W.b_dt, W.A_log, W.D, u, s, nullptr, nullptr, 0,
                                                             ord));
  GemmArgs go;
  go.A = u; go.lda = E; go.W = W.W_out; go.ldw = E; go.C = H; go.ldc = d;
  go.Mdev = offs + B; go.Mmax = Mmax; go.N = d; go.K = E;
  if (W.W_out_h2 && W.out_h2_ok && gemm_f16acc_supports(go, kResid))
    TCL_LAUNCH(T, (tag + "gemm_out_proj").c_str(), launch_gemm_f16acc(go, W.W_out_h2, (E + 7) & ~7, kResid, s));
  else
    TCL_LAUNCH(T, (tag + "gemm_out_proj").c_str(), model_gemm(m, go, W.W_out_s, E, kResid, s));
  return TCL_OK;
}

tcl_status run_score_part(tcl_model* m, int B, int L, const float* d_feats, const int* d_lengths,
                          float* d_scores, char* ws, hipStream_t s, int part) {
  const tcl_config& c = m->cfg;
  const bool front = part == 0, tail = part == c.n_layers + 1;
  const int layer = part - 1;  // the block this part runs, when neither front nor tail
  const ScorePlan p = score_plan(c, B, L);
  int* offs = reinterpret_cast<int*>(ws + p.offs);
  float* H = reinterpret_cast<float*>(ws + p.H);
  float* xdbl = reinterpret_cast<float*>(ws + p.xdbl);
  const int d = c.d_model, E = c.d_inner, N = c.d_state, R = c.dt_rank, XW = R + 2 * N;
  const int Mmax = B * L;
  const int chunks = scan_chunks_for(B, E, L);
  Timing& T = m->timing;

  int* ord = reinterpret_cast<int*>(ws + p.ord);  // the programs longest first
  if (front) TCL_LAUNCH(T, "offsets", launch_offsets(d_lengths, B, L, offs, s, ord));
  uint8_t* tpos = reinterpret_cast<uint8_t*>(ws + p.tpos);
  // features whose row length is not a multiple of 4 are first copied into
  // rows padded with zeros (the input Linear reads 16-byte vectors)
  const float* feats = d_feats;
  const int ldf = (c.F + 3) & ~3;
  if (front && ldf != c.F) {
    float* fp = reinterpret_cast<float*>(ws + p.feats);
    TCL_LAUNCH(T, "pad_features", launch_pad_rows(d_feats, (int64_t)B * L, c.F, ldf, fp, s));
    feats = fp;
  }
  if (tail) {
    if (c.dec_hidden2 > 0)
      TCL_LAUNCH(T, "tail", launch_tail3_f32(B, L, d, c.head_hidden, c.dec_hidden2, offs, d_lengths, H, m->g_f,
                                             c.final_norm, c.norm_eps, m->W1T, m->b1, m->W2T, m->b2, m->W3,
                                             m->b3, d_scores, s));
    else
      TCL_LAUNCH(T, "tail", launch_tail_f32(B, L, d, c.head_hidden, offs, d_lengths, H, m->g_f,
                                            c.final_norm, c.norm_eps, m->W1T, m->b1, m->W2, m->b2,
                                            d_scores, s));
    return TCL_OK;
  }
  if (c.dtype == TCL_F32) {
    float* xz = reinterpret_cast<float*>(ws + p.xz);
    float* u = reinterpret_cast<float*>(ws + p.u);
    // encoder: the gathered input Linear, then (multi-layer encoder) the
    // hidden Linear layers on the packed rows, a ReLU after every layer but
    // the last
    if (front) {
      const int n_enc = blob_layout(c).n_enc;
      float* bufs[2] = {reinterpret_cast<float*>(ws + p.enc1), reinterpret_cast<float*>(ws + p.enc2)};
      bool tpos_done = false;
      for (int i = 0; i < n_enc; ++i) {
        const bool last = i == n_enc - 1;
        tcl_status st = enqueue_encoder_layer_f32(m, T, "", i, B, L, offs, i == 0 ? feats : bufs[i - 1],
                                                  last ? H : bufs[i], !last, s, m->split ? tpos : nullptr,
                                                  i == 0 ? &tpos_done : nullptr);
        if (st != TCL_OK) return st;
      }
      // the token positions for the conv fused into x_proj, unless the input Linear wrote them
      if (m->split && !tpos_done) TCL_LAUNCH(T, "token_pos", launch_token_pos(offs, B, tpos, s));
      return TCL_OK;
    }
    return enqueue_block_f32(m, T, "", layer, B, L, offs, m->split ? tpos : nullptr, H, xz, u, xdbl, s,
                             L <= kOrderMaxL ? ord : nullptr);
  } else {
    uint16_t* xz = reinterpret_cast<uint16_t*>(ws + p.xz);
    uint16_t* u = reinterpret_cast<uint16_t*>(ws + p.u);
    if (front) {
      GemmArgsBF16 g;
      g.A = feats; g.lda = ldf; g.offs = offs; g.B = B; g.L = L;
      g.W = m->W0_h; g.ldw = m->ldw0_h; g.bias = m->b0; g.C = H; g.ldc = d;
      g.Mdev = offs + B; g.Mmax = Mmax; g.N = d; g.K = ldf;
      TCL_LAUNCH(T, "gemm_input", launch_gemm_bf16(g, kInputF32toF32, -1, s));
    }

    // the conv + SiLU fused in front of x_proj where the shape allows
    auto conv_args = [&](int l) {
      const auto& W = m->layers[l];
      ConvArgsBF16 a;
      a.x = xz; a.ldx = 2 * E; a.w = W.conv_w; a.b = W.conv_b; a.tpos = tpos; a.u = u;
      a.W = W.W_x_h; a.ldw = E; a.C = xdbl; a.ldc = XW; a.Mdev = offs + B; a.Mmax = Mmax; a.N = XW; a.E = E;
      return a;
    };
    const bool fuse = gemm_bf16_conv_supports(conv_args(0), c.d_conv);
    if (front) {
      if (fuse) TCL_LAUNCH(T, "token_pos", launch_token_pos(offs, B, tpos, s));
      return TCL_OK;
    }
    {
      const int l = layer;
      const auto& W = m->layers[l];
      GemmArgsBF16 gi;
      gi.A = H; gi.lda = d; gi.W = W.W_in_h; gi.ldw = d; gi.gain = W.g; gi.C = xz; gi.ldc = 2 * E;
      gi.Mdev = offs + B; gi.Mmax = Mmax; gi.N = 2 * E; gi.K = d; gi.eps = c.norm_eps;
      TCL_LAUNCH(T, "gemm_in_proj", launch_gemm_bf16(gi, kNormF32toBF16, -1, s));

      if (fuse) {
        TCL_LAUNCH(T, "gemm_x_proj_conv", launch_gemm_bf16_conv(conv_args(l), s));
      } else {
        TCL_LAUNCH(T, "conv_silu", launch_conv_silu<uint16_t>(B, E, c.d_conv, offs, xz, 2 * E,
                                                              W.conv_w, W.conv_b, u, s));
        GemmArgsBF16 gx;
        gx.A = u; gx.lda = E; gx.W = W.W_x_h; gx.ldw = E; gx.C = xdbl; gx.ldc = XW;
        gx.Mdev = offs + B; gx.Mmax = Mmax; gx.N = XW; gx.K = E;
        TCL_LAUNCH(T, "gemm_x_proj", launch_gemm_bf16(gx, kBF16toF32, -1, s));
      }

      if (chunks > 0)
        TCL_LAUNCH(T, "scan_chunked", launch_scan_chunked<uint16_t>(B, E, N, R, chunks, offs, u, xdbl,
                                                                    xz + E, 2 * E, W.W_dt, W.b_dt,
                                                                    W.A_log, W.D, u, s));
      else
        TCL_LAUNCH(T, "scan", launch_scan<uint16_t>(B, E, N, R, offs, u, xdbl, xz + E, 2 * E, W.W_dt,
                                                    W.b_dt, W.A_log, W.D, u, s, nullptr, nullptr, 0,
                                                    L <= kOrderMaxL ? ord : nullptr));
      GemmArgsBF16 go;
      go.A = u; go.lda = E; go.W = W.W_out_h; go.ldw = E; go.C = H; go.ldc = d;
      go.Mdev = offs + B; go.Mmax = Mmax; go.N = d; go.K = E;
      TCL_LAUNCH(T, "gemm_out_proj", launch_gemm_bf16(go, kBF16ResidF32, -1, s));
    }
  }
  return TCL_OK;
}

tcl_status run_score(tcl_model* m, int B, int L, const float* d_feats, const int* d_lengths,
                     float* d_scores, char* ws, hipStream_t s) {
  for (int part = 0; part <= m->cfg.n_layers + 1; ++part) {
    const tcl_status st = run_score_part(m, B, L, d_feats, d_lengths, d_scores, ws, s, part);
    if (st != TCL_OK) return st;
  }
  return TCL_OK;
}

tcl_status check_config(const tcl_config* c) {
  if (!c) return fail(TCL_ERR_INVALID_ARG, "config is NULL");
  if (c->F <= 0 || c->d_model <= 0 || c->d_inner <= 0 || c->d_state <= 0 || c->d_conv <= 0 ||
      c->dt_rank <= 0 || c->n_layers <= 0 || c->head_hidden <= 0 || !(c->norm_eps > 0.f))
    return fail(TCL_ERR_INVALID_ARG, "config has a non-positive field");
  if (c->dtype != TCL_F32 && c->dtype != TCL_BF16)
    return fail(TCL_ERR_INVALID_ARG, "unknown dtype %d", c->dtype);
  if (c->f32_matmul != TCL_F32_MATMUL_SPLIT && c->f32_matmul != TCL_F32_MATMUL_NATIVE &&
      c->f32_matmul != TCL_F32_MATMUL_SPLIT_BF16)
    return fail(TCL_ERR_INVALID_ARG, "unknown f32_matmul %d", c->f32_matmul);
  if (c->F > 1024) return fail(TCL_ERR_UNSUPPORTED, "F must be <= 1024 (got %d)", c->F);
  if (c->d_model != 64 && c->d_model != 128 && c->d_model != 256)
    return fail(TCL_ERR_UNSUPPORTED, "d_model must be 64, 128 or 256 (got %d)", c->d_model);
  if (c->d_inner % 64 || c->d_inner > 2048)
    return fail(TCL_ERR_UNSUPPORTED, "d_inner must be a multiple of 64, <= 2048 (got %d)", c->d_inner);
  if (c->d_state != 16 && c->d_state != 8)
    return fail(TCL_ERR_UNSUPPORTED, "d_state must be 16 or 8 (got %d)", c->d_state);
  if (c->d_conv > 4) return fail(TCL_ERR_UNSUPPORTED, "d_conv must be <= 4 (got %d)", c->d_conv);
  if (c->d_state == 16 && (c->dt_rank % 4 || c->dt_rank > 32))
    return fail(TCL_ERR_UNSUPPORTED, "dt_rank must be a multiple of 4, <= 32 (got %d)", c->dt_rank);
  if (c->d_state == 8 && c->dt_rank != 4 && c->dt_rank != 8 && c->dt_rank != 16)
    return fail(TCL_ERR_UNSUPPORTED, "with d_state 8, dt_rank must be 4, 8 or 16 (got %d)", c->dt_rank);
  const int e1 = c->enc_hidden[0], e2 = c->enc_hidden[1];
  if (e1 < 0 || e2 < 0 || (e1 == 0 && e2 != 0))
    return fail(TCL_ERR_INVALID_ARG, "enc_hidden must be {0, 0}, {e1, 0} or {e1, e2} with e1, e2 > 0");
  if (e1 > 0 && c->dtype != TCL_F32)
    return fail(TCL_ERR_UNSUPPORTED, "a multi-layer encoder needs an fp32 model");
  if (e1 % 4 || e2 % 4 || e1 > 512 || e2 > 512)
    return fail(TCL_ERR_UNSUPPORTED, "enc_hidden widths must be multiples of 4, <= 512 (got %d, %d)", e1, e2);
  if (c->dec_hidden2 < 0 || c->dec_hidden2 > 256)
    return fail(TCL_ERR_UNSUPPORTED, "dec_hidden2 must be in [0, 256] (got %d)", c->dec_hidden2);
  if (c->head_hidden % 64 || c->head_hidden > 256)
    return fail(TCL_ERR_UNSUPPORTED, "head_hidden must be a multiple of 64, <= 256 (got %d)",
                c->head_hidden);
  if (c->n_layers > 16) return fail(TCL_ERR_UNSUPPORTED, "n_layers must be <= 16");
  return TCL_OK;
}

}  // namespace tcl

namespace {

bool uses_split(const tcl_config& c) {
  return c.dtype == TCL_F32 && (c.f32_matmul == TCL_F32_MATMUL_SPLIT || c.f32_matmul == TCL_F32_MATMUL_SPLIT_BF16);
}
// the two-part fp16 GEMMs where their shapes allow (in_proj, the encoder)
bool uses_f16_split(const tcl_config& c) { return c.dtype == TCL_F32 && c.f32_matmul == TCL_F32_MATMUL_SPLIT; }

// Plan of the model's device block: every derived layout, then the master
// blob, then the job table that derives the former from the latter.
struct ModelPlan {
  std::vector<DeriveJob> jobs;
  int64_t total = 0;
  size_t bytes = 0, master = 0, jobtab = 0;
  size_t W0 = 0, b0 = 0, W0_h = 0, W0_s = 0, W0_h2 = 0, g_f = 0, W1 = 0, W1T = 0, b1 = 0, W2 = 0, b2 = 0;
  size_t We[3] = {0, 0, 0}, be[3] = {0, 0, 0}, We_s[3] = {0, 0, 0}, We_h2[3] = {0, 0, 0};
  size_t W2T = 0, W3 = 0, b3 = 0;
  int ldw0 = 0;
  struct L {
    size_t W_in_fold, g, conv_w, conv_b, W_x, W_dt, b_dt, A_log, D, W_out;
    size_t W_outT, W_xT, W_inT, W_dtT, W_in_h, W_x_h, W_out_h, W_in_s, W_x_s, W_out_s, W_in_h2, W_out_h2;
    size_t W_outT_h, W_xT_h, W_inT_h;
  };
  std::vector<L> layers;
  int ldw0_h = 0;
};

// Derived layouts:
//  - fp32 copies of every tensor (bf16-rounded for bf16 models);
//  - W_in with the pre-norm gain folded in, RMSNorm(h; g) W_in^T =
//    rstd(h) * h (W_in diag(g))^T, for the fp32 in_proj (rstd only);
//  - transposed fp32 copies of W_out, W_x, W_in, W_dt (backward GEMMs) and W1
//    (coalesced head reads);
//  - bf16 copies of the projections for bf16 models, W0 zero-padded in K to
//    a multiple of 8 (the padding is zeroed once at create);
//  - three-way bf16 splits of W0, W_in (gain folded) and W_out for fp32
//    models on the split path, [3][rows][ld] each, and two-part fp16 splits
//    of W0, the hidden encoder layers and W_in (gain folded), [2][rows][ld].
ModelPlan plan_model(const tcl_config& c) {
  ModelPlan P;
  const BlobLayout bl = blob_layout(c);
  const bool bf = c.dtype == TCL_BF16;
  const bool sp = uses_split(c);
  const bool h2 = uses_f16_split(c);
  const int d = c.d_model, E = c.d_inner, N = c.d_state, K = c.d_conv, R = c.dt_rank, XW = R + 2 * N;
  const int F = c.F, h = c.head_hidden;
  P.ldw0_h = (F + 7) & ~7;
  P.ldw0 = (F + 3) & ~3;
  size_t o = 0;
  auto job = [&](size_t src, int rows, int cols, int kind, int transpose, int elem_bytes, int ld = -1,
                 size_t src2 = 0) {
    const size_t dst = o;
    const int ldd = ld > 0 ? ld : (transpose ? rows : cols);
    const int parts = (kind == kDeriveSplit || kind == kDeriveFoldSplit) ? 3
                      : (kind == kDeriveSplitF16 || kind == kDeriveFoldSplitF16 || kind == kDeriveSplitF16Flat)
                          ? 2
                          : 1;
    const size_t n_out = parts * (transpose ? (size_t)cols * ldd : (size_t)rows * ldd);
    o = align256(o + n_out * elem_bytes);
    DeriveJob J{};
    J.start = P.total;
    J.src = (int64_t)src;
    J.src2 = (int64_t)src2;
    J.dst = (int64_t)dst;
    J.rows = rows;
    J.cols = cols;
    J.ld = ldd;
    J.transpose = transpose;
    J.kind = kind;
    P.jobs.push_back(J);
    P.total += (int64_t)rows * cols;
    return dst;
  };
  // the encoder's first Linear, K zero-padded; then the hidden layers of a
  // multi-layer encoder
  const int e0 = bl.enc_dims[1];
  P.W0 = job(bl.W0, e0, F, kDeriveF32, 0, 4, P.ldw0);
  P.b0 = job(bl.b0, 1, e0, kDeriveF32, 0, 4);
  if (bf) P.W0_h = job(bl.W0, e0, F, kDeriveBF16, 0, 2, P.ldw0_h);
  if (sp) P.W0_s = job(bl.W0, e0, F, kDeriveSplit, 0, 2, P.ldw0_h);
  if (h2) P.W0_h2 = job(bl.W0, e0, F, kDeriveSplitF16, 0, 2, P.ldw0_h);
  for (int i = 1; i < bl.n_enc; ++i) {
    const int in = bl.enc_dims[i], out = bl.enc_dims[i + 1];
    P.We[i] = job(bl.We[i], out, in, kDeriveF32, 0, 4);
    P.be[i] = job(bl.be[i], 1, out, kDeriveF32, 0, 4);
    if (sp) P.We_s[i] = job(bl.We[i], out, in, kDeriveSplit, 0, 2, (in + 7) & ~7);
    if (h2) P.We_h2[i] = job(bl.We[i], out, in, kDeriveSplitF16, 0, 2, (in + 7) & ~7);
  }
  for (int l = 0; l < c.n_layers; ++l) {
    const auto& B = bl.layers[l];
    ModelPlan::L L{};
    L.W_in_fold = job(B.W_in, 2 * E, d, kDeriveFold, 0, 4, -1, B.g);
    L.g = job(B.g, 1, d, kDeriveF32, 0, 4);
    L.conv_w = job(B.conv_w, E, K, kDeriveF32, 0, 4);
    L.conv_b = job(B.conv_b, 1, E, kDeriveF32, 0, 4);
    L.W_x = job(B.W_x, XW, E, kDeriveF32, 0, 4);
    L.W_dt = job(B.W_dt, E, R, kDeriveF32, 0, 4);
    L.b_dt = job(B.b_dt, 1, E, kDeriveF32, 0, 4);
    L.A_log = job(B.A_log, E, N, kDeriveF32, 0, 4);
    L.D = job(B.D, 1, E, kDeriveF32, 0, 4);
    L.W_out = job(B.W_out, d, E, kDeriveF32, 0, 4);
    L.W_outT = job(B.W_out, d, E, kDeriveF32, 1, 4);
    L.W_xT = job(B.W_x, XW, E, kDeriveF32, 1, 4);
    L.W_inT = job(B.W_in, 2 * E, d, kDeriveF32, 1, 4);
    L.W_dtT = job(B.W_dt, E, R, kDeriveF32, 1, 4);
    if (bf) {
      L.W_in_h = job(B.W_in, 2 * E, d, kDeriveBF16, 0, 2);
      L.W_x_h = job(B.W_x, XW, E, kDeriveBF16, 0, 2);
      L.W_out_h = job(B.W_out, d, E, kDeriveBF16, 0, 2);
      L.W_outT_h = job(B.W_out, d, E, kDeriveBF16, 1, 2);
      L.W_xT_h = job(B.W_x, XW, E, kDeriveBF16, 1, 2);
      L.W_inT_h = job(B.W_in, 2 * E, d, kDeriveBF16, 1, 2);
    }
    if (sp) {
      L.W_in_s = job(B.W_in, 2 * E, d, kDeriveFoldSplit, 0, 2, -1, B.g);
      L.W_x_s = job(B.W_x, XW, E, kDeriveSplit, 0, 2);
      L.W_out_s = job(B.W_out, d, E, kDeriveSplit, 0, 2);
    }
    if (h2) {
      L.W_in_h2 = job(B.W_in, 2 * E, d, kDeriveFoldSplitF16, 0, 2, (d + 7) & ~7, B.g);
      L.W_out_h2 = job(B.W_out, d, E, kDeriveSplitF16Flat, 0, 2, (E + 7) & ~7);
    }
    P.layers.push_back(L);
  }
  P.g_f = job(bl.g_f, 1, d, kDeriveF32, 0, 4);
  P.W1 = job(bl.W1, h, d, kDeriveF32, 0, 4);
  P.W1T = job(bl.W1, h, d, kDeriveF32, 1, 4);
  P.b1 = job(bl.b1, 1, h, kDeriveF32, 0, 4);
  if (c.dec_hidden2 > 0) {
    const int h2 = c.dec_hidden2;
    P.W2 = job(bl.W2, h2, h, kDeriveF32, 0, 4);
    P.W2T = job(bl.W2, h2, h, kDeriveF32, 1, 4);
    P.b2 = job(bl.b2, 1, h2, kDeriveF32, 0, 4);
    P.W3 = job(bl.W3, 1, h2, kDeriveF32, 0, 4);
    P.b3 = job(bl.b3, 1, 1, kDeriveF32, 0, 4);
  } else {
    P.W2 = job(bl.W2, 1, h, kDeriveF32, 0, 4);
    P.b2 = job(bl.b2, 1, 1, kDeriveF32, 0, 4);
  }
  P.master = o;
  o = align256(o + bl.total * 4);
  P.jobtab = o;
  o = align256(o + P.jobs.size() * sizeof(DeriveJob));
  P.bytes = o;
  return P;
}

// Upload a host blob into the model's master and derive every layout.
// Synchronous.
// Which matrices the two-part fp16 GEMMs may take: every (gain-folded)
// weight below 32 in magnitude, so that its 2^10 scale stays in fp16's range
// (the others keep the three-part bf16 split).
void check_f16_ranges(tcl_model* m, const float* hp) {
  const tcl_config& c = m->cfg;
  if (!uses_f16_split(c)) return;
  const BlobLayout bl = blob_layout(c);
  auto fits = [&](size_t off, int rows, int cols, const float* g) {
    for (int r = 0; r < rows; ++r)
      for (int k = 0; k < cols; ++k) {
        const float v = hp[off + (size_t)r * cols + k] * (g ? g[k] : 1.0f);
        if (!(fabsf(v) < 32.0f)) return false;
      }
    return true;
  };
  m->W0_h2_ok = fits(bl.W0, bl.enc_dims[1], c.F, nullptr);
  for (int i = 1; i < bl.n_enc; ++i) m->We_h2_ok[i] = fits(bl.We[i], bl.enc_dims[i + 1], bl.enc_dims[i], nullptr);
  for (int l = 0; l < c.n_layers; ++l) {
    m->layers[l].in_h2_ok = fits(bl.layers[l].W_in, 2 * c.d_inner, c.d_model, hp + bl.layers[l].g);
    m->layers[l].out_h2_ok = fits(bl.layers[l].W_out, c.d_model, c.d_inner, nullptr);
  }
}

tcl_status load_params(tcl_model* m, const float* h_params) {
  check_f16_ranges(m, h_params);
  TCL_HIP(hipMemcpy(m->master, h_params, m->n_params * 4, hipMemcpyHostToDevice));
  tcl_status st = derive_weights(m, nullptr);
  if (st != TCL_OK) return st;
  TCL_HIP(hipStreamSynchronize(nullptr));
  return TCL_OK;
}

}  // namespace

TCL_API size_t tcl_param_count(const tcl_config* cfg) {
  if (!cfg || cfg->n_layers < 0) return 0;
  return blob_layout(*cfg).total;
}

TCL_API const char* tcl_last_error(void) { return last_error(); }

namespace {
// Batches of at least this many programs are scored as two concurrent halves.
// Measured at L = 25, d_model 256, 4 blocks: two halves take 0.98x (B =
// 2048), 0.86x (3072), 0.97x (4096), 0.98x (8192) the time of one pass,
// 0.99x at 1536, 1.0x at 1024 and up to 1.07x below 768, where each half's
// kernels are bound by the latency of their few workgroups; four quarters
// at B = 4096 took 1.1x.
constexpr int kScoreSplitMinB = 2048;

bool score_split(const tcl_model* m, int B, int L) {
  return m->score_streams == 2 && m->aux[0] && m->aux[1] && B >= kScoreSplitMinB &&
         ((int64_t)(B / 2) * L * m->cfg.F * 4) % 16 == 0;  // the second half's features stay 16-byte aligned
}

size_t score_ws_bytes(const tcl_model* m, int B, int L) {
  if (!score_split(m, B, L)) return score_plan(m->cfg, B, L).total;
  const int h = B / 2;
  return align256(score_plan(m->cfg, h, L).total) + score_plan(m->cfg, B - h, L).total;
}

void release_streams(tcl_model* m) {
  for (auto& e : m->ev)
    if (e) (void)hipEventDestroy(e), e = nullptr;
  for (auto& q : m->aux)
    if (q) (void)hipStreamDestroy(q), q = nullptr;
}
}  // namespace

// ------------------------------------------------------------------ scratch for tcl_score_noalloc
// tcl_score's workspace for callers that cannot allocate: one file-scope
// device array per GPU, held until the process ends. Host code never uses
// the array's name as an address (on the host it names a stand-in, not
// device memory): each device's copy is looked up once with
// hipGetSymbolAddress, with that device current, and kept in g_scratch.
constexpr size_t kScratchBytes = (size_t)256 << 20;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

namespace {
constexpr int kMaxScratchDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch[kMaxScratchDevices] = {};

// This device's copy of `scratch`; `dev` must be the current device.
tcl_status scratch_ptr(int dev, void** out) {
  *out = nullptr;
  if (dev < 0 || dev >= kMaxScratchDevices)
    return fail(TCL_ERR_UNSUPPORTED, "device %d beyond the %d the scratch table holds", dev, kMaxScratchDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p) {
      (void)hipGetLastError();
      return fail(TCL_ERR_HIP, "hipGetSymbolAddress of the scratch buffer failed on device %d: %s", dev,
                  hipGetErrorString(e));
    }
    g_scratch[dev] = p;
  }
  *out = g_scratch[dev];
  return TCL_OK;
}
}  // namespace

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
  m->n_params = n_params;
  if (hipGetDevice(&m->device) != hipSuccess) {
    delete m;
    return fail(TCL_ERR_HIP, "hipGetDevice failed");
  }
  const ModelPlan P = plan_model(*cfg);
  if (hipMalloc(&m->dev, P.bytes) != hipSuccess) {
    delete m;
    return fail(TCL_ERR_OOM, "hipMalloc of %zu bytes for the weights failed", P.bytes);
  }
  m->dev_bytes = P.bytes;
  uint8_t* base = static_cast<uint8_t*>(m->dev);
  auto F32 = [&](size_t off) { return reinterpret_cast<float*>(base + off); };
  auto B16 = [&](size_t off) { return reinterpret_cast<uint16_t*>(base + off); };
  const bool bf = cfg->dtype == TCL_BF16;
  m->master = F32(P.master);
  m->jobs = reinterpret_cast<DeriveJob*>(base + P.jobtab);
  m->njobs = (int)P.jobs.size();
  m->derive_total = P.total;
  m->W0 = F32(P.W0);
  m->b0 = F32(P.b0);
  m->W0_h = bf ? B16(P.W0_h) : nullptr;
  m->ldw0_h = P.ldw0_h;
  m->ldw0 = P.ldw0;
  m->split = uses_split(*cfg);
  m->W0_s = m->split ? B16(P.W0_s) : nullptr;
  m->W0_h2 = uses_f16_split(*cfg) ? B16(P.W0_h2) : nullptr;
  for (const auto& L : P.layers) {
    tcl_model::Layer W{};
    W.W_in_fold = F32(L.W_in_fold);
    W.g = F32(L.g);
    W.conv_w = F32(L.conv_w);
    W.conv_b = F32(L.conv_b);
    W.W_x = F32(L.W_x);
    W.W_dt = F32(L.W_dt);
    W.b_dt = F32(L.b_dt);
    W.A_log = F32(L.A_log);
    W.D = F32(L.D);
    W.W_out = F32(L.W_out);
    W.W_outT = F32(L.W_outT);
    W.W_xT = F32(L.W_xT);
    W.W_inT = F32(L.W_inT);
    W.W_dtT = F32(L.W_dtT);
    if (bf) {
      W.W_in_h = B16(L.W_in_h);
      W.W_x_h = B16(L.W_x_h);
      W.W_out_h = B16(L.W_out_h);
      W.W_outT_h = B16(L.W_outT_h);
      W.W_xT_h = B16(L.W_xT_h);
      W.W_inT_h = B16(L.W_inT_h);
    }
    if (m->split) {
      W.W_in_s = B16(L.W_in_s);
      W.W_x_s = B16(L.W_x_s);
      W.W_out_s = B16(L.W_out_s);
    }
    W.W_in_h2 = uses_f16_split(*cfg) ? B16(L.W_in_h2) : nullptr;
    W.W_out_h2 = uses_f16_split(*cfg) ? B16(L.W_out_h2) : nullptr;
    m->layers.push_back(W);
  }
  m->g_f = F32(P.g_f);
  m->W1 = F32(P.W1);
  m->W1T = F32(P.W1T);
  m->b1 = F32(P.b1);
  m->b2 = F32(P.b2);
  m->W2 = F32(P.W2);
  if (cfg->dec_hidden2 > 0) {
    m->W2T = F32(P.W2T);
    m->W3 = F32(P.W3);
    m->b3 = F32(P.b3);
  }
  {
    const BlobLayout bl = blob_layout(*cfg);
    for (int i = 1; i < bl.n_enc; ++i) {
      m->We[i] = F32(P.We[i]);
      m->be[i] = F32(P.be[i]);
      if (m->split) m->We_s[i] = B16(P.We_s[i]);
      if (uses_f16_split(*cfg)) m->We_h2[i] = B16(P.We_h2[i]);
    }
  }
  auto cleanup = [&](tcl_status s2) {
    (void)hipFree(m->dev);
    delete m;
    return s2;
  };
  // zero the block once: padding (W0's bf16 K tail) is never written again
  if (hipMemset(m->dev, 0, P.bytes) != hipSuccess) return cleanup(fail(TCL_ERR_HIP, "hipMemset failed"));
  if (hipMemcpy(m->jobs, P.jobs.data(), P.jobs.size() * sizeof(DeriveJob), hipMemcpyHostToDevice) !=
      hipSuccess)
    return cleanup(fail(TCL_ERR_HIP, "upload of the derivation table failed"));
  st = load_params(m, h_params);
  if (st != TCL_OK) return cleanup(st);
  {
    // set-up of tcl_score_noalloc's buffer on this device (the model's
    // device is current here); a failure is reported by that entry point
    void* unused = nullptr;
    if (scratch_ptr(m->device, &unused) != TCL_OK) (void)hipGetLastError();
  }
  // default-priority streams for tcl_score's half batches
  bool ok = true;
  for (int i = 0; i < 2 && ok; ++i) ok = hipStreamCreateWithFlags(&m->aux[i], hipStreamNonBlocking) == hipSuccess;
  for (int i = 0; i < 3 && ok; ++i) ok = hipEventCreateWithFlags(&m->ev[i], hipEventDisableTiming) == hipSuccess;
  if (!ok) {
    release_streams(m);
    (void)hipGetLastError();
  }
  *out = m;
  return TCL_OK;
}

TCL_API tcl_status tcl_cost_model_destroy(tcl_model* m) {
  if (!m) return TCL_OK;
  release_streams(m);
  m->timing.release();
  if (m->dev) (void)hipFree(m->dev);
  delete m;
  return TCL_OK;
}

TCL_API tcl_status tcl_get_params(const tcl_model* m, float* h_out, size_t n) {
  if (!m || !h_out) return fail(TCL_ERR_INVALID_ARG, "NULL argument");
  if (n != m->n_params)
    return fail(TCL_ERR_INVALID_ARG, "buffer has %zu values, model has %zu", n, m->n_params);
  TCL_HIP(hipDeviceSynchronize());
  TCL_HIP(hipMemcpy(h_out, m->master, n * 4, hipMemcpyDeviceToHost));
  return TCL_OK;
}

TCL_API tcl_status tcl_set_params(tcl_model* m, const float* h_params, size_t n) {
  if (!m || !h_params) return fail(TCL_ERR_INVALID_ARG, "NULL argument");
  if (n != m->n_params)
    return fail(TCL_ERR_INVALID_ARG, "blob has %zu values, model has %zu", n, m->n_params);
  TCL_HIP(hipDeviceSynchronize());
  return load_params(m, h_params);
}

TCL_API size_t tcl_score_workspace_bytes(const tcl_model* m, int32_t B, int32_t L) {
  if (!m || B <= 0 || L <= 0) return 0;
  return score_ws_bytes(m, B, L);
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
  const size_t need = score_ws_bytes(m, B, L);
  if (ws_bytes < need) return fail(TCL_ERR_WORKSPACE, "workspace has %zu bytes, needs %zu", ws_bytes, need);
  const hipStream_t s = static_cast<hipStream_t>(stream);
  char* ws = static_cast<char*>(d_ws);
  if (!score_split(m, B, L)) return run_score(m, B, L, d_feats, d_lengths, d_scores, ws, s);
  // two half batches on the model's two streams, forked from and joined
  // back into the caller's stream: each half's kernels fill the CUs the
  // other's leave idle (launch gaps, the last round of a grid)
  const int h = B / 2;
  const size_t off2 = align256(score_plan(m->cfg, h, L).total);
  TCL_HIP(hipEventRecord(m->ev[0], s));
  TCL_HIP(hipStreamWaitEvent(m->aux[0], m->ev[0], 0));
  TCL_HIP(hipStreamWaitEvent(m->aux[1], m->ev[0], 0));
  // the halves' launches alternate part by part (the front, each block, the
  // tail), so that the second half starts after the first half's first part
  // is enqueued rather than after all of it
  for (int part = 0; part <= m->cfg.n_layers + 1; ++part) {
    tcl_status st = run_score_part(m, h, L, d_feats, d_lengths, d_scores, ws, m->aux[0], part);
    if (st != TCL_OK) return st;
    st = run_score_part(m, B - h, L, d_feats + (int64_t)h * L * m->cfg.F, d_lengths + h, d_scores + h,
                        ws + off2, m->aux[1], part);
    if (st != TCL_OK) return st;
  }
  TCL_HIP(hipEventRecord(m->ev[1], m->aux[0]));
  TCL_HIP(hipEventRecord(m->ev[2], m->aux[1]));
  TCL_HIP(hipStreamWaitEvent(s, m->ev[1], 0));
  TCL_HIP(hipStreamWaitEvent(s, m->ev[2], 0));
  return TCL_OK;
}

TCL_API size_t tcl_score_noalloc_max_bytes(void) { return kScratchBytes; }

TCL_API tcl_status tcl_score_noalloc(tcl_model* m, int32_t B, int32_t L, const float* d_feats,
                                     const int32_t* d_lengths, float* d_scores, void* stream) {
  if (!m) return fail(TCL_ERR_INVALID_ARG, "model is NULL");
  if (B <= 0 || L <= 0) return fail(TCL_ERR_INVALID_ARG, "B and L must be positive (B=%d L=%d)", B, L);
  if (!d_feats || !d_lengths || !d_scores) return fail(TCL_ERR_INVALID_ARG, "NULL device pointer");
  if (reinterpret_cast<uintptr_t>(d_feats) % 16) return fail(TCL_ERR_INVALID_ARG, "d_feats must be 16-byte aligned");
  if (m->timing.on)
    return fail(TCL_ERR_INVALID_ARG, "per-kernel timing creates events: disable it for tcl_score_noalloc");
  const size_t need = score_plan(m->cfg, B, L).total;
  if ((int64_t)B * L > (int64_t)1 << 30 || need > kScratchBytes)
    return fail(TCL_ERR_UNSUPPORTED,
                "B=%d L=%d needs %zu bytes of workspace, more than the %zu of the library's scratch buffer "
                "(use tcl_score with a caller-owned workspace)", B, L, need, kScratchBytes);
  int cur = -1;
  TCL_HIP(hipGetDevice(&cur));
  if (cur != m->device)
    return fail(TCL_ERR_INVALID_ARG, "the model's device %d must be current (current: %d)", m->device, cur);
  void* ws = nullptr;
  const tcl_status st = scratch_ptr(m->device, &ws);
  if (st != TCL_OK) return st;
  // one pass on the caller's stream (no fork onto the model's streams)
  return run_score(m, B, L, d_feats, d_lengths, d_scores, static_cast<char*>(ws),
                   static_cast<hipStream_t>(stream));
}

// ------------------------------------------------------------------ timing

TCL_API tcl_status tcl_set_score_streams(tcl_model* m, int32_t n) {
  if (!m) return fail(TCL_ERR_INVALID_ARG, "model is NULL");
  if (n != 1 && n != 2) return fail(TCL_ERR_INVALID_ARG, "n must be 1 or 2 (got %d)", n);
  m->score_streams = n;
  return TCL_OK;
}

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

// ------------------------------------------------------------------ score consumers

TCL_API tcl_status tcl_topk(int32_t n_seg, const int32_t* d_seg_offsets, const float* d_scores, int32_t K,
                            int32_t* d_out, void* stream) {
  if (n_seg <= 0) return fail(TCL_ERR_INVALID_ARG, "n_seg must be positive");
  if (K < 1 || K > 1024) return fail(TCL_ERR_UNSUPPORTED, "K must be in [1, 1024] (got %d)", K);
  if (!d_seg_offsets || !d_scores || !d_out) return fail(TCL_ERR_INVALID_ARG, "NULL device pointer");
  TCL_HIP(launch_topk(n_seg, d_seg_offsets, d_scores, K, d_out, static_cast<hipStream_t>(stream)));
  return TCL_OK;
}

TCL_API size_t tcl_topk_score_workspace_bytes(int32_t n_seg, int32_t k) {
  if (n_seg <= 0 || k < 1 || k > 1024) return 0;
  return topk_score_workspace_bytes(n_seg, k);
}

TCL_API tcl_status tcl_topk_score(int32_t n_seg, const int32_t* d_seg_offsets, const float* d_scores,
                                  const float* d_latency, const float* d_weight, int32_t k, double* d_out,
                                  void* d_workspace, size_t ws_bytes, void* stream) {
  if (n_seg <= 0) return fail(TCL_ERR_INVALID_ARG, "n_seg must be positive");
  if (k < 1 || k > 1024) return fail(TCL_ERR_UNSUPPORTED, "k must be in [1, 1024] (got %d)", k);
  if (!d_seg_offsets || !d_scores || !d_latency || !d_weight || !d_out || !d_workspace)
    return fail(TCL_ERR_INVALID_ARG, "NULL device pointer");
  if (reinterpret_cast<uintptr_t>(d_workspace) % 256) return fail(TCL_ERR_INVALID_ARG, "d_workspace must be 256-byte aligned");
  const size_t need = topk_score_workspace_bytes(n_seg, k);
  if (ws_bytes < need) return fail(TCL_ERR_WORKSPACE, "workspace has %zu bytes, needs %zu", ws_bytes, need);
  TCL_HIP(launch_topk_score(n_seg, d_seg_offsets, d_scores, d_latency, d_weight, k, d_out, d_workspace,
                            static_cast<hipStream_t>(stream)));
  return TCL_OK;
}

TCL_API size_t tcl_rdu_workspace_bytes(int32_t N, int32_t n_ops) {
  if (N <= 0 || n_ops <= 0 || n_ops > 4096) return 0;
  return rdu_workspace_bytes(N, n_ops);
}

TCL_API tcl_status tcl_rdu_select(int32_t N, const float* d_scores, const int32_t* d_op, int32_t n_ops,
                                  const int32_t* d_initial, int32_t n_initial, int32_t n_select,
                                  int32_t* d_selected, int32_t* d_count, void* d_workspace, size_t ws_bytes,
                                  void* stream) {
  if (N <= 0 || n_select < 0 || n_initial < 1)
    return fail(TCL_ERR_INVALID_ARG, "need N > 0, n_initial > 0 (Eq. (1) needs a labeled set), n_select >= 0");
  if (n_ops <= 0 || n_ops > 4096) return fail(TCL_ERR_UNSUPPORTED, "n_ops must be in [1, 4096] (got %d)", n_ops);
  if (!d_scores || !d_op || !d_initial || !d_count || (n_select > 0 && !d_selected) || !d_workspace)
    return fail(TCL_ERR_INVALID_ARG, "NULL device pointer");
  if (reinterpret_cast<uintptr_t>(d_workspace) % 256) return fail(TCL_ERR_INVALID_ARG, "d_workspace must be 256-byte aligned");
  const size_t need = rdu_workspace_bytes(N, n_ops);
  if (ws_bytes < need) return fail(TCL_ERR_WORKSPACE, "workspace has %zu bytes, needs %zu", ws_bytes, need);
  TCL_HIP(launch_rdu_select(N, d_scores, d_op, n_ops, d_initial, n_initial, n_select, d_selected, d_count,
                            d_workspace, static_cast<hipStream_t>(stream)));
  return TCL_OK;
}

// ------------------------------------------------------------------ kernel-level entry points

TCL_API tcl_status tcl_test_gemm_f32(int32_t M, int32_t N, int32_t K, const float* d_A,
                                     const float* d_W, const float* d_bias, float* d_C, int32_t tile,
                                     int32_t epilogue, void* stream) {
  if (M <= 0 || N <= 0 || K <= 0 || K % 4) return fail(TCL_ERR_INVALID_ARG, "bad M/N/K");
  if (tile < -1 || tile >= kNumGemmTiles) return fail(TCL_ERR_INVALID_ARG, "bad tile id %d", tile);
  if (epilogue < 0 || epilogue > 2) return fail(TCL_ERR_INVALID_ARG, "bad epilogue %d", epilogue);
  if (epilogue == 1 && d_bias) return fail(TCL_ERR_INVALID_ARG, "bias and residual are exclusive");
  if (!d_A || !d_W || !d_C) return fail(TCL_ERR_INVALID_ARG, "NULL device pointer");
  if (reinterpret_cast<uintptr_t>(d_A) % 16 || reinterpret_cast<uintptr_t>(d_W) % 16)
    return fail(TCL_ERR_INVALID_ARG, "A and W must be 16-byte aligned");
  GemmArgs g;
  g.A = d_A; g.lda = K; g.W = d_W; g.ldw = K; g.bias = d_bias; g.C = d_C; g.ldc = N;
  g.Mmax = M; g.N = N; g.K = K;
  g.eps = 1e-5f;
  const int flags = epilogue == 1 ? kResid : epilogue == 2 ? kRowNorm : (d_bias ? kBias : 0);
  if (epilogue == 2 && d_bias) return fail(TCL_ERR_INVALID_ARG, "bias and row norm are exclusive");
  TCL_HIP(launch_gemm_f32(g, flags, tile, static_cast<hipStream_t>(stream)));
  return TCL_OK;
}

TCL_API tcl_status tcl_test_gemm_split(int32_t M, int32_t N, int32_t K, const float* d_A,
                                       const int32_t* d_offs, int32_t B, int32_t L, const float* d_W,
                                       const float* d_bias, float* d_C, int32_t variant,
                                       int32_t epilogue, uint16_t* d_Wsplit, void* stream) {
  if (epilogue < 0 || epilogue > 3) return fail(TCL_ERR_INVALID_ARG, "bad epilogue %d", epilogue);
  if (epilogue == 3) {
    if (B <= 0 || L <= 0 || !d_offs) return fail(TCL_ERR_INVALID_ARG, "gather needs d_offs, B > 0, L > 0");
    if (!d_bias) return fail(TCL_ERR_INVALID_ARG, "the gathered input Linear needs d_bias");
    M = B * L;
  }
  if (M <= 0 || N <= 0 || K <= 0 || K % 4) return fail(TCL_ERR_INVALID_ARG, "bad M/N/K");
  if (variant < -1 || variant > 6 || variant == 0)
    return fail(TCL_ERR_INVALID_ARG, "variant must be -1 or 1..6 (got %d)", variant);
  if ((epilogue == 1 || epilogue == 2) && d_bias)
    return fail(TCL_ERR_INVALID_ARG, "bias goes with epilogues 0 and 3 only");
  if (!d_A || !d_W || !d_C || !d_Wsplit) return fail(TCL_ERR_INVALID_ARG, "NULL device pointer");
  if (reinterpret_cast<uintptr_t>(d_A) % 16 || reinterpret_cast<uintptr_t>(d_Wsplit) % 16)
    return fail(TCL_ERR_INVALID_ARG, "A and the split buffer must be 16-byte aligned");
  const hipStream_t s = static_cast<hipStream_t>(stream);
  const int Kw = (K + 7) & ~7;
  GemmArgs g;
  g.A = d_A; g.lda = K; g.W = d_W; g.ldw = K; g.bias = d_bias; g.C = d_C; g.ldc = N;
  g.Mmax = M; g.N = N; g.K = K; g.eps = 1e-5f;
  int flags = epilogue == 1 ? kResid : epilogue == 2 ? kRowNorm : (d_bias ? kBias : 0);
  if (epilogue == 3) {
    g.offs = d_offs; g.B = B; g.L = L; g.Mdev = d_offs + B;
    flags = kBias | kGather;
  }
  if (variant == 6) {  // the two-part fp16 panels with all N in registers
    if (!gemm_f16acc_supports(g, flags))
      return fail(TCL_ERR_UNSUPPORTED, "no fp16 all-N kernel for N=%d K=%d with epilogue %d", N, K, epilogue);
    TCL_HIP(launch_split_weights_f16(d_W, N, K, Kw, d_Wsplit, s, true));
    TCL_HIP(launch_gemm_f16acc(g, d_Wsplit, Kw, flags, s));
    return TCL_OK;
  }
  if (variant == 5) {  // the two-part fp16 panels
    if (!gemm_f16s_supports(g, flags))
      return fail(TCL_ERR_UNSUPPORTED, "no fp16 split kernel for N=%d K=%d with epilogue %d", N, K, epilogue);
    TCL_HIP(launch_split_weights_f16(d_W, N, K, Kw, d_Wsplit, s));
    TCL_HIP(launch_gemm_f16s(g, d_Wsplit, Kw, flags, s));
    return TCL_OK;
  }
  const int v = variant < 0 ? gemm_split_variant(g, flags) : variant;
  if (v < 0 || !gemm_split_supports(g, flags, v))
    return fail(TCL_ERR_UNSUPPORTED, "no split kernel for N=%d K=%d with epilogue %d (variant %d)", N, K,
                epilogue, variant);
  TCL_HIP(launch_split_weights(d_W, N, K, Kw, d_Wsplit, s));
  TCL_HIP(launch_gemm_split(g, d_Wsplit, Kw, flags, v, s));
  return TCL_OK;
}

TCL_API tcl_status tcl_test_gemm_bf16(int32_t kind, int32_t tile, int32_t M, int32_t N, int32_t K,
                                      const void* d_A, const int32_t* d_offs, int32_t B, int32_t L,
                                      const uint16_t* d_W, const float* d_bias, const float* d_gain,
                                      void* d_C, void* stream) {
  static const GemmBF16Kind kinds[7] = {kBF16toF32, kBF16toBF16, kNormF32toBF16, kBF16ResidF32,
                                        kInputF32toF32, kF32toF32, kF32ResidF32};
  if (kind < 0 || kind > 6) return fail(TCL_ERR_INVALID_ARG, "kind must be 0..6 (got %d)", kind);
  if (tile < -1 || tile >= kNumGemmBF16Tiles) return fail(TCL_ERR_INVALID_ARG, "tile must be -1..%d", kNumGemmBF16Tiles - 1);
  const bool f32a = kind == 2 || kind == 4 || kind == 5 || kind == 6;
  if (kind == 4) {
    if (B <= 0 || L <= 0 || !d_offs) return fail(TCL_ERR_INVALID_ARG, "gather needs d_offs, B > 0, L > 0");
    M = B * L;
  }
  if (M <= 0 || N <= 0 || K <= 0 || N % 4) return fail(TCL_ERR_INVALID_ARG, "bad M/N/K (N %% 4 == 0 required)");
  if (K % (f32a ? 4 : 8)) return fail(TCL_ERR_INVALID_ARG, "K must be a multiple of %d", f32a ? 4 : 8);
  if (!d_A || !d_W || !d_C) return fail(TCL_ERR_INVALID_ARG, "NULL device pointer");
  if (kind == 2 && !d_gain) return fail(TCL_ERR_INVALID_ARG, "kind 2 needs d_gain");
  if (kind == 4 && !d_bias) return fail(TCL_ERR_INVALID_ARG, "kind 4 needs d_bias");
  if (reinterpret_cast<uintptr_t>(d_A) % 16 || reinterpret_cast<uintptr_t>(d_W) % 16 ||
      reinterpret_cast<uintptr_t>(d_C) % 16 || (d_gain && reinterpret_cast<uintptr_t>(d_gain) % 16))
    return fail(TCL_ERR_INVALID_ARG, "A, W, C and gain must be 16-byte aligned");
  GemmArgsBF16 g;
  g.A = d_A; g.lda = K; g.W = d_W; g.ldw = (K + 7) & ~7; g.bias = d_bias; g.gain = d_gain;
  g.C = d_C; g.ldc = N; g.Mmax = M; g.N = N; g.K = K; g.eps = 1e-5f;
  if (kind == 4) { g.offs = d_offs; g.B = B; g.L = L; g.Mdev = d_offs + B; }
  GemmBF16Kind k = kinds[kind];
  if (k == kBF16toF32 && d_bias) k = kBF16toF32Bias;
  TCL_HIP(launch_gemm_bf16(g, k, tile, static_cast<hipStream_t>(stream)));
  return TCL_OK;
}

TCL_API tcl_status tcl_test_offsets(int32_t B, int32_t L, const int32_t* d_lengths, int32_t* d_offs,
                                    int32_t* d_ord, void* stream) {
  if (B <= 0 || L <= 0) return fail(TCL_ERR_INVALID_ARG, "B and L must be positive (B=%d L=%d)", B, L);
  if (!d_lengths || !d_offs) return fail(TCL_ERR_INVALID_ARG, "NULL device pointer");
  TCL_HIP(launch_offsets(d_lengths, B, L, d_offs, static_cast<hipStream_t>(stream), d_ord));
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

TCL_API tcl_status tcl_test_xproj_conv_f32(int32_t B, int32_t rows, int32_t E, int32_t N,
                                           const int32_t* d_offs, const float* d_x, int32_t ldx,
                                           const float* d_w, const float* d_b, const float* d_W,
                                           uint16_t* d_Wsplit, uint8_t* d_tpos, float* d_u,
                                           float* d_xdbl, void* stream) {
  if (B <= 0 || rows <= 0 || E <= 0 || N <= 0 || ldx < E) return fail(TCL_ERR_INVALID_ARG, "bad sizes");
  if (!d_offs || !d_x || !d_w || !d_b || !d_W || !d_Wsplit || !d_tpos || !d_u || !d_xdbl)
    return fail(TCL_ERR_INVALID_ARG, "NULL device pointer");
  GemmArgs g;
  g.A = d_u; g.lda = E; g.W = d_W; g.ldw = E; g.C = d_xdbl; g.ldc = N;
  g.Mdev = d_offs + B; g.Mmax = rows; g.N = N; g.K = E;
  ConvIn cv;
  cv.x = d_x; cv.ldx = ldx; cv.w = d_w; cv.b = d_b; cv.tpos = d_tpos; cv.u = d_u;
  if (!gemm_split_conv_supports(g, cv, 4))
    return fail(TCL_ERR_UNSUPPORTED, "shape or alignment not supported by the fused conv + x_proj kernel");
  const hipStream_t s = static_cast<hipStream_t>(stream);
  TCL_HIP(launch_split_weights(d_W, N, E, E, d_Wsplit, s));
  TCL_HIP(launch_token_pos(d_offs, B, d_tpos, s));
  TCL_HIP(launch_gemm_split_conv(g, cv, d_Wsplit, E, s));
  return TCL_OK;
}

TCL_API tcl_status tcl_test_xproj_conv_bf16(int32_t B, int32_t rows, int32_t E, int32_t N,
                                            const int32_t* d_offs, const uint16_t* d_x, int32_t ldx,
                                            const float* d_w, const float* d_b, const uint16_t* d_W,
                                            uint8_t* d_tpos, uint16_t* d_u, float* d_xdbl, void* stream) {
  if (B <= 0 || rows <= 0 || E <= 0 || N <= 0 || ldx < E) return fail(TCL_ERR_INVALID_ARG, "bad sizes");
  if (!d_offs || !d_x || !d_w || !d_b || !d_W || !d_tpos || !d_u || !d_xdbl)
    return fail(TCL_ERR_INVALID_ARG, "NULL device pointer");
  ConvArgsBF16 a;
  a.x = d_x; a.ldx = ldx; a.w = d_w; a.b = d_b; a.tpos = d_tpos; a.u = d_u; a.W = d_W; a.ldw = E;
  a.C = d_xdbl; a.ldc = N; a.Mdev = d_offs + B; a.Mmax = rows; a.N = N; a.E = E;
  if (!gemm_bf16_conv_supports(a, 4))
    return fail(TCL_ERR_UNSUPPORTED, "shape or alignment not supported by the fused bf16 conv + x_proj kernel");
  const hipStream_t s = static_cast<hipStream_t>(stream);
  TCL_HIP(launch_token_pos(d_offs, B, d_tpos, s));
  TCL_HIP(launch_gemm_bf16_conv(a, s));
  return TCL_OK;
}

TCL_API tcl_status tcl_test_scan_f32(int32_t B, int32_t E, int32_t N, int32_t R, int32_t chunks,
                                     const int32_t* d_offs, const float* d_u, const float* d_xdbl,
                                     const float* d_z, int32_t ldz, const float* d_W_dt,
                                     const float* d_b_dt, const float* d_A_log, const float* d_D,
                                     float* d_out, void* stream) {
  if (B <= 0 || E <= 0 || ldz < E) return fail(TCL_ERR_INVALID_ARG, "bad sizes");
  if (chunks < 0 || chunks > 8) return fail(TCL_ERR_INVALID_ARG, "chunks must be in [0, 8]");
  if (N != 16) return fail(TCL_ERR_UNSUPPORTED, "d_state must be 16");
  if (R % 4 || R <= 0 || R > 32) return fail(TCL_ERR_UNSUPPORTED, "dt_rank must be 4..32, step 4");
  if (!d_offs || !d_u || !d_xdbl || !d_z || !d_W_dt || !d_b_dt || !d_A_log || !d_D || !d_out)
    return fail(TCL_ERR_INVALID_ARG, "NULL device pointer");
  if (chunks > 0)
    TCL_HIP(launch_scan_chunked<float>(B, E, N, R, chunks, d_offs, d_u, d_xdbl, d_z, ldz, d_W_dt,
                                       d_b_dt, d_A_log, d_D, d_out, static_cast<hipStream_t>(stream)));
  else
    TCL_HIP(launch_scan<float>(B, E, N, R, d_offs, d_u, d_xdbl, d_z, ldz, d_W_dt, d_b_dt, d_A_log,
                               d_D, d_out, static_cast<hipStream_t>(stream)));
  return TCL_OK;
}
