// The teacher -> student distillation step (tcl_trainer_*, tcl_distill_step).
//
// One step: the frozen teacher scores the batch; the student runs its
// forward pass keeping what the backward needs; the loss
// L = mean (s - t)^2 + mean (s - y)^2 is differentiated through the head,
// the pool, the final norm and every Mamba block (projections on the fp32
// matrix cores, the selective scan with recomputed states, the conv, the
// norms); per-block partial sums are reduced in a fixed order into one
// gradient blob; Adam updates the fp32 master weights; and the student's
// compute layouts (bf16 and fp32 copies) are re-derived from the master.
// Everything is enqueued on the caller's stream.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstring>

#include "model.h"

using namespace tcl;

struct tcl_trainer {
  tcl_model* teacher = nullptr;
  tcl_model* student = nullptr;
  float lr = 1e-3f, beta1 = 0.9f, beta2 = 0.999f, eps = 1e-8f;
  int64_t* d_step = nullptr;  // steps taken (device): Adam's bias correction
  int max_B = 0, max_L = 0;
  void* dev = nullptr;  // gradient blob, Adam moments, reduction table
  float *grad = nullptr, *m = nullptr, *v = nullptr;
  ReduceJob* d_jobs = nullptr;
  int max_jobs = 0;
  int njobs = 0;
  // the jobs in groups, one per block: group l (its first job, count and
  // largest output) is reduced once block l's partial sums are written
  std::vector<int> grp_first, grp_count, grp_blocks;
  int plan_B = -1, plan_L = -1;
  Timing timing;
  // the backward's weight-gradient GEMMs run on a stream of their own,
  // forked from and joined back to the step's stream by events
  hipStream_t side = nullptr;
  hipEvent_t ev_fork = nullptr, ev_dh = nullptr, ev_layer = nullptr, ev_end = nullptr;
};

namespace {

// Workspace layout of one step (byte offsets, 256-aligned).
struct TrainPlan {
  size_t teacher_ws = 0, t_scores = 0, s_scores = 0, offs = 0;
  size_t prow = 0;  // per packed token: its row of the padded feature tensor
  size_t ord = 0;   // the programs longest first
  struct Layer {
    size_t Hin, n, rstd, xz, u, xdbl, y, yg, ckpt;
    size_t p_Wout, p_Wdt, p_bdt, p_A, p_D, p_Wx, p_conv, p_Win, p_g;
    int s_Wout, s_Wdt, s_Wx, s_Win;
  };
  std::vector<Layer> layers;
  size_t H_last = 0, pooled = 0, a1 = 0;
  size_t dH = 0, dyg = 0, dxz = 0, du = 0, dv = 0, dxdbl = 0, dbc_part = 0, dN = 0, da1 = 0, dpooled = 0;
  size_t p_lh = 0, p_W1 = 0, p_gf = 0, p_W0 = 0, p_b0 = 0;
  size_t rank_ws = 0, ds = 0, rloss = 0, ewc_part = 0;  // ranking objective (tcl_distill_step_kd)
  int s_W1 = 0, s_W0 = 0, cs = 0, lh_blocks = 0, rn_blocks = 0;
  size_t total = 0;
};

TrainPlan plan_step(const tcl_trainer* tr, int B, int L) {
  const tcl_config& c = tr->student->cfg;
  TrainPlan P;
  const size_t rows = (size_t)B * L;
  const int d = c.d_model, E = c.d_inner, N = c.d_state, K = c.d_conv, R = c.dt_rank, XW = R + 2 * N;
  const int h = c.head_hidden, F = c.F, Mmax = B * L;
  size_t o = 0;
  auto take = [&](size_t bytes) {
    const size_t at = o;
    o = align256(o + bytes);
    return at;
  };
  P.teacher_ws = take(score_plan(tr->teacher->cfg, B, L).total);
  P.t_scores = take((size_t)B * 4);
  P.s_scores = take((size_t)B * 4);
  P.offs = take((size_t)(B + 1) * 4);
  P.ord = take((size_t)B * 4);
  P.prow = take((size_t)B * L * 4);
  P.cs = colsum_splits(Mmax);
  P.lh_blocks = loss_head_blocks(B);
  P.rn_blocks = rmsnorm_bwd_blocks(Mmax);
  for (int l = 0; l < c.n_layers; ++l) {
    TrainPlan::Layer Ly{};
    Ly.Hin = take(rows * d * 4);
    Ly.n = take(rows * d * 2);
    Ly.rstd = take(rows * 4);
    Ly.xz = take(rows * 2 * E * 2);
    Ly.u = take(rows * E * 2);
    Ly.xdbl = take(rows * XW * 4);
    Ly.y = take(rows * E * 2);
    Ly.yg = take(rows * E * 2);
    Ly.ckpt = take(scan_bwd_ckpt_floats(B, E, L, N) * 4);
    Ly.s_Wout = gemm_tn_splits(Mmax, d, E);
    Ly.s_Wdt = gemm_tn_splits(Mmax, E, R);
    Ly.s_Wx = gemm_tn_splits(Mmax, XW, E);
    Ly.s_Win = gemm_tn_splits(Mmax, 2 * E, d);
    Ly.p_Wout = take((size_t)Ly.s_Wout * d * E * 4);
    Ly.p_Wdt = take((size_t)Ly.s_Wdt * E * R * 4);
    Ly.p_bdt = take((size_t)P.cs * E * 4);
    Ly.p_A = take((size_t)B * E * N * 4);
    Ly.p_D = take((size_t)B * E * 4);
    Ly.p_Wx = take((size_t)Ly.s_Wx * XW * E * 4);
    Ly.p_conv = take((size_t)B * (K + 1) * E * 4);
    Ly.p_Win = take((size_t)Ly.s_Win * 2 * E * d * 4);
    Ly.p_g = take((size_t)P.rn_blocks * d * 4);
    P.layers.push_back(Ly);
  }
  P.H_last = take(rows * d * 4);
  P.pooled = take((size_t)B * d * 4);
  P.a1 = take((size_t)B * h * 4);
  P.dH = take(rows * d * 4);
  P.dyg = take(rows * E * 4);
  P.dxz = take(rows * 2 * E * 4);
  P.du = take(rows * E * 4);
  P.dv = take(rows * E * 4);
  P.dxdbl = take(rows * XW * 4);
  P.dbc_part = take(scan_bwd_part_floats(B, L, N) * 4);
  P.dN = take(rows * d * 4);
  P.da1 = take((size_t)B * h * 4);
  P.dpooled = take((size_t)B * d * 4);
  P.p_lh = take((size_t)P.lh_blocks * (2 * h + 4) * 4);
  P.s_W1 = gemm_tn_splits(B, h, d);
  P.p_W1 = take((size_t)P.s_W1 * h * d * 4);
  P.p_gf = take((size_t)B * d * 4);
  P.s_W0 = gemm_tn_splits(Mmax, d, F);
  P.p_W0 = take((size_t)P.s_W0 * d * F * 4);
  P.p_b0 = take((size_t)P.cs * d * 4);
  P.rank_ws = take(rank_workspace_floats(B, 2) * 4);
  P.ds = take((size_t)B * 4);
  P.rloss = take(4 * 4);
  P.ewc_part = take((size_t)ewc_part_floats() * 4);
  P.total = o;
  return P;
}

// The reductions that turn the step's partial sums into the gradient blob
// (canonical layout) and the three loss values.
// Jobs in the order the backward pass finishes their partial sums: the head,
// then the blocks from the last to the first, then the input layer. Group l
// is block l's jobs, with the head's in the last block's group and the input
// layer's in block 0's; first[l] and count[l] locate it.
std::vector<ReduceJob> reduce_jobs(const tcl_trainer* tr, const TrainPlan& P, int B, std::vector<int>& first,
                                   std::vector<int>& count) {
  const tcl_config& c = tr->student->cfg;
  const BlobLayout bl = blob_layout(c);
  const int64_t d = c.d_model, E = c.d_inner, N = c.d_state, K = c.d_conv, R = c.dt_rank;
  const int64_t XW = R + 2 * N, h = c.head_hidden, F = c.F;
  std::vector<ReduceJob> J;
  auto add = [&](size_t src_bytes, int64_t split_stride, int64_t src_stride, int nsplit, int dst_buf,
                 int64_t dst, int64_t dst_stride, int64_t n) {
    ReduceJob r{};
    r.src = (int64_t)(src_bytes / 4);
    r.split_stride = split_stride;
    r.src_stride = src_stride;
    r.nsplit = nsplit;
    r.dst_buf = dst_buf;
    r.dst = dst;
    r.dst_stride = dst_stride;
    r.n = n;
    J.push_back(r);
  };
  const int64_t lw = 2 * h + 4;
  add(P.p_lh, lw, 1, P.lh_blocks, 0, bl.W2, 1, h);                 // dW2
  add(P.p_lh + h * 4, lw, 1, P.lh_blocks, 0, bl.b1, 1, h);         // db1
  add(P.p_lh + 2 * h * 4, lw, 1, P.lh_blocks, 0, bl.b2, 1, 1);     // db2
  add(P.p_lh + (2 * h + 3) * 4, lw, 1, P.lh_blocks, 1, 0, 1, 1);   // loss total
  add(P.p_lh + (2 * h + 1) * 4, lw, 1, P.lh_blocks, 1, 1, 1, 1);   // mse(s, teacher)
  add(P.p_lh + (2 * h + 2) * 4, lw, 1, P.lh_blocks, 1, 2, 1, 1);   // mse(s, label)
  add(P.p_W1, h * d, 1, P.s_W1, 0, bl.W1, 1, h * d);               // dW1
  add(P.p_gf, d, 1, B, 0, bl.g_f, 1, d);                           // dg_f
  const int nl = c.n_layers;
  first.assign(nl, 0);
  count.assign(nl, 0);
  for (int l = nl - 1; l >= 0; --l) {
    const auto& Ly = P.layers[l];
    const auto& Bl = bl.layers[l];
    first[l] = l == nl - 1 ? 0 : (int)J.size();
    add(Ly.p_Wout, d * E, 1, Ly.s_Wout, 0, Bl.W_out, 1, d * E);
    add(Ly.p_Wdt, E * R, 1, Ly.s_Wdt, 0, Bl.W_dt, 1, E * R);
    add(Ly.p_bdt, E, 1, P.cs, 0, Bl.b_dt, 1, E);
    add(Ly.p_A, E * N, 1, B, 0, Bl.A_log, 1, E * N);
    add(Ly.p_D, E, 1, B, 0, Bl.D, 1, E);
    add(Ly.p_Wx, XW * E, 1, Ly.s_Wx, 0, Bl.W_x, 1, XW * E);
    for (int k = 0; k < K; ++k) add(Ly.p_conv + (size_t)k * E * 4, (K + 1) * E, 1, B, 0, Bl.conv_w + k, K, E);
    add(Ly.p_conv + (size_t)K * E * 4, (K + 1) * E, 1, B, 0, Bl.conv_b, 1, E);
    add(Ly.p_Win, 2 * E * d, 1, Ly.s_Win, 0, Bl.W_in, 1, 2 * E * d);
    add(Ly.p_g, d, 1, P.rn_blocks, 0, Bl.g, 1, d);
    count[l] = (int)J.size() - first[l];
  }
  add(P.p_W0, d * F, 1, P.s_W0, 0, bl.W0, 1, d * F);
  add(P.p_b0, d, 1, P.cs, 0, bl.b0, 1, d);
  count[0] = (int)J.size() - first[0];
  return J;
}

tcl_status ensure_plan(tcl_trainer* tr, int B, int L, const TrainPlan& P, bool capturing) {
  if (tr->plan_B == B && tr->plan_L == L) return TCL_OK;
  if (capturing)
    return fail(TCL_ERR_INVALID_ARG, "a step with a new (B, L) = (%d, %d) cannot be captured: run one "
                "step of that shape first", B, L);
  std::vector<int> first, count;
  std::vector<ReduceJob> J = reduce_jobs(tr, P, B, first, count);
  std::vector<int> blocks(first.size());
  for (size_t g = 0; g < first.size(); ++g) blocks[g] = reduce_blocks(J.data() + first[g], count[g]);
  if ((int)J.size() > tr->max_jobs) return fail(TCL_ERR_UNSUPPORTED, "too many reduction jobs");
  // the table changes only with the batch shape; the copy waits for
  // earlier steps that may still read the previous table
  TCL_HIP(hipDeviceSynchronize());
  TCL_HIP(hipMemcpy(tr->d_jobs, J.data(), J.size() * sizeof(ReduceJob), hipMemcpyHostToDevice));
  tr->njobs = (int)J.size();
  tr->grp_first = first;
  tr->grp_count = count;
  tr->grp_blocks = blocks;
  tr->plan_B = B;
  tr->plan_L = L;
  return TCL_OK;
}

}  // namespace

namespace {
void release_side(tcl_trainer* tr) {
  for (hipEvent_t* e : {&tr->ev_fork, &tr->ev_dh, &tr->ev_layer, &tr->ev_end})
    if (*e) {
      (void)hipEventDestroy(*e);
      *e = nullptr;
    }
  if (tr->side) {
    (void)hipStreamSynchronize(tr->side);
    (void)hipStreamDestroy(tr->side);
    tr->side = nullptr;
  }
}
}  // namespace

TCL_API tcl_status tcl_trainer_create(tcl_model* teacher, tcl_model* student, float lr, float beta1,
                                      float beta2, float eps, int32_t max_B, int32_t max_L,
                                      tcl_trainer** out) {
  if (!out) return fail(TCL_ERR_INVALID_ARG, "out is NULL");
  *out = nullptr;
  if (!teacher || !student) return fail(TCL_ERR_INVALID_ARG, "teacher and student are required");
  if (teacher == student) return fail(TCL_ERR_INVALID_ARG, "teacher and student must differ");
  if (!(lr > 0.f) || !(beta1 >= 0.f && beta1 < 1.f) || !(beta2 >= 0.f && beta2 < 1.f) || !(eps > 0.f))
    return fail(TCL_ERR_INVALID_ARG, "bad Adam hyper-parameters");
  if (max_B <= 0 || max_L <= 0) return fail(TCL_ERR_INVALID_ARG, "max_B and max_L must be positive");
  const tcl_config& sc = student->cfg;
  const tcl_config& tc = teacher->cfg;
  if (sc.dtype != TCL_BF16) return fail(TCL_ERR_UNSUPPORTED, "the student must be a bf16 model");
  if (sc.F != tc.F) return fail(TCL_ERR_INVALID_ARG, "teacher and student feature widths differ");
  if (sc.d_inner > 256) return fail(TCL_ERR_UNSUPPORTED, "student d_inner must be <= 256");
  if (sc.d_state != 16 || sc.F % 4 || sc.enc_hidden[0] != 0 || sc.dec_hidden2 != 0)
    return fail(TCL_ERR_UNSUPPORTED,
                "the student must have d_state 16, F %% 4 == 0, a one-Linear encoder and a two-layer decoder");
  if (sc.dt_rank != 4 && sc.dt_rank != 8 && sc.dt_rank != 16)
    return fail(TCL_ERR_UNSUPPORTED, "student dt_rank must be 4, 8 or 16");
  tcl_trainer* tr = new tcl_trainer();
  tr->teacher = teacher;
  tr->student = student;
  tr->lr = lr;
  tr->beta1 = beta1;
  tr->beta2 = beta2;
  tr->eps = eps;
  tr->max_B = max_B;
  tr->max_L = max_L;
  tr->max_jobs = 64 + 16 * sc.n_layers;
  const size_t n = student->n_params;
  const size_t bytes = align256(n * 4) * 3 + align256((size_t)tr->max_jobs * sizeof(ReduceJob)) + 256;
  if (hipMalloc(&tr->dev, bytes) != hipSuccess) {
    delete tr;
    return fail(TCL_ERR_OOM, "hipMalloc of %zu bytes for the trainer failed", bytes);
  }
  char* base = static_cast<char*>(tr->dev);
  tr->grad = reinterpret_cast<float*>(base);
  tr->m = reinterpret_cast<float*>(base + align256(n * 4));
  tr->v = reinterpret_cast<float*>(base + 2 * align256(n * 4));
  tr->d_jobs = reinterpret_cast<ReduceJob*>(base + 3 * align256(n * 4));
  tr->d_step = reinterpret_cast<int64_t*>(base + 3 * align256(n * 4) +
                                          align256((size_t)tr->max_jobs * sizeof(ReduceJob)));
  if (hipMemset(tr->dev, 0, bytes) != hipSuccess) {
    (void)hipFree(tr->dev);
    delete tr;
    return fail(TCL_ERR_HIP, "hipMemset failed");
  }
  // default priority; without them the backward runs on one stream
  bool ok = hipStreamCreateWithFlags(&tr->side, hipStreamNonBlocking) == hipSuccess;
  for (hipEvent_t* e : {&tr->ev_fork, &tr->ev_dh, &tr->ev_layer, &tr->ev_end})
    ok = ok && hipEventCreateWithFlags(e, hipEventDisableTiming) == hipSuccess;
  if (!ok) {
    release_side(tr);
    (void)hipGetLastError();
  }
  *out = tr;
  return TCL_OK;
}

TCL_API tcl_status tcl_trainer_destroy(tcl_trainer* tr) {
  if (!tr) return TCL_OK;
  release_side(tr);
  tr->timing.release();
  if (tr->dev) (void)hipFree(tr->dev);
  delete tr;
  return TCL_OK;
}

TCL_API size_t tcl_distill_workspace_bytes(const tcl_trainer* tr, int32_t B, int32_t L) {
  if (!tr || B <= 0 || L <= 0 || B > tr->max_B || L > tr->max_L) return 0;
  return plan_step(tr, B, L).total;
}

TCL_API tcl_status tcl_trainer_get_grads(const tcl_trainer* tr, float* h_out, size_t n) {
  if (!tr || !h_out) return fail(TCL_ERR_INVALID_ARG, "NULL argument");
  if (n != tr->student->n_params) return fail(TCL_ERR_INVALID_ARG, "size mismatch");
  TCL_HIP(hipDeviceSynchronize());
  TCL_HIP(hipMemcpy(h_out, tr->grad, n * 4, hipMemcpyDeviceToHost));
  return TCL_OK;
}

namespace {

// One step on either objective: kd == NULL is the two-MSE loss, else the
// ranking objective of Eq. (9).
// rank_keys (may be null): what the student's score ranks are counted from
// instead of its own scores; scores_out (may be null): [2B] receives the
// student's then the teacher's scores of the step.
tcl_status distill_step(tcl_trainer* tr, int32_t B, int32_t L, const float* d_feats, const int32_t* d_lengths,
                        const float* d_labels, const tcl_kd_loss* kd, float* d_loss, void* d_ws,
                        size_t ws_bytes, void* stream, const float* rank_keys = nullptr,
                        float* scores_out = nullptr) {
  if (!tr) return fail(TCL_ERR_INVALID_ARG, "trainer is NULL");
  if (B <= 0 || L <= 0 || B > tr->max_B || L > tr->max_L)
    return fail(TCL_ERR_INVALID_ARG, "B=%d L=%d outside [1, max_B=%d] x [1, max_L=%d]", B, L,
                tr->max_B, tr->max_L);
  if (!d_feats || !d_lengths || !d_labels || !d_loss || !d_ws)
    return fail(TCL_ERR_INVALID_ARG, "NULL device pointer");
  if (reinterpret_cast<uintptr_t>(d_feats) % 16 || reinterpret_cast<uintptr_t>(d_ws) % 256)
    return fail(TCL_ERR_INVALID_ARG, "d_feats must be 16-byte and d_workspace 256-byte aligned");
  const TrainPlan P = plan_step(tr, B, L);
  if (ws_bytes < P.total)
    return fail(TCL_ERR_WORKSPACE, "workspace has %zu bytes, needs %zu", ws_bytes, P.total);
  hipStream_t s = static_cast<hipStream_t>(stream);
  // a step may be captured into a graph on `stream` once its shape has run
  hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
  TCL_HIP(hipStreamIsCapturing(s, &cap));
  const bool capturing = cap != hipStreamCaptureStatusNone;
  if (capturing && (tr->timing.on || tr->teacher->timing.on))
    return fail(TCL_ERR_INVALID_ARG, "per-kernel timing is on: a timed step cannot be captured");
  tcl_status st = ensure_plan(tr, B, L, P, capturing);
  if (st != TCL_OK) return st;

  char* ws = static_cast<char*>(d_ws);
  auto F32 = [&](size_t off) { return reinterpret_cast<float*>(ws + off); };
  auto B16 = [&](size_t off) { return reinterpret_cast<uint16_t*>(ws + off); };
  tcl_model* S = tr->student;
  const tcl_config& c = S->cfg;
  const int d = c.d_model, E = c.d_inner, N = c.d_state, K = c.d_conv, R = c.dt_rank, XW = R + 2 * N;
  const int h = c.head_hidden, F = c.F, Mmax = B * L;
  int* offs = reinterpret_cast<int*>(ws + P.offs);
  const int* Mdev = offs + B;
  Timing& T = tr->timing;

  // 1. frozen teacher, on the teacher model's first stream where it has one:
  // it shares nothing with the student's forward but the inputs, so the two
  // forwards run side by side until the loss needs the teacher's scores
  tcl_model* Tm = tr->teacher;
  const bool fork = Tm->aux[0] && Tm->ev[0] && Tm->ev[1];
  if (fork) {
    TCL_HIP(hipEventRecord(Tm->ev[0], s));
    TCL_HIP(hipStreamWaitEvent(Tm->aux[0], Tm->ev[0], 0));
  }
  // the teacher's parts (front, blocks, tail) are enqueued between the
  // student's layers, so that neither forward waits for the host to finish
  // enqueueing the other
  const int t_parts = Tm->cfg.n_layers + 2;
  int t_next = 0;
  auto teacher_parts = [&](int upto) -> tcl_status {
    for (; t_next < upto && t_next < t_parts; ++t_next) {
      const tcl_status ts = run_score_part(Tm, B, L, d_feats, d_lengths, F32(P.t_scores), ws + P.teacher_ws,
                                           fork ? Tm->aux[0] : s, t_next);
      if (ts != TCL_OK) return ts;
    }
    return TCL_OK;
  };
  st = teacher_parts(1);
  if (st != TCL_OK) return st;

  // 2. student forward, keeping activations
  const int* ord = L <= kOrderMaxL ? reinterpret_cast<const int*>(ws + P.ord) : nullptr;
  TCL_LAUNCH(T, "offsets", launch_offsets(d_lengths, B, L, offs, s, reinterpret_cast<int*>(ws + P.ord)));
  TCL_LAUNCH(T, "packed_rows", launch_packed_rows(offs, B, L, reinterpret_cast<int*>(ws + P.prow), s));
  {
    GemmArgsBF16 g;
    g.A = d_feats; g.lda = F; g.offs = offs; g.B = B; g.L = L;
    g.W = S->W0_h; g.ldw = S->ldw0_h; g.bias = S->b0; g.C = F32(P.layers[0].Hin); g.ldc = d;
    g.Mdev = Mdev; g.Mmax = Mmax; g.N = d; g.K = F;
    TCL_LAUNCH(T, "gemm_input", launch_gemm_bf16(g, kInputF32toF32, -1, s));
  }
  for (int l = 0; l < c.n_layers; ++l) {
    st = teacher_parts(l + 2);
    if (st != TCL_OK) return st;
    const auto& W = S->layers[l];
    const auto& Ly = P.layers[l];
    float* Hout = l + 1 < c.n_layers ? F32(P.layers[l + 1].Hin) : F32(P.H_last);
    TCL_LAUNCH(T, "rmsnorm", launch_rmsnorm_fwd(d, Mmax, Mdev, F32(Ly.Hin), W.g, c.norm_eps, B16(Ly.n),
                                                F32(Ly.rstd), s));
    GemmArgsBF16 gi;
    gi.A = B16(Ly.n); gi.lda = d; gi.W = W.W_in_h; gi.ldw = d; gi.C = B16(Ly.xz); gi.ldc = 2 * E;
    gi.Mdev = Mdev; gi.Mmax = Mmax; gi.N = 2 * E; gi.K = d;
    TCL_LAUNCH(T, "gemm_in_proj", launch_gemm_bf16(gi, kBF16toBF16, -1, s));
    TCL_LAUNCH(T, "conv_silu", launch_conv_silu<uint16_t>(B, E, K, offs, B16(Ly.xz), 2 * E, W.conv_w,
                                                          W.conv_b, B16(Ly.u), s));
    GemmArgsBF16 gx;
    gx.A = B16(Ly.u); gx.lda = E; gx.W = W.W_x_h; gx.ldw = E; gx.C = F32(Ly.xdbl); gx.ldc = XW;
    gx.Mdev = Mdev; gx.Mmax = Mmax; gx.N = XW; gx.K = E;
    TCL_LAUNCH(T, "gemm_x_proj", launch_gemm_bf16(gx, kBF16toF32, -1, s));
    TCL_LAUNCH(T, "scan", launch_scan<uint16_t>(B, E, N, R, offs, B16(Ly.u), F32(Ly.xdbl),
                                                B16(Ly.xz) + E, 2 * E, W.W_dt, W.b_dt, W.A_log, W.D,
                                                B16(Ly.yg), s, B16(Ly.y), F32(Ly.ckpt), L, ord));
    GemmArgsBF16 go;
    go.A = B16(Ly.yg); go.lda = E; go.W = W.W_out_h; go.ldw = E; go.C = Hout; go.ldc = d;
    go.R = F32(Ly.Hin); go.Mdev = Mdev; go.Mmax = Mmax; go.N = d; go.K = E;
    TCL_LAUNCH(T, "gemm_out_proj", launch_gemm_bf16(go, kBF16ResidF32, -1, s));
  }
  st = teacher_parts(t_parts);
  if (st != TCL_OK) return st;
  if (fork) TCL_HIP(hipEventRecord(Tm->ev[1], Tm->aux[0]));
  TCL_LAUNCH(T, "tail", launch_tail_f32(B, L, d, h, offs, d_lengths, F32(P.H_last), S->g_f, c.final_norm,
                                        c.norm_eps, S->W1T, S->b1, S->W2, S->b2, F32(P.s_scores), s,
                                        F32(P.pooled), F32(P.a1)));

  // 3. loss, head, pool and final norm (the teacher's scores are needed from here)
  if (fork) TCL_HIP(hipStreamWaitEvent(s, Tm->ev[1], 0));
  if (kd) {
    // beta L(s; labels) + (1 - beta) phi L(s; teacher): dL/ds and the loss
    // the gate phi is a host value, or a device value (e.g. an entry of
    // tcl_teacher_gate's output) that scales (1 - beta) inside the kernels
    const float w1 = kd->d_phi ? 1.0f - kd->beta : (1.0f - kd->beta) * kd->phi;
    TCL_LAUNCH(T, "lambdarank", launch_lambdarank(B, 2, F32(P.s_scores), d_labels, F32(P.t_scores), kd->sigma,
                                                  kd->beta, w1, F32(P.rank_ws), F32(P.ds), F32(P.rloss), s,
                                                  rank_keys, kd->d_phi));
  }
  TCL_LAUNCH(T, "loss_head_bwd", launch_loss_head_bwd(B, d, h, F32(P.s_scores), F32(P.t_scores), d_labels,
                                                      F32(P.a1), S->W1, S->W2, F32(P.da1),
                                                      F32(P.dpooled), F32(P.p_lh), s,
                                                      kd ? F32(P.ds) : nullptr, kd ? F32(P.rloss) : nullptr));
  {
    GemmTNArgs a;
    a.A = F32(P.da1); a.lda = h; a.Bm = F32(P.pooled); a.ldb = d; a.P = F32(P.p_W1);
    a.Mmax = B; a.NI = h; a.NJ = d;
    TCL_LAUNCH(T, "gemm_dW", launch_gemm_tn(a, kTN_F32_F32, P.s_W1, s));
  }
  TCL_LAUNCH(T, "normf_pool_bwd", launch_normf_pool_bwd(B, d, offs, F32(P.H_last), S->g_f, c.final_norm,
                                                        c.norm_eps, F32(P.dpooled), F32(P.dH),
                                                        F32(P.p_gf), s));

  // 4. blocks in reverse. The data gradients form the chain on `s`; the
  // weight gradients (which feed only the final reduction) run on the
  // trainer's side stream beside it, each forked once its inputs are
  // ready. Joins guard the buffers the chain overwrites while a side GEMM
  // may still read them: dH (rewritten by this block's RMSNorm backward)
  // and dv, dxdbl, dxz (rewritten by the next block's scan backward).
  const hipStream_t sd = tr->side ? tr->side : s;
  auto fork_side = [&]() -> tcl_status {
    if (sd != s) {
      TCL_HIP(hipEventRecord(tr->ev_fork, s));
      TCL_HIP(hipStreamWaitEvent(sd, tr->ev_fork, 0));
    }
    return TCL_OK;
  };
  auto mark = [&](hipEvent_t e) -> tcl_status {
    if (sd != s) TCL_HIP(hipEventRecord(e, sd));
    return TCL_OK;
  };
  auto join = [&](hipEvent_t e) -> tcl_status {
    if (sd != s) TCL_HIP(hipStreamWaitEvent(s, e, 0));
    return TCL_OK;
  };
#define TCL_SIDE(NAME, CALL)            \
  do {                                  \
    const hipStream_t s = sd;           \
    TCL_LAUNCH(T, NAME, CALL);          \
  } while (0)
#define TCL_TRY(X)                        \
  do {                                    \
    const tcl_status st_ = (X);           \
    if (st_ != TCL_OK) return st_;        \
  } while (0)
  // Weight-gradient GEMMs (partial sums per token split): on the bf16
  // matrix cores for a bf16 student, else on the fp32 ones.
  auto gemm_tn = [&](const GemmTNArgs& a, TNKind kind, int splits, hipStream_t st) -> hipError_t {
    return c.dtype == TCL_BF16 ? launch_gemm_tn_bf16(a, kind, splits, st) : launch_gemm_tn(a, kind, splits, st);
  };
  // Data-gradient GEMMs C (+)= A W with A an fp32 gradient: for a bf16
  // student on the bf16 matrix cores (A rounded to bf16 as it is staged, W
  // the transposed bf16 copy, fp32 accumulation), else on the fp32 ones.
  const bool bf16_dx = c.dtype == TCL_BF16;
  auto gemm_dx = [&](const float* A, int lda, const float* Wt32, const uint16_t* Wt16, int ldw, float* C,
                     int ldc, int N_, int K_, bool accumulate) -> hipError_t {
    if (bf16_dx) {
      GemmArgsBF16 g;
      g.A = A; g.lda = lda; g.W = Wt16; g.ldw = ldw; g.C = C; g.ldc = ldc;
      g.Mdev = Mdev; g.Mmax = Mmax; g.N = N_; g.K = K_;
      return launch_gemm_bf16(g, accumulate ? kF32ResidF32 : kF32toF32, -1, s);
    }
    GemmArgs g;
    g.A = A; g.lda = lda; g.W = Wt32; g.ldw = ldw; g.C = C; g.ldc = ldc;
    g.Mdev = Mdev; g.Mmax = Mmax; g.N = N_; g.K = K_;
    return launch_gemm_f32(g, accumulate ? kResid : 0, -1, s);
  };
  for (int l = c.n_layers - 1; l >= 0; --l) {
    const auto& W = S->layers[l];
    const auto& Ly = P.layers[l];
    // dyg = dH W_out
    TCL_LAUNCH(T, "gemm_dX", gemm_dx(F32(P.dH), d, W.W_outT, W.W_outT_h, d, F32(P.dyg), E, E, d, false));
    TCL_TRY(fork_side());
    {  // dW_out = dH^T yg
      GemmTNArgs a;
      a.A = F32(P.dH); a.lda = d; a.Bm = B16(Ly.yg); a.ldb = E; a.P = F32(Ly.p_Wout);
      a.Mdev = Mdev; a.Mmax = Mmax; a.NI = d; a.NJ = E;
      TCL_SIDE("gemm_dW", gemm_tn(a, kTN_F32_BF16, Ly.s_Wout, s));
    }
    TCL_TRY(mark(tr->ev_dh));
    // the block after this one has written every partial sum (its side
    // GEMMs earlier on the side stream, the rest before the fork): reduce
    // them there, beside this block's backward
    if (l + 1 < c.n_layers)
      TCL_SIDE("reduce", launch_reduce(tr->d_jobs + tr->grp_first[l + 1], tr->grp_count[l + 1],
                                       tr->grp_blocks[l + 1], reinterpret_cast<float*>(ws), tr->grad, d_loss, s));
    // the block above's side GEMMs are done with dv, dxdbl and dxz
    if (l + 1 < c.n_layers) TCL_TRY(join(tr->ev_layer));
    TCL_LAUNCH(T, "scan_bwd", launch_scan_bwd(B, E, L, N, R, offs, B16(Ly.u), F32(Ly.xdbl), B16(Ly.xz),
                                              B16(Ly.y), F32(P.dyg), W.W_dt, W.b_dt, W.A_log, W.D,
                                              F32(Ly.ckpt), F32(P.dv), F32(P.du), F32(P.dxz),
                                              F32(P.dxdbl), F32(Ly.p_A), F32(Ly.p_D), F32(P.dbc_part), s, ord));
    {  // d dt_r = dv W_dt  -> columns [0, R) of dxdbl
      GemmArgs g;
      g.A = F32(P.dv); g.lda = E; g.W = W.W_dtT; g.ldw = E; g.C = F32(P.dxdbl); g.ldc = XW;
      g.Mdev = Mdev; g.Mmax = Mmax; g.N = R; g.K = E;
      TCL_LAUNCH(T, "gemm_dX", launch_gemm_f32(g, 0, kNarrow, s));
    }
    TCL_TRY(fork_side());
    {  // dW_dt = dv^T dt_r
      GemmTNArgs a;
      a.A = F32(P.dv); a.lda = E; a.Bm = F32(Ly.xdbl); a.ldb = XW; a.P = F32(Ly.p_Wdt);
      a.Mdev = Mdev; a.Mmax = Mmax; a.NI = E; a.NJ = R;
      TCL_SIDE("gemm_dW", gemm_tn(a, kTN_F32_F32, Ly.s_Wdt, s));
    }
    TCL_SIDE("colsum", launch_colsum(Mdev, Mmax, F32(P.dv), E, E, P.cs, F32(Ly.p_bdt), s));
    // du += dxdbl W_x
    TCL_LAUNCH(T, "gemm_dX", gemm_dx(F32(P.dxdbl), XW, W.W_xT, W.W_xT_h, XW, F32(P.du), E, E, XW, true));
    TCL_TRY(fork_side());
    {  // dW_x = dxdbl^T u
      GemmTNArgs a;
      a.A = F32(P.dxdbl); a.lda = XW; a.Bm = B16(Ly.u); a.ldb = E; a.P = F32(Ly.p_Wx);
      a.Mdev = Mdev; a.Mmax = Mmax; a.NI = XW; a.NJ = E;
      TCL_SIDE("gemm_dW", gemm_tn(a, kTN_F32_BF16, Ly.s_Wx, s));
    }
    TCL_LAUNCH(T, "conv_bwd", launch_conv_bwd(B, E, K, offs, B16(Ly.xz), 2 * E, W.conv_w, W.conv_b,
                                              F32(P.du), F32(P.dxz), 2 * E, F32(Ly.p_conv), s));
    // dN = dxz W_in
    TCL_LAUNCH(T, "gemm_dX", gemm_dx(F32(P.dxz), 2 * E, W.W_inT, W.W_inT_h, 2 * E, F32(P.dN), d, d, 2 * E, false));
    TCL_TRY(fork_side());
    {  // dW_in = dxz^T n
      GemmTNArgs a;
      a.A = F32(P.dxz); a.lda = 2 * E; a.Bm = B16(Ly.n); a.ldb = d; a.P = F32(Ly.p_Win);
      a.Mdev = Mdev; a.Mmax = Mmax; a.NI = 2 * E; a.NJ = d;
      TCL_SIDE("gemm_dW", gemm_tn(a, kTN_F32_BF16, Ly.s_Win, s));
    }
    TCL_TRY(mark(tr->ev_layer));
    TCL_TRY(join(tr->ev_dh));  // dW_out is done with dH
    TCL_LAUNCH(T, "rmsnorm_bwd", launch_rmsnorm_bwd(d, Mmax, Mdev, F32(P.dN), F32(Ly.Hin), F32(Ly.rstd),
                                                    W.g, F32(P.dH), F32(Ly.p_g), s));
  }
  // the input layer's gradients on this stream (nothing else is left to
  // overlap them with), while the side stream finishes the first block's
  TCL_TRY(mark(tr->ev_end));
  {  // dW0 = dH^T X (gathered), db0 = column sums of dH
    GemmTNArgs a;
    a.A = F32(P.dH); a.lda = d; a.Bm = d_feats; a.ldb = F; a.offs = offs; a.B = B; a.L = L;
    a.rows = reinterpret_cast<const int*>(ws + P.prow);
    a.P = F32(P.p_W0); a.Mdev = Mdev; a.Mmax = Mmax; a.NI = d; a.NJ = F;
    TCL_LAUNCH(T, "gemm_dW", gemm_tn(a, kTN_F32_GatherF32, P.s_W0, s));
  }
  TCL_LAUNCH(T, "colsum", launch_colsum(Mdev, Mmax, F32(P.dH), d, d, P.cs, F32(P.p_b0), s));
  TCL_TRY(join(tr->ev_end));  // every partial sum is written
#undef TCL_TRY
#undef TCL_SIDE

  if (scores_out) {
    TCL_HIP(hipMemcpyAsync(scores_out, F32(P.s_scores), (size_t)B * 4, hipMemcpyDeviceToDevice, s));
    TCL_HIP(hipMemcpyAsync(scores_out + B, F32(P.t_scores), (size_t)B * 4, hipMemcpyDeviceToDevice, s));
  }

  // 5. reduce partials, Adam, refresh the compute layouts
  // block 0's group (with the input layer's jobs) after the rest
  TCL_LAUNCH(T, "reduce", launch_reduce(tr->d_jobs + tr->grp_first[0], tr->grp_count[0], tr->grp_blocks[0],
                                        reinterpret_cast<float*>(ws), tr->grad, d_loss, s));
  if (kd)  // EWC on the master weights: gradient and loss[3] (zero when lambda = 0)
    TCL_LAUNCH(T, "ewc", launch_ewc((int64_t)S->n_params, S->master, kd->d_theta_prev, kd->d_fisher,
                                    kd->ewc_lambda, tr->grad, F32(P.ewc_part), d_loss, s));
  // the step count lives on the device (Adam reads it, derive advances it),
  // so that a captured step replays as a fresh one
  TCL_LAUNCH(T, "adam", launch_adam((int64_t)S->n_params, S->master, tr->m, tr->v, tr->grad, tr->lr,
                                    tr->beta1, tr->beta2, tr->eps, tr->d_step, s));
  TCL_LAUNCH(T, "derive", launch_derive(S->master, S->jobs, S->njobs, S->derive_total, S->dev, 1, s,
                                        tr->d_step));
  return TCL_OK;
}

}  // namespace

TCL_API tcl_status tcl_distill_step(tcl_trainer* tr, int32_t B, int32_t L, const float* d_feats,
                                    const int32_t* d_lengths, const float* d_labels, float* d_loss,
                                    void* d_ws, size_t ws_bytes, void* stream) {
  return distill_step(tr, B, L, d_feats, d_lengths, d_labels, nullptr, d_loss, d_ws, ws_bytes, stream);
}

namespace {

tcl_status check_kd(const tcl_kd_loss* kd) {
  if (!kd) return fail(TCL_ERR_INVALID_ARG, "kd is NULL");
  if (!(kd->beta >= 0.f && kd->beta <= 1.f) || !(kd->phi >= 0.f && kd->phi <= 1.f) || !(kd->sigma > 0.f) ||
      !(kd->ewc_lambda >= 0.f))
    return fail(TCL_ERR_INVALID_ARG, "kd needs beta, phi in [0, 1], sigma > 0, ewc_lambda >= 0");
  if (kd->ewc_lambda > 0.f && (!kd->d_fisher || !kd->d_theta_prev))
    return fail(TCL_ERR_INVALID_ARG, "the EWC penalty needs d_fisher and d_theta_prev");
  return TCL_OK;
}

}  // namespace

TCL_API tcl_status tcl_distill_step_kd(tcl_trainer* tr, int32_t B, int32_t L, const float* d_feats,
                                       const int32_t* d_lengths, const float* d_labels, const tcl_kd_loss* kd,
                                       float* d_loss, void* d_ws, size_t ws_bytes, void* stream) {
  const tcl_status st = check_kd(kd);
  if (st != TCL_OK) return st;
  return distill_step(tr, B, L, d_feats, d_lengths, d_labels, kd, d_loss, d_ws, ws_bytes, stream);
}

TCL_API tcl_status tcl_test_distill_step_kd_ranked(tcl_trainer* tr, int32_t B, int32_t L, const float* d_feats,
                                                   const int32_t* d_lengths, const float* d_labels,
                                                   const tcl_kd_loss* kd, const float* d_rank_keys,
                                                   float* d_scores_out, float* d_loss, void* d_ws,
                                                   size_t ws_bytes, void* stream) {
  const tcl_status st = check_kd(kd);
  if (st != TCL_OK) return st;
  return distill_step(tr, B, L, d_feats, d_lengths, d_labels, kd, d_loss, d_ws, ws_bytes, stream, d_rank_keys,
                      d_scores_out);
}

TCL_API tcl_status tcl_teacher_gate(int32_t n, const float* d_e, float* d_phi, void* stream) {
  if (n <= 0) return fail(TCL_ERR_INVALID_ARG, "n=%d must be positive", n);
  if (!d_e || !d_phi) return fail(TCL_ERR_INVALID_ARG, "NULL device pointer");
  TCL_HIP(launch_teacher_gate(n, d_e, d_phi, static_cast<hipStream_t>(stream)));
  return TCL_OK;
}

TCL_API size_t tcl_lambdarank_workspace_bytes(int32_t B) {
  return B > 0 ? rank_workspace_floats(B, 1) * 4 : 0;
}

TCL_API tcl_status tcl_lambdarank(int32_t B, const float* d_scores, const float* d_labels, float sigma,
                                  float* d_loss, float* d_grad, void* d_ws, size_t ws_bytes, void* stream) {
  if (B <= 0 || B > (1 << 16)) return fail(TCL_ERR_INVALID_ARG, "B=%d outside [1, 65536]", B);
  if (!(sigma > 0.f)) return fail(TCL_ERR_INVALID_ARG, "sigma must be positive");
  if (!d_scores || !d_labels || !d_loss || !d_ws) return fail(TCL_ERR_INVALID_ARG, "NULL device pointer");
  if (reinterpret_cast<uintptr_t>(d_ws) % 16) return fail(TCL_ERR_INVALID_ARG, "d_workspace must be 16-byte aligned");
  if (ws_bytes < rank_workspace_floats(B, 1) * 4)
    return fail(TCL_ERR_WORKSPACE, "workspace has %zu bytes, needs %zu", ws_bytes, rank_workspace_floats(B, 1) * 4);
  TCL_HIP(launch_lambdarank(B, 1, d_scores, d_labels, nullptr, sigma, 1.0f, 0.0f, static_cast<float*>(d_ws),
                            d_grad, d_loss, static_cast<hipStream_t>(stream)));
  return TCL_OK;
}

TCL_API tcl_status tcl_trainer_timing_enable(tcl_trainer* tr, int32_t enable) {
  if (!tr) return fail(TCL_ERR_INVALID_ARG, "trainer is NULL");
  tr->timing.on = enable != 0;
  return TCL_OK;
}

TCL_API int32_t tcl_trainer_timing_count(const tcl_trainer* tr) {
  return tr ? (int32_t)tr->timing.names.size() : 0;
}

TCL_API tcl_status tcl_trainer_timing_get(tcl_trainer* tr, int32_t idx, const char** name,
                                          double* total_ms, int64_t* launches) {
  if (!tr) return fail(TCL_ERR_INVALID_ARG, "trainer is NULL");
  TCL_HIP(tr->timing.flush());
  if (idx < 0 || idx >= (int32_t)tr->timing.names.size())
    return fail(TCL_ERR_INVALID_ARG, "timing index %d out of range", idx);
  if (name) *name = tr->timing.names[idx].c_str();
  if (total_ms) *total_ms = tr->timing.total_ms[idx];
  if (launches) *launches = tr->timing.count[idx];
  return TCL_OK;
}

TCL_API tcl_status tcl_trainer_timing_reset(tcl_trainer* tr) {
  if (!tr) return fail(TCL_ERR_INVALID_ARG, "trainer is NULL");
  TCL_HIP(tr->timing.flush());
  for (auto& t : tr->timing.total_ms) t = 0.0;
  for (auto& c : tr->timing.count) c = 0;
  return TCL_OK;
}
