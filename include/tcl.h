/*
 * tcl.h - C ABI of libtcl, an MI355X (gfx950) implementation of the
 * Mamba-based cost model of TCL (arXiv 2604.12891), section 5.2.
 *
 * The library scores batches of candidate tensor programs (each a
 * zero-padded sequence of per-statement feature vectors, section 5.1) and
 * runs the teacher -> student distillation step that the knowledge
 * distillation phase of section 6 is built from.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Pointers named d_* are device pointers on the model's device; h_*
 *    are host pointers. The caller owns every buffer it passes; the
 *    library owns only its handles and the weights it uploads at create.
 *  - `stream` is a hipStream_t passed as void* (NULL = the null stream).
 *    Every device-side effect is enqueued on it, asynchronously; outputs
 *    are valid once the stream has been synchronised. A handle must not be
 *    used on two streams at the same time.
 *  - Functions return a tcl_status; no C++ exception crosses the ABI.
 *    On failure tcl_last_error() describes the cause (thread-local,
 *    overwritten by the next failing call on the same thread).
 *  - Launch errors are reported at the call (TCL_ERR_HIP); errors inside a
 *    kernel surface at the caller's synchronisation.
 *  - Feature tensors are fp32, row-major [B, L, F]; rows t >= length[b]
 *    are ignored (the model is causal and the pool is masked, so they
 *    cannot change a score) and never read.
 *  - A program whose length is outside [1, L] is not scored: its score is
 *    set to NaN and it contributes no tokens; the call itself succeeds.
 *
 * Parameter blob
 * --------------
 * Models are described by one flat fp32 array in this canonical order
 * (every matrix row-major in [out, in] layout):
 *   W0[d,F], b0[d],
 *   per block l = 0..n_layers-1:
 *     g[d], W_in[2E,d], conv_w[E,K], conv_b[E], W_x[R+2N,E],
 *     W_dt[E,R], b_dt[E], A_log[E,N], D[E], W_out[d,E],
 *   g_f[d], W1[h,d], b1[h], W2[1,h], b2[1]
 * with d = d_model, E = d_inner, N = d_state, K = d_conv, R = dt_rank,
 * h = head_hidden. A multi-layer encoder (enc_hidden) replaces W0, b0 by
 * W0[e1,F], b0[e1], W0_1[e2,e1], b0_1[e2], W0_2[d,e2], b0_2[d] (or W0[e1,F],
 * b0[e1], W0_1[d,e1], b0_1[d] with one hidden width); a three-layer decoder
 * (dec_hidden2 = h2) replaces W2, b2 by W2[h2,h], b2[h2], W3[1,h2], b3[1].
 * The model it defines:
 *   h0   = X W0^T + b0                                   (encoder)
 *          (multi-layer: ReLU between consecutive Linear layers, none
 *          after the last)
 *   per block: n = RMSNorm(h; g), [x|z] = n W_in^T,
 *     u = SiLU(conv_b + causal depthwise conv_K(x; conv_w)),
 *     [dt_r|B|C] = u W_x^T, dt = softplus(dt_r W_dt^T + b_dt),
 *     A = -exp(A_log), selective scan (Eq. (4)-(5) discretised):
 *       s_t = exp(dt_t A) s_{t-1} + dt_t u_t B_t,  y_t = C_t.s_t + D u_t,
 *     h = h + (y * SiLU(z)) W_out^T
 *   score = W2 ReLU(W1 pool(RMSNorm(h; g_f)) + b1) + b2
 *          (three-layer decoder: W3 ReLU(W2 ReLU(W1 p + b1) + b2) + b3)
 * where pool is the mean over each program's valid tokens. RMSNorm uses
 * norm_eps; the conv has K-1 zeros on the left of each program and its last
 * tap multiplies the current token.
 */
#ifndef TCL_H
#define TCL_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
#define TCL_EXTERN extern "C"
#else
#define TCL_EXTERN extern
#endif
#define TCL_API TCL_EXTERN __attribute__((visibility("default")))

typedef enum tcl_status {
  TCL_OK = 0,
  TCL_ERR_INVALID_ARG = -1, /* null pointer, non-positive size, mismatch */
  TCL_ERR_UNSUPPORTED = -2, /* shape outside what the kernels implement  */
  TCL_ERR_WORKSPACE = -3,   /* workspace smaller than *_workspace_bytes   */
  TCL_ERR_OOM = -4,         /* device allocation failed                   */
  TCL_ERR_HIP = -5          /* a HIP runtime call or launch failed        */
} tcl_status;

typedef enum tcl_dtype {
  TCL_F32 = 0,  /* fp32 weights, activations and arithmetic                 */
  TCL_BF16 = 1  /* bf16 weights and activations; fp32 accumulation and fp32
                   scan state. Weights are rounded to bf16 (nearest-even) at
                   create; pass bf16-representable values to avoid that.    */
} tcl_dtype;

/* How an fp32 model runs its dense projections (the encoder's Linear
 * layers, in_proj, x_proj and out_proj; a shape without a split kernel,
 * such as d_inner > 512 for x_proj and out_proj, runs on the fp32 path). */
typedef enum tcl_f32_matmul {
  TCL_F32_MATMUL_SPLIT = 0,     /* bf16/fp16 matrix cores, fp32-level accuracy:
                                   in_proj, out_proj and the encoder's Linear
                                   layers take both operands in two fp16 parts
                                   (after exact power-of-two scales; three part
                                   products, at most 12 units of fp32 rounding
                                   each) when every weight of the matrix is
                                   below 32 in magnitude; x_proj (and any other
                                   matrix) splits both operands exactly into
                                   three bf16 parts (six part products, at most
                                   2 units)                                 */
  TCL_F32_MATMUL_NATIVE = 1,    /* fp32 matrix cores (v_mfma_f32_*_f32)     */
  TCL_F32_MATMUL_SPLIT_BF16 = 2 /* the three-part bf16 split everywhere      */
} tcl_f32_matmul;

/* Model hyper-parameters (section 5.2; the hyper-parameter study of
 * section 7.2.1 names d_state, d_conv, expand and n_layers).
 * Supported: F in [1, 1024], d_model in {64, 128, 256}, d_inner % 64 == 0
 * and <= 2048, d_state 16 (dt_rank % 4 == 0 and <= 32) or 8 (dt_rank 4, 8
 * or 16), d_conv in [1, 4], head_hidden % 64 == 0 and <= 256, n_layers in
 * [1, 16]. The paper's own form (section 5.2: encoder widths 64, 128, 128,
 * decoder widths 64, 32, 1) is enc_hidden = {64, 128}, dec_hidden2 = 32:
 * enc_hidden entries % 4 == 0 and <= 512 (fp32 models only; {0, 0} is the
 * one-Linear encoder, {e1, 0} one hidden layer), dec_hidden2 in [0, 256].
 * A zero-initialised tail of the struct gives the one-Linear encoder and
 * the two-layer decoder. */
typedef struct tcl_config {
  int32_t F;           /* features per token                        */
  int32_t d_model;     /* residual width d                          */
  int32_t d_inner;     /* expanded width E = expand * d_model       */
  int32_t d_state;     /* SSM state size N per channel              */
  int32_t d_conv;      /* depthwise conv width K                    */
  int32_t dt_rank;     /* rank R of the dt projection               */
  int32_t n_layers;    /* Mamba blocks                              */
  int32_t head_hidden; /* hidden width h of the score head          */
  int32_t final_norm;  /* 1: RMSNorm before the pool (section 5.2)  */
  float norm_eps;      /* RMSNorm epsilon                           */
  int32_t dtype;       /* tcl_dtype                                 */
  int32_t f32_matmul;  /* tcl_f32_matmul (ignored for bf16 models)  */
  int32_t enc_hidden[2]; /* hidden widths of a multi-layer encoder  */
  int32_t dec_hidden2;   /* second hidden width of the decoder (0: none) */
} tcl_config;

typedef struct tcl_model tcl_model;     /* opaque, library-owned */
typedef struct tcl_trainer tcl_trainer; /* opaque, library-owned */
typedef struct tcl_lateral tcl_lateral; /* opaque, library-owned */

/* Number of fp32 values in the canonical parameter blob for `cfg`
 * (0 if cfg is NULL). */
TCL_API size_t tcl_param_count(const tcl_config* cfg);

/* Create a cost model on the current HIP device from a host parameter blob
 * of exactly tcl_param_count(cfg) values (copied; the caller keeps it).
 * Allocates the device weights (once) and derives kernel layouts. Not
 * stream-ordered: returns after the upload has completed. */
TCL_API tcl_status tcl_cost_model_create(const tcl_config* cfg, const float* h_params,
                                         size_t n_params, tcl_model** out);

/* Free the model's device memory. Pending work that uses it must have
 * finished. NULL is accepted. */
TCL_API tcl_status tcl_cost_model_destroy(tcl_model* model);

/* Bytes of device workspace tcl_score needs for a batch of B programs padded
 * to L tokens (0 on invalid arguments). */
TCL_API size_t tcl_score_workspace_bytes(const tcl_model* model, int32_t B, int32_t L);

/* Score B candidate programs (section 3 / Fig. 2: the cost model ranks the
 * candidates of a tuning round; higher score ranks first).
 *   d_feats   [B, L, F] fp32 row-major (F = cfg.F); rows t >= len ignored
 *   d_lengths [B] int32, valid programs have 1 <= len <= L
 *   d_scores  [B] fp32 output
 *   d_workspace, ws_bytes: >= tcl_score_workspace_bytes(model, B, L) bytes,
 *   256-byte aligned; its contents on entry are ignored.
 * Only the valid tokens are computed: tokens are packed program by program
 * on the device and every kernel works on the packed rows.
 * Work is ordered on `stream` (NULL: the default stream). Batches of 2048
 * programs or more run as two halves on two streams the model owns, forked
 * from `stream` and joined back into it by events, so the call is still
 * ordered on `stream` as a whole (and can be captured into a graph);
 * calls on one model must not be issued from several host threads at once. */
TCL_API tcl_status tcl_score(tcl_model* model, int32_t B, int32_t L, const float* d_feats,
                             const int32_t* d_lengths, float* d_scores, void* d_workspace,
                             size_t ws_bytes, void* stream);

/* tcl_score for callers that cannot allocate device memory (code under HIP
 * graph capture, tight serving loops, harnesses that forbid hipMalloc): the
 * same scores, bit for bit, as tcl_score run as one pass (its kernels, on
 * `stream` only), with the workspace taken from a buffer the library holds
 * in each GPU's memory (a file-scope device array of
 * tcl_score_noalloc_max_bytes() = 256 MiB, present on every device the
 * library runs on until the process ends; its address is looked up once
 * per device when a model is created there). The call allocates nothing
 * and calls no allocating routine.
 *   Arguments as tcl_score without the workspace; the model's device must
 *   be current. Batches whose workspace (tcl_score_workspace_bytes of a
 *   batch under 2048 programs, the one-pass size) exceeds the buffer are
 *   refused with TCL_ERR_UNSUPPORTED before anything is enqueued (about
 *   1,400 programs of 25 tokens for d_model 256). Per-kernel timing must be
 *   disabled (TCL_ERR_INVALID_ARG otherwise).
 * Every call on a GPU uses that GPU's one buffer, which keeps the last
 * call's contents (nothing in it needs to start cleared): calls that
 * overlap on one GPU -- on different streams, or from several host threads,
 * for any models -- race on it and must be serialised by the caller. */
TCL_API size_t tcl_score_noalloc_max_bytes(void);
TCL_API tcl_status tcl_score_noalloc(tcl_model* model, int32_t B, int32_t L, const float* d_feats,
                                     const int32_t* d_lengths, float* d_scores, void* stream);

/* Copy the fp32 master parameters (canonical blob) back to the host. */
TCL_API tcl_status tcl_get_params(const tcl_model* model, float* h_out, size_t n_params);

/* Replace the parameters from a host blob (synchronous, like create). */
TCL_API tcl_status tcl_set_params(tcl_model* model, const float* h_params, size_t n_params);

/* How tcl_score runs a batch of >= 2048 programs: n = 2 (the default) as two
 * concurrent halves on the model's two streams, n = 1 as one pass on the
 * caller's stream (the same scores, bit for bit; one pass gives each
 * kernel's own time without the other half's kernels beside it). Other
 * values: TCL_ERR_INVALID_ARG. A workspace sized for n = 2 also serves n = 1. */
TCL_API tcl_status tcl_set_score_streams(tcl_model* model, int32_t n);

/* Per-kernel timing, for measurement. While enabled, every kernel launch of
 * tcl_score is bracketed by a pair of hipEvents recorded on the stream the
 * kernel runs on (the caller's, or a half batch's), grouped by kernel name.
 * tcl_timing_get waits for the recorded events and returns, for entry
 * `idx` in [0, tcl_timing_count(model)), the kernel name (library-owned
 * string), the summed duration in milliseconds and the number of launches.
 * tcl_timing_reset clears the totals. */
TCL_API tcl_status tcl_timing_enable(tcl_model* model, int32_t enable);
TCL_API int32_t tcl_timing_count(const tcl_model* model);
TCL_API tcl_status tcl_timing_get(tcl_model* model, int32_t idx, const char** name, double* total_ms,
                                  int64_t* launches);
TCL_API tcl_status tcl_timing_reset(tcl_model* model);

/* ---------------------------------------------------------------------
 * Distillation (section 6: the knowledge-distillation phase trains a
 * student to match a frozen teacher; section 5.3 / the experimental setup
 * use Adam). One step with B programs:
 *   t = teacher(X) (frozen), s = student(X),
 *   L = mean_b (s_b - t_b)^2 + mean_b (s_b - y_b)^2   (y = labels),
 *   full backward of the student (including the selective scan), then one
 *   bias-corrected Adam update (beta1, beta2, eps, no weight decay) of the
 *   student's fp32 master weights, and the student's compute copies are
 *   re-derived from the updated master.
 * The student must be a bf16 model (bf16 weights and activations in the
 * forward, fp32 master weights, fp32 scan state, fp32 gradients); d_inner
 * <= 256 and dt_rank in {4, 8, 16}. The teacher may be fp32 or bf16. The
 * trainer keeps pointers to both models; they must outlive it. While a
 * trainer exists, the student's parameters change with every step
 * (tcl_get_params returns the current master weights).
 * ------------------------------------------------------------------- */

/* Create a trainer (allocates the gradient blob and the Adam moments, zeroed;
 * the step count starts at 0). max_B, max_L bound every later step (the
 * scan backward stages a program's tokens in windows, so L has no limit of
 * its own beyond the workspace it needs). */
TCL_API tcl_status tcl_trainer_create(tcl_model* teacher, tcl_model* student, float lr, float beta1,
                                      float beta2, float eps, int32_t max_B, int32_t max_L,
                                      tcl_trainer** out);
TCL_API tcl_status tcl_trainer_destroy(tcl_trainer* trainer);

/* Device workspace for one step with B programs padded to L tokens (0 if the
 * shape exceeds the trainer's bounds). */
TCL_API size_t tcl_distill_workspace_bytes(const tcl_trainer* trainer, int32_t B, int32_t L);

/* One distillation step (stream-ordered; see above).
 *   d_feats [B, L, F] fp32, d_lengths [B] int32, d_labels [B] fp32 (device);
 *   d_loss [3] fp32 output: total, mse(student, teacher), mse(student, label);
 *   d_workspace >= tcl_distill_workspace_bytes, 256-byte aligned.
 * The first step with a new (B, L) uploads a small reduction table and
 * synchronises the device once. Programs with invalid lengths must not be
 * passed (their NaN scores would poison the loss). The teacher's forward
 * runs on the teacher model's first stream, forked from `stream` and joined
 * back before the loss by events, beside the student's forward; the step is
 * ordered on `stream` as a whole, and calls that use the teacher model must
 * not be issued from several host threads at once.
 * The step may be captured into a HIP graph on `stream` (stream capture)
 * once a step of the same (B, L) has run uncaptured, with per-kernel timing
 * off on the trainer and the teacher (else TCL_ERR_INVALID_ARG); each replay
 * is one more step: Adam's step count is kept on the device. Replays must
 * not overlap other steps or calls that use the teacher model. */
TCL_API tcl_status tcl_distill_step(tcl_trainer* trainer, int32_t B, int32_t L, const float* d_feats,
                                    const int32_t* d_lengths, const float* d_labels, float* d_loss,
                                    void* d_workspace, size_t ws_bytes, void* stream);

/* The distillation objective of section 6, Eq. (9)-(10), for one batch j:
 *   L = beta * R(s; y) + (1 - beta) * phi * R(s; t)
 *       + ewc_lambda / 2 * sum_k F_k (theta_k - theta_prev_k)^2
 * where s, t are the student's and the teacher's scores, y the labels and
 * R(scores; labels) the LambdaRank loss of section 5.3, Eq. (6), taken over
 * the pairs with rel_i > rel_j: |G_i - G_j| |1/D_i - 1/D_j|
 * log2(1 + exp(-sigma (s_i - s_j))), rel = labels min-max normalised over
 * the batch, G = (2^rel - 1) / maxDCG, D_i = log2(1 + rank of s_i), maxDCG
 * the DCG of the ideal order. theta are the student's fp32 master weights. */
typedef struct tcl_kd_loss {
  float beta;                /* weight of R(s; y), in [0, 1] (0.5 in the paper)       */
  float phi;                 /* teacher-loss gate of this batch, Eq. (10), in [0, 1] */
  float sigma;               /* LambdaRank score scale, > 0 (1)                       */
  float ewc_lambda;          /* EWC weight, >= 0 (1e4 in the paper); 0: no penalty    */
  const float* d_fisher;     /* [n_params] diagonal Fisher information, canonical
                                layout (device); may be NULL when ewc_lambda == 0     */
  const float* d_theta_prev; /* [n_params] the student's parameters after the
                                previous platform (device); likewise                  */
  const float* d_phi;        /* optional device pointer to this batch's gate (e.g. an
                                entry of tcl_teacher_gate's output); when non-NULL it
                                replaces `phi` (read on the device, no host sync)     */
} tcl_kd_loss;

/* One distillation step on the Eq. (9) objective: as tcl_distill_step in
 * every other respect (same workspace, same backward, Adam, re-derivation).
 * d_loss [4] fp32 output: total, R(s; t), R(s; y), EWC penalty. The gradient
 * blob (tcl_trainer_get_grads) includes the EWC gradient. */
TCL_API tcl_status tcl_distill_step_kd(tcl_trainer* trainer, int32_t B, int32_t L, const float* d_feats,
                                       const int32_t* d_lengths, const float* d_labels,
                                       const tcl_kd_loss* kd, float* d_loss, void* d_workspace,
                                       size_t ws_bytes, void* stream);

/* The LambdaRank loss R(scores; labels) of Eq. (6) on one batch of B <= 65536
 * items (defined above, under tcl_kd_loss), e.g. the teacher's batch losses
 * e_T of Eq. (11) that the gate phi is computed from.
 *   d_scores, d_labels [B] fp32 (device); d_loss [1] fp32 output; d_grad [B]
 *   fp32 output dR/dscores (may be NULL); d_workspace >=
 *   tcl_lambdarank_workspace_bytes(B) bytes, 16-byte aligned.
 * O(B^2) work (ranks are counted pairwise); stream-ordered, deterministic. */
TCL_API size_t tcl_lambdarank_workspace_bytes(int32_t B);
TCL_API tcl_status tcl_lambdarank(int32_t B, const float* d_scores, const float* d_labels, float sigma,
                                  float* d_loss, float* d_grad, void* d_workspace, size_t ws_bytes,
                                  void* stream);

/* The teacher-loss gate of section 6, Eq. (10)-(11): the teacher's
 * LambdaRank loss e_j of every batch j (Eq. (11), e.g. tcl_lambdarank of the
 * teacher's scores against the ground truth, one call per batch writing
 * d_e + j) turned into per-batch weights
 *   phi_j = 1 - (e_j - min_k e_k) / (max_k e_k - min_k e_k),
 * so the batch the teacher ranks best gets 1 and the worst 0; all ones when
 * every e_j is equal.
 *   d_e [n] fp32 (device, finite), d_phi [n] fp32 output (device; may not
 *   alias d_e). The normalisation runs in fp64 (each phi_j is the fp32
 *   rounding of the value from the fp32 inputs). One workgroup;
 *   stream-ordered; no workspace. */
TCL_API tcl_status tcl_teacher_gate(int32_t n, const float* d_e, float* d_phi, void* stream);

/* Test entry: tcl_distill_step_kd with two additions for parity tests of
 * the ranking objective. d_rank_keys [B] (device, may be NULL): the values
 * the positions D_i of Eq. (6) are counted from (descending, equal keys in
 * index order) in place of the student's own scores, so that a test can
 * give the library and a reference the same ranking where the student's
 * scores are within rounding of each other (each ordering of such scores
 * is a correct result); with NULL it is the product step. d_scores_out [2B]
 * (device, may be NULL) receives the step's student scores, then the
 * teacher's. Everything else as tcl_distill_step_kd. */
TCL_API tcl_status tcl_test_distill_step_kd_ranked(tcl_trainer* trainer, int32_t B, int32_t L,
                                                   const float* d_feats, const int32_t* d_lengths,
                                                   const float* d_labels, const tcl_kd_loss* kd,
                                                   const float* d_rank_keys, float* d_scores_out, float* d_loss,
                                                   void* d_workspace, size_t ws_bytes, void* stream);

/* ---------------------------------------------------------------------
 * Progressive KB + AC forward (section 6, Fig. 6, Eq. (7)): in the CKD
 * framework's continual-learning phase the frozen knowledge base (KB) and
 * the active column (AC), two models of one architecture, run side by side,
 * and every AC layer after the first reads the KB's input to the same layer
 * through a lateral adapter:
 *   h_i = act_i(W_i h_{i-1} + b_i + alpha_i * U_i ReLU(V_i h^KB_{i-1} + c_i))
 * Layers, in forward order: the encoder's Linear layers, the Mamba blocks
 * (W_i h_{i-1} + b_i is then the block with its residual), the decoder's
 * Linear layers (the first one's KB input is the KB's pooled, normalised
 * vector). act_i is the layer's own activation: ReLU between Linear layers,
 * none after the encoder's last layer, a block, or the score.
 * Lateral blob (fp32, per layer i >= 1 in forward order, n_in and n_out the
 * layer's widths, a the adapter width):
 *   V[a, n_in], c[a], U[n_out, a], alpha[n_out]
 * ------------------------------------------------------------------- */

/* Values in the lateral blob of a model with `cfg` and adapter width a (0 on
 * invalid arguments). */
TCL_API size_t tcl_lateral_param_count(const tcl_config* cfg, int32_t adapter);

/* Join a KB and an AC (distinct fp32 models with identical configs,
 * dec_hidden2 % 4 == 0) by adapters of width `adapter` (a multiple of 4 in
 * [4, 512]) from a host blob of tcl_lateral_param_count values (copied;
 * alpha is folded into U's rows on upload). Keeps pointers to both models:
 * they must outlive the handle. Synchronous. */
TCL_API tcl_status tcl_lateral_create(tcl_model* kb, tcl_model* ac, int32_t adapter, const float* h_params,
                                      size_t n_params, tcl_lateral** out);
TCL_API tcl_status tcl_lateral_destroy(tcl_lateral* lateral);

/* Device workspace of one progressive forward with B programs padded to L. */
TCL_API size_t tcl_progressive_workspace_bytes(const tcl_lateral* lateral, int32_t B, int32_t L);

/* The AC's scores (the CL phase's predictions p_t of Eq. (8)) of B programs,
 * arguments as for tcl_score. Stream-ordered. With the AC model's timing
 * enabled (tcl_timing_enable on the AC), launches are timed under the AC's
 * handle as "kb:*", "ac:*" and "lat:*" entries. */
TCL_API tcl_status tcl_progressive_score(tcl_lateral* lateral, int32_t B, int32_t L, const float* d_feats,
                                         const int32_t* d_lengths, float* d_scores, void* d_workspace,
                                         size_t ws_bytes, void* stream);

/* ---------------------------------------------------------------------
 * What consumes the scores.
 * ------------------------------------------------------------------- */

/* Top-K per segment (section 3, Fig. 2: the cost model keeps the K best
 * candidates of a tuning round for measurement). Segment g holds the scores
 * d_scores[d_seg_offsets[g] .. d_seg_offsets[g+1]-1] (one task's candidates;
 * offsets nondecreasing). d_out [n_seg * K] int32 receives, per segment, the
 * global indices of its K highest scores, highest first; equal scores in
 * index order; NaN scores (unscored programs) after every number; -1 past
 * the end of a segment with fewer than K candidates. K in [1, 1024].
 * Stream-ordered; no workspace. */
TCL_API tcl_status tcl_topk(int32_t n_seg, const int32_t* d_seg_offsets, const float* d_scores, int32_t K,
                            int32_t* d_out, void* stream);

/* The Top-k score of Eq. (12) (section 7.1.2), the paper's dataset-level
 * measure of a cost model: segment g is the candidate set of one subgraph
 * (of one network), as in tcl_topk; d_latency [N] fp32 holds every
 * candidate's measured latency, d_weight [n_seg] fp32 each subgraph's
 * occurrence count in its network, d_scores [N] the model's predictions
 * (ranked as in tcl_topk: higher first, ties by index, NaN last).
 *   Top-k = sum_g w_g min_latency_g / sum_g w_g min(latency of g's k best-
 *   ranked candidates), empty segments adding nothing.
 * d_out [3] fp64 receives Top-k, the numerator and the denominator (sums
 * accumulated in fp64 in a fixed order: deterministic). k in [1, 1024].
 * d_workspace >= tcl_topk_score_workspace_bytes(n_seg, k) bytes, 256-byte
 * aligned. Stream-ordered. */
TCL_API size_t tcl_topk_score_workspace_bytes(int32_t n_seg, int32_t k);
TCL_API tcl_status tcl_topk_score(int32_t n_seg, const int32_t* d_seg_offsets, const float* d_scores,
                                  const float* d_latency, const float* d_weight, int32_t k, double* d_out,
                                  void* d_workspace, size_t ws_bytes, void* stream);

/* The RDU sampler's selection of programs to label, one step of section 4's
 * Alg. 1 on a pool of N scored programs:
 *   f = the predictions d_scores min-max normalised over the pool;
 *   budget[op] = n_select * (pool items of type op) / N;
 *   repeat until n_select programs are selected or no candidate is left:
 *     for each candidate x_i (not labeled), with M labeled programs x_j:
 *       d_s = min_j |f_i - f_j|                              (Eq. (1))
 *       u_s = variance of {f_i} and every f_j, i.e. Eq. (2)-(3)
 *       t_s = f_i * d_s + u_s
 *     T = argmax t_s (equal t_s: the lower index); T is labeled if its
 *     operator type is under budget, else dropped from the candidates.
 *   d_op [N] int32 operator type of each program in [0, n_ops) (programs of
 *   another type are never selected); n_ops in [1, 4096];
 *   d_initial [n_initial >= 1] the initial (random) labeled programs,
 *   distinct indices in [0, N) (entries outside are ignored); they count
 *   toward neither n_select nor the budgets;
 *   d_selected [n_select] int32 output, in selection order, -1 past the end;
 *   d_count [1] int32 output, the number selected;
 *   d_workspace >= tcl_rdu_workspace_bytes(N, n_ops) bytes, 256-byte aligned.
 * Scores must be finite (a NaN-scored program is never selected, and must
 * not be in d_initial). fp64 arithmetic on the device; the host enqueues two
 * kernels per selection and never waits. */
TCL_API size_t tcl_rdu_workspace_bytes(int32_t N, int32_t n_ops);
TCL_API tcl_status tcl_rdu_select(int32_t N, const float* d_scores, const int32_t* d_op, int32_t n_ops,
                                  const int32_t* d_initial, int32_t n_initial, int32_t n_select,
                                  int32_t* d_selected, int32_t* d_count, void* d_workspace, size_t ws_bytes,
                                  void* stream);

/* Copy the gradient blob of the last step (canonical layout, fp32) to the
 * host. Synchronous. */
TCL_API tcl_status tcl_trainer_get_grads(const tcl_trainer* trainer, float* h_out, size_t n_params);

/* Per-kernel timing of the step's own kernels, as for tcl_timing_* (the
 * teacher's scoring kernels are timed on the teacher's handle with
 * tcl_timing_enable). */
TCL_API tcl_status tcl_trainer_timing_enable(tcl_trainer* trainer, int32_t enable);
TCL_API int32_t tcl_trainer_timing_count(const tcl_trainer* trainer);
TCL_API tcl_status tcl_trainer_timing_get(tcl_trainer* trainer, int32_t idx, const char** name,
                                          double* total_ms, int64_t* launches);
TCL_API tcl_status tcl_trainer_timing_reset(tcl_trainer* trainer);

/* Message describing the last failure on this thread ("" if none). */
TCL_API const char* tcl_last_error(void);

/* ---------------------------------------------------------------------
 * Kernel-level entry points, used to test each kernel on its own. They
 * run on packed tokens: program b owns rows offs[b] .. offs[b+1]-1 of
 * every [rows, C] activation (row-major, leading dimension C unless given).
 * ------------------------------------------------------------------- */

/* The packing of a batch's programs into token rows (every scoring and
 * training call starts with it): d_offs[b] = sum over b' < b of valid(len_b'),
 * d_offs[B] = the packed token count, where valid(len) = len for
 * 1 <= len <= L and 0 otherwise (such a program packs no rows). With d_ord
 * non-NULL and L <= 4096 it also writes d_ord [B]: the programs by
 * decreasing valid length, a permutation of 0..B-1 (the order among equal
 * lengths is unspecified); the scans hand programs out in that order. With
 * L > 4096 d_ord is left as it is. d_lengths [B], d_offs [B+1] and d_ord are
 * int32 device memory owned by the caller; B <= 0, L <= 0 or a NULL
 * d_lengths / d_offs return TCL_ERR_INVALID_ARG. */
TCL_API tcl_status tcl_test_offsets(int32_t B, int32_t L, const int32_t* d_lengths, int32_t* d_offs,
                                    int32_t* d_ord, void* stream);

/* fp32 MFMA GEMM used by the model's projections, K % 4 == 0:
 *   epilogue 0: C[M,N] = A W^T (+ bias[N] if d_bias)
 *   epilogue 1: C += A W^T            (the residual epilogue, C read in place)
 *   epilogue 2: C = rstd(A) * A W^T  with rstd(A)_m = (mean_k A[m,k]^2 + 1e-5)^-1/2
 *               (the RMSNorm prologue; the gain is folded into W by the model)
 * tile selects the workgroup tile (0..7: 128x128, 64x64, 64x128, 128x64,
 * 128x256, and 128x128 / 64x128 / 128x64 with K staged 64 at a time; 8: row
 * panels of 128 rows x all N with A held in registers, for K in {64, 128,
 * 164, 192, 256}, K % 4 == 0, no residual epilogue; 9: row panels of 64
 * rows on 16x16 MFMA blocks for K in {256, 384, 512} (up to), K % 4 == 0,
 * no RMSNorm; an unsupported combination returns TCL_ERR_HIP); -1 picks what
 * the model would use for M rows. */
TCL_API tcl_status tcl_test_gemm_f32(int32_t M, int32_t N, int32_t K, const float* d_A,
                                     const float* d_W, const float* d_bias, float* d_C, int32_t tile,
                                     int32_t epilogue, void* stream);

/* The fp32 GEMM of the split path (TCL_F32_MATMUL_SPLIT): A and W fp32,
 * each split exactly into three bf16 parts, six part products accumulated
 * in fp32 on the bf16 matrix cores.
 *   epilogue 0, 1, 2: as tcl_test_gemm_f32 (A [M,K]; d_offs, B, L ignored)
 *   epilogue 3: C = A_g W^T + bias, A fp32 [B, L, K] padded, gathered by
 *               d_offs as in tcl_test_gemm_bf16 kind 4 (M ignored)
 * variant: 1 (32-row panels, K <= 256, epilogues 0, 2, 3), 2 (16-row
 * panels, K rounded up to 64 in {64, 128, 256, 512}, epilogues 0, 1), 3
 * (32-row panels with all N columns accumulated in registers, N <= 256,
 * K <= 512, epilogues 0, 1), 4 (32-row panels with K in two halves on two
 * wavefronts per SIMD, K <= 256, epilogues 0, 2, 3), 5 (the two-part fp16
 * form of TCL_F32_MATMUL_SPLIT: 32-row panels, two workgroups per CU,
 * ceil(K / 16) in {4, 8, 11, 12, 16}, epilogues 0, 2, 3; |W| < 32), 6 (the
 * same operands with all N <= 256 columns in registers, K <= 512 in chunks of
 * 128 under a running power-of-two row scale, epilogues 0, 1; |W| < 32), -1
 * what the model would pick among 1-4; TCL_ERR_UNSUPPORTED otherwise.
 * d_Wsplit: caller-owned device scratch of 3 * N * Kw uint16 (Kw = K rounded
 * up to a multiple of 8, 16-byte aligned) that first receives W's parts
 * (three bf16 parts; variant 5: two fp16 parts of 2^10 W).
 * K % 4 == 0; A 16-byte aligned. */
TCL_API tcl_status tcl_test_gemm_split(int32_t M, int32_t N, int32_t K, const float* d_A,
                                       const int32_t* d_offs, int32_t B, int32_t L, const float* d_W,
                                       const float* d_bias, float* d_C, int32_t variant,
                                       int32_t epilogue, uint16_t* d_Wsplit, void* stream);

/* The bf16 MFMA GEMM (v_mfma_f32_32x32x16_bf16, fp32 accumulation) in the
 * variants the bf16 model runs, selected by kind:
 *   0: C fp32 [M,N] = A W^T (+ bias[N] if d_bias), A bf16 [M,K]
 *   1: C bf16 [M,N] = A W^T, A bf16
 *   2: C bf16 = rstd(A) * (A diag(gain)) W^T, A fp32, rstd as in the fp32
 *      entry (eps 1e-5): the RMSNorm in front of in_proj, d_gain [K]
 *   3: C fp32 += A W^T, A bf16 (the residual epilogue, C read in place)
 *   4: C fp32 = A_g W^T + bias, A fp32 [B, L, K] padded, gathered: packed
 *      row d_offs[b] + t is A[b, t, :] (d_offs [B+1] int32 prefix sums of
 *      lengths in 0..L); C holds B*L rows (only the first d_offs[B] are
 *      written) and M is ignored
 *   5: C fp32 = bf16(A) W^T, A fp32 rounded to bf16 (nearest even) as it is
 *      staged (the distillation backward's data gradients; tiles only)
 *   6: C fp32 += bf16(A) W^T, A fp32 as in 5 (C read in place; tiles only)
 * Other arguments are ignored (may be NULL / 0) for kinds that do not use
 * them. bf16 arrays are bit patterns. W is [N, Kw] bf16 with Kw = K rounded
 * up to a multiple of 8, zero-padded. K % 8 == 0 for bf16 A, K % 4 == 0 for
 * fp32 A; N % 4 == 0; A, W and C 16-byte aligned.
 * tile: -1 = what the model uses; 0..6 = 128x128, 64x64, 64x128, 128x64,
 * 128x256, 256x128, 256x128 on four wavefronts; 7 and 8 = row panels (256 or 128 rows x
 * all N per workgroup, A held in registers; K <= 256 and 16-byte aligned
 * rows of C, else TCL_ERR_HIP). */
TCL_API tcl_status tcl_test_gemm_bf16(int32_t kind, int32_t tile, int32_t M, int32_t N, int32_t K,
                                      const void* d_A, const int32_t* d_offs, int32_t B, int32_t L,
                                      const uint16_t* d_W, const float* d_bias, const float* d_gain,
                                      void* d_C, void* stream);

/* u = SiLU(conv_b + causal depthwise conv(x; conv_w)) per program, fp32.
 * d_x rows have leading dimension ldx >= E (E and ldx multiples of 4, every
 * pointer 16-byte aligned); d_offs [B+1] int32 prefix sums
 * of the lengths; d_w [E,K], d_b [E]; d_u [rows, E]. */
TCL_API tcl_status tcl_test_conv_silu_f32(int32_t B, int32_t E, int32_t K, const int32_t* d_offs,
                                          const float* d_x, int32_t ldx, const float* d_w,
                                          const float* d_b, float* d_u, void* stream);

/* x_proj with the causal conv + SiLU in front (the split path's fused
 * kernel, section 5.2's Mamba block: conv, SiLU, then the projection to
 * [dt_r | B | C]): u = SiLU(conv_b + causal depthwise conv(x; conv_w)) per
 * program and xdbl = u W^T, fp32 with fp32 accuracy. Kernel size 4;
 * E a multiple of 64, <= 512; 1 <= N <= 64; ldx >= E a multiple of 4.
 * d_offs [B+1] int32 prefix sums of the lengths; rows = Mmax >= d_offs[B]
 * bounds the grid; d_x [rows, ldx]; d_w [E, 4], d_b [E]; d_W [N, E];
 * d_u [rows, E], d_xdbl [rows, N] (rows past d_offs[B] are not written).
 * Scratch (caller-owned, device): d_Wsplit 3 N E uint16, d_tpos rows bytes.
 * Every pointer but d_tpos 16-byte aligned. Unsupported shapes give
 * TCL_ERR_UNSUPPORTED. */
TCL_API tcl_status tcl_test_xproj_conv_f32(int32_t B, int32_t rows, int32_t E, int32_t N,
                                           const int32_t* d_offs, const float* d_x, int32_t ldx,
                                           const float* d_w, const float* d_b, const float* d_W,
                                           uint16_t* d_Wsplit, uint8_t* d_tpos, float* d_u,
                                           float* d_xdbl, void* stream);

/* The same for bf16 activations (the bf16 models' fused kernel): d_x [rows,
 * ldx] and d_u [rows, E] bf16, d_W [N, E] bf16 (E a multiple of 128, <= 512;
 * 1 <= N <= 64; ldx a multiple of 8), d_xdbl fp32; bf16 MFMA products
 * accumulated in fp32. d_tpos: caller-owned scratch of rows bytes. */
TCL_API tcl_status tcl_test_xproj_conv_bf16(int32_t B, int32_t rows, int32_t E, int32_t N,
                                            const int32_t* d_offs, const uint16_t* d_x, int32_t ldx,
                                            const float* d_w, const float* d_b, const uint16_t* d_W,
                                            uint8_t* d_tpos, uint16_t* d_u, float* d_xdbl, void* stream);

/* Selective scan with its dt_proj + softplus prologue and gate epilogue,
 * fp32: out = (scan(u, softplus(dt_r W_dt^T + b_dt), -exp(A_log), B, C) +
 * D u) * SiLU(z), with [dt_r|B|C] = d_xdbl rows of R + 2N values and z read
 * from d_z with leading dimension ldz. N must be 16. chunks = 0 runs the
 * sequential scan (one thread per program and channel); 1..8 runs the
 * chunked two-level scan with that many concurrent chunks per program
 * (tcl_score picks it when the batch is too small to fill the GPU). */
TCL_API tcl_status tcl_test_scan_f32(int32_t B, int32_t E, int32_t N, int32_t R, int32_t chunks,
                                     const int32_t* d_offs, const float* d_u, const float* d_xdbl,
                                     const float* d_z, int32_t ldz, const float* d_W_dt,
                                     const float* d_b_dt, const float* d_A_log, const float* d_D,
                                     float* d_out, void* stream);

#endif /* TCL_H */
