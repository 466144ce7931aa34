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
  kXBlk = 16,     // the first xblk_cols columns of C channel-blocked, the rest
                  // packed after them (GemmArgs::xblk_rows; in_proj on the split path)
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
  const float* R = nullptr;   // residual source for kResid (null: C itself), leading dim ldc
  const int* Mdev = nullptr;  // device row count (null: use Mmax)
  int Mmax = 0;               // upper bound on the row count (grid size)
  int N = 0, K = 0;
  float eps = 0.f;
  int relu = 0;               // nonzero: C = max(result, 0) (after bias and residual)
  uint8_t* tpos = nullptr;    // gather on the split path: also write each packed row's position
                              // in its program, clamped to 255 (launch_token_pos's array)
  // kXBlk: C holds [xblk_cols / 64 blocks][xblk_rows][64] (column c of row r
  // at ((c / 64) * xblk_rows + r) * 64 + c % 64), then the other N - xblk_cols
  // columns as [xblk_rows][N - xblk_cols]; ldc is not used
  int64_t xblk_rows = 0;
  int xblk_cols = 0;
};

// Tile shapes (rows x columns of C per workgroup, 4 or 8 wavefronts, K staged
// in chunks of 32 or 64): kWide = 128x128, kNarrow = 64x64 (small-N
// projections), and the variants below.
enum GemmTile {
  kWide = 0,
  kNarrow = 1,
  kTile64x128 = 2,
  kTile128x64 = 3,
  kTile128x256 = 4,
  kTile128x128K64 = 5,
  kTile64x128K64 = 6,
  kTile128x64K64 = 7,
  kPanel = 8,    // row panels: 128 rows x all N per workgroup, A in registers (K <= 256, no residual)
  kPanel16 = 9,  // row panels of 64 rows on 16x16 MFMA blocks (K <= 512, no RMSNorm or gather)
  kNumGemmTiles = 10
};

// tile < 0: the tile pick_gemm_f32_tile chooses for these arguments.
hipError_t launch_gemm_f32(const GemmArgs& a, int flags, int tile, hipStream_t s);
// The tile the scoring and training passes use for this GEMM (up to Mmax rows).
GemmTile pick_gemm_f32_tile(const GemmArgs& a, int flags);
bool gemm_f32_panel_fits(const GemmArgs& a, int flags);
hipError_t launch_gemm_f32_panel(const GemmArgs& a, int flags, hipStream_t s);
bool gemm_f32_panel16_fits(const GemmArgs& a, int flags);
hipError_t launch_gemm_f32_panel16(const GemmArgs& a, int flags, hipStream_t s);

// fp32 GEMM on the bf16 matrix cores, with fp32 accuracy: A (fp32, from
// GemmArgs) and W split three ways into bf16 parts, six of the nine part
// products accumulated in fp32. Ws holds W's parts as [3][N][ldws] bf16
// (ldws >= K, a multiple of 8, the padding zero; launch_split_weights or the
// model's derived weights). GemmArgs.W is not read. Variants:
//   kSplit32: 32-row MFMA blocks, K <= 256, no residual;
//   kSplit16: 16-row blocks, K rounded up to 64 in {64, 128, 256, 512}, no
//             RMSNorm or gather;
//   kSplit32Acc: 32-row blocks with all N columns accumulated in registers,
//             N <= 256, K <= 512, no RMSNorm or gather;
//   kSplit32H: 32-row blocks with K split between two wavefronts per SIMD
//             (half the A registers each), K <= 256, no residual.
enum GemmSplitVariant { kSplit32 = 1, kSplit16 = 2, kSplit32Acc = 3, kSplit32H = 4 };
bool gemm_split_supports(const GemmArgs& a, int flags, int variant);
int gemm_split_variant(const GemmArgs& a, int flags);  // the variant the model uses, or -1 (none)
// variant < 0: gemm_split_variant's pick; hipErrorInvalidValue if unsupported
hipError_t launch_gemm_split(const GemmArgs& a, const uint16_t* Ws, int ldws, int flags, int variant,
                             hipStream_t s);
hipError_t launch_split_weights(const float* W, int N, int K, int ldw, uint16_t* out, hipStream_t s);

// fp32 GEMM on the fp16 matrix cores with two-part operands, fp32-level
// accuracy (each operand in two fp16 parts after an exact power-of-two
// scale, three of the four part products accumulated in fp32; per product
// at most 12 units of fp32 rounding beyond the exact value). Wh holds W's
// parts as [2][N][ldwh] fp16 (launch_split_weights_f16 or the model's
// derived weights: W scaled by 2^kF16WeightExp, so |W| < 32). 32-row panels
// of 128 rows per workgroup, two workgroups per CU; ceil(K / 16) in {4, 8,
// 11, 12, 16}; flags 0, kBias, kRowNorm or kBias | kGather.
bool gemm_f16s_supports(const GemmArgs& a, int flags);
hipError_t launch_gemm_f16s(const GemmArgs& a, const uint16_t* Wh, int ldwh, int flags, hipStream_t s);
// The same operands with the low parts unscaled (all three part products in
// one accumulator), all N <= 256 columns' accumulators in registers and
// K <= 512 walked in chunks of 128 under a running power-of-two row scale: flags
// 0, kBias or kResid (out_proj). Wh: launch_split_weights_f16(flat = true).
bool gemm_f16acc_supports(const GemmArgs& a, int flags);
hipError_t launch_gemm_f16acc(const GemmArgs& a, const uint16_t* Wh, int ldwh, int flags, hipStream_t s);
// flat: the low parts unscaled (gemm_f16acc's operand form), else scaled by 2^11
hipError_t launch_split_weights_f16(const float* W, int N, int K, int ldw, uint16_t* out, hipStream_t s,
                                    bool flat = false);

// x_proj with the causal depthwise conv + SiLU in front (split path, 32-row
// blocks, all N in registers): u = SiLU(b + sum_k w[e,k] x[t-3+k, e]) within
// each program is computed per 128-channel chunk, stored to u [rows, K] and
// contracted with W (Ws as above) into C = u W^T. GemmArgs.A is not read;
// a.K = d_inner. tpos[r] is the position of packed row r in its program
// (clamped to 255). Kernel size 4, K a multiple of 64 and <= 512, N <= 64.
struct ConvIn {
  const float* x = nullptr;   // conv input [rows, ldx] (the x half of in_proj's output)
  int64_t ldx = 0;
  const float* w = nullptr;   // [K, 4]
  const float* b = nullptr;   // [K]
  const uint8_t* tpos = nullptr;
  float* u = nullptr;         // [rows, K]
  // > 0: x is channel-blocked, [K / 64][xblk_rows][64] (in_proj's kXBlk
  // output; ldx is not used), so that a chunk's rows are contiguous
  int64_t xblk_rows = 0;
};
bool gemm_split_conv_supports(const GemmArgs& a, const ConvIn& cv, int d_conv);

// The same fusion for bf16 models: x and u bf16, W bf16 [N][ldw] (the
// model's bf16 x_proj weights), C fp32 [rows, ldc]. Kernel size 4, E a
// multiple of 128 and <= 512, N <= 64.
struct ConvArgsBF16 {
  const uint16_t* x = nullptr;  // conv input [rows, ldx] (the x half of in_proj's output)
  int64_t ldx = 0;
  const float* w = nullptr;     // [E, 4]
  const float* b = nullptr;     // [E]
  const uint8_t* tpos = nullptr;
  uint16_t* u = nullptr;        // [rows, E]
  const uint16_t* W = nullptr;
  int64_t ldw = 0;
  float* C = nullptr;
  int64_t ldc = 0;
  const int* Mdev = nullptr;
  int Mmax = 0, N = 0, E = 0;
};
bool gemm_bf16_conv_supports(const ConvArgsBF16& a, int d_conv);
hipError_t launch_gemm_bf16_conv(const ConvArgsBF16& a, hipStream_t s);
hipError_t launch_gemm_split_conv(const GemmArgs& a, const ConvIn& cv, const uint16_t* Ws, int ldws,
                                  hipStream_t s);

// bf16 GEMM: C = A W^T with A fp32 (converted while staged) or bf16, W bf16
// ([N, ldw] row-major, zero-padded in K to a multiple of 8, ldw % 8 == 0),
// C fp32 or bf16, fp32 accumulation. kRowNorm also scales A by gain[k]
// before the conversion (the RMSNorm gain). An fp32 A needs K % 4 == 0, a
// bf16 A K % 8 == 0.
struct GemmArgsBF16 {
  const void* A = nullptr;
  int64_t lda = 0;
  const int* offs = nullptr;
  int B = 0, L = 0;
  const uint16_t* W = nullptr;
  int64_t ldw = 0;
  const float* bias = nullptr;
  const float* gain = nullptr;
  void* C = nullptr;
  int64_t ldc = 0;
  const float* R = nullptr;   // residual source for kResid (null: C itself), leading dim ldc
  const int* Mdev = nullptr;
  int Mmax = 0;
  int N = 0, K = 0;
  float eps = 0.f;
};

enum GemmBF16Kind {
  kInputF32toF32,    // fp32 features (gathered) -> fp32, + bias
  kNormF32toBF16,    // fp32 residual -> RMSNorm (rstd, gain) -> bf16
  kBF16ResidF32,     // bf16 -> fp32 C += result
  kBF16toF32,        // bf16 -> fp32
  kBF16toF32Bias,    // bf16 -> fp32, + bias
  kBF16toBF16,       // bf16 -> bf16
  kF32toF32,         // fp32 (rounded to bf16 as staged) -> fp32
  kF32ResidF32,      // fp32 (rounded to bf16 as staged) -> fp32 C += result
};

// Workgroup tiles (rows x columns of C): 4 wavefronts unless noted.
enum GemmBF16Tile {
  kB128x128 = 0,
  kB64x64 = 1,
  kB64x128 = 2,
  kB128x64 = 3,
  kB128x256 = 4,    // 8 wavefronts
  kB256x128 = 5,    // 8 wavefronts
  kB256x128W4 = 6,  // 4 wavefronts of 128x64 each
  kBPanel = 7,      // row panels: 256 rows x all N per workgroup (K <= 256)
  kBPanel128 = 8,   // row panels of 128 rows (32 per wavefront)
  kNumGemmBF16Tiles = 9
};

// tile < 0: the tile pick_gemm_bf16_tile chooses. N and ldc must be
// multiples of 4 (hipErrorInvalidValue otherwise).
hipError_t launch_gemm_bf16(const GemmArgsBF16& a, GemmBF16Kind kind, int tile, hipStream_t s);
GemmBF16Tile pick_gemm_bf16_tile(GemmBF16Kind kind, int Mmax, int N, int K);
// the row-panel kernel (kBPanel): K <= 256, C (and R) 16-byte aligned rows
bool gemm_bf16_panel_fits(const GemmArgsBF16& a, bool bf16_out);
hipError_t launch_gemm_bf16_panel(const GemmArgsBF16& a, GemmBF16Kind kind, int rows_per_wave, hipStream_t s);

// ---------------------------------------------------------------- weight-gradient GEMM
// P[s][i][j] = sum over tokens m of split s of A[m, i] * B[m, j]
// (A: [M, NI] fp32 with leading dimension lda; B: [M, NJ] fp32 or bf16, or
// fp32 gathered from a padded [B, L, ldb] tensor by token offsets).
// P holds `splits` partial [NI, NJ] tiles; sum them with launch_reduce.
struct GemmTNArgs {
  const float* A = nullptr;
  int64_t lda = 0;
  const void* Bm = nullptr;
  int64_t ldb = 0;
  const int* offs = nullptr;  // gather: token offsets of B's programs
  int B = 0, L = 0;
  const int* rows = nullptr;  // gather (optional): B's row of each packed token, else found from offs
  float* P = nullptr;
  const int* Mdev = nullptr;
  int Mmax = 0;
  int NI = 0, NJ = 0;
};
enum TNKind { kTN_F32_F32, kTN_F32_BF16, kTN_F32_GatherF32 };
int gemm_tn_splits(int Mmax, int NI, int NJ);
hipError_t launch_gemm_tn(const GemmTNArgs& a, TNKind kind, int splits, hipStream_t s);
// rows[offs[b] + t] = b * L + t for the valid tokens of every program b
hipError_t launch_packed_rows(const int* offs, int B, int L, int* rows, hipStream_t s);
// the same on the bf16 matrix cores, both operands rounded to bf16 (nearest
// even), fp32 accumulation: for models that compute in bf16
hipError_t launch_gemm_tn_bf16(const GemmTNArgs& a, TNKind kind, int splits, hipStream_t s);

// ---------------------------------------------------------------- per-program kernels
// offs[b] = sum of valid lengths before b; offs[B] = total packed rows.
// Lengths outside [1, L] count as 0 tokens. ord (optional, B entries, used
// when L <= 4096): the programs longest first.
constexpr int kOrderMaxL = 4096;
hipError_t launch_offsets(const int* lengths, int B, int L, int* offs, hipStream_t s, int* ord = nullptr);
// tpos[r] = position of packed row r in its program, clamped to 255 (rows
// past offs[B] are not written).
hipError_t launch_token_pos(const int* offs, int B, uint8_t* tpos, hipStream_t s);

// Activations are stored as fp32 (T = float) or bf16 (T = uint16_t); the
// arithmetic is fp32 either way.

// u = SiLU(conv_b + sum_k w[e,k] x[t-(K-1)+k, e]) within each program.
// E and ldx are multiples of 4 (fp32) or 8 (bf16); pointers 16-byte aligned.
template <typename T>
hipError_t launch_conv_silu(int B, int E, int K, const int* offs, const T* x, int ldx,
                            const float* w, const float* b, T* u, hipStream_t s);

// Selective scan with dt_proj+softplus prologue, D skip and SiLU(z) gate.
// xdbl rows ([dt_r | B | C], R + 2N values) are fp32. out may alias u (each
// element is read then written by the same thread).
// ysave (optional) keeps y before the gate, for the backward pass; ckpt (optional, N = 16, with the
// padded length L) keeps the state after every kScanCkptTokens-th token of a
// program but its last chunk, [B][E][ceil(L / kScanCkptTokens)][N], which is
// where the backward scan restarts its recomputation. ord (optional): the
// order in which programs are handed to workgroups (launch_offsets' ord).
constexpr int kScanCkptTokens = 4;
template <typename T>
hipError_t launch_scan(int B, int E, int N, int R, const int* offs, const T* u, const float* xdbl,
                       const T* z, int ldz, const float* W_dt, const float* b_dt, const float* A_log,
                       const float* D, T* out, hipStream_t s, T* ysave = nullptr, float* ckpt = nullptr,
                       int L = 0, const int* ord = nullptr);

// The same scan as a chunked two-level scan: each program's tokens are split
// into `chunks` (1..8) that are scanned concurrently and stitched through
// their affine summaries. scan_chunks_for picks the chunk count the batch
// needs to fill the GPU (0: the sequential kernel already does).
template <typename T>
hipError_t launch_scan_chunked(int B, int E, int N, int R, int chunks, const int* offs, const T* u,
                               const float* xdbl, const T* z, int ldz, const float* W_dt,
                               const float* b_dt, const float* A_log, const float* D, T* out,
                               hipStream_t s);
int scan_chunks_for(int B, int E, int L);

// Final RMSNorm (optional) + masked mean-pool + Linear-ReLU-Linear head.
// W1T is W1 transposed ([d, h]). Programs with invalid lengths get NaN.
// pooled_out [B, d] and a1_out [B, h] (optional) keep the pooled vector and
// the head's pre-ReLU activation for the backward pass.
hipError_t launch_tail_f32(int B, int L, int d, int h, const int* offs, const int* lengths,
                           const float* H, const float* g_f, int final_norm, float eps,
                           const float* W1T, const float* b1, const float* W2, const float* b2,
                           float* scores, hipStream_t s, float* pooled_out = nullptr,
                           float* a1_out = nullptr);
// The same with a three-layer decoder Linear(d,h) ReLU Linear(h,h2) ReLU
// Linear(h2,1): W2T is the second layer transposed, [h][h2], b2 its bias
// [h2], W3 [h2] and b3 [1] the output layer. h, h2 <= 256.
// scores[b] = NaN where lengths[b] is outside [1, L] (an invalid program)
hipError_t launch_mask_scores(int B, int L, const int* lengths, float* scores, hipStream_t s);
// dst[r][c] = c < F ? src[r][c] : 0 for rows x ld (row-major, src rows of F)
hipError_t launch_pad_rows(const float* src, int64_t rows, int F, int ld, float* dst, hipStream_t s);
hipError_t launch_tail3_f32(int B, int L, int d, int h, int h2, const int* offs, const int* lengths,
                            const float* H, const float* g_f, int final_norm, float eps,
                            const float* W1T, const float* b1, const float* W2T, const float* b2,
                            const float* W3, const float* b3, float* scores, hipStream_t s);

// ---------------------------------------------------------------- distillation step
// Reductions of per-block partials: dst[i * dst_stride] =
// sum_s src[s * split_stride + i * src_stride], i < n. Offsets are in floats,
// relative to the workspace (src) and to the gradient blob or the loss
// vector (dst), so a job table depends only on the batch shape.
struct ReduceJob {
  int64_t src, split_stride, src_stride;
  int64_t dst, dst_stride;
  int64_t n;
  int32_t nsplit;
  int32_t dst_buf;  // 0: gradient blob, 1: loss vector
  // the job's blocks in the launch: [block0, block0 + nblocks), numbered
  // from the first job of the launch (reduce_blocks assigns them)
  int32_t block0, nblocks;
};
// Assign block ranges to jobs[0 .. njobs) for one launch; returns the
// launch's block count.
int reduce_blocks(ReduceJob* jobs, int njobs);
// njobs <= kMaxReduceJobs; nblocks = reduce_blocks' result for the same jobs
constexpr int kMaxReduceJobs = 1024;
hipError_t launch_reduce(const ReduceJob* d_jobs, int njobs, int nblocks, const float* ws, float* grad,
                         float* loss, hipStream_t s);

// Weight layouts derived from the fp32 master blob: one flat index space over
// all jobs (job j covers [start_j, start_j + rows*cols)); the destination is a
// byte offset in the model's device block. kDeriveFold multiplies column c by
// master[src2 + c]. With round_bf16 every master value is first rounded to
// bf16 (bf16 models compute with the rounded weights). The split kinds write
// the three bf16 parts of the (folded) value to dst as [3][rows][ld].
enum DeriveKind {
  kDeriveF32 = 0,
  kDeriveBF16 = 1,
  kDeriveFold = 2,
  kDeriveSplit = 3,        // three bf16 parts
  kDeriveFoldSplit = 4,
  kDeriveSplitF16 = 5,     // two fp16 parts of 2^kF16WeightExp W (split2_f16_scaled)
  kDeriveFoldSplitF16 = 6,
  kDeriveSplitF16Flat = 7  // the same, low part unscaled (split2_f16_flat)
};
struct DeriveJob {
  int64_t start, src, src2, dst;
  int32_t rows, cols, ld, transpose, kind, pad_;
};
// step_bump (may be null): a training step's device step count, advanced by one
hipError_t launch_derive(const float* master, const DeriveJob* d_jobs, int njobs, int64_t total,
                         void* base, int round_bf16, hipStream_t s, int64_t* step_bump = nullptr);

hipError_t launch_rmsnorm_fwd(int d, int Mmax, const int* Mdev, const float* H, const float* g,
                              float eps, uint16_t* n, float* rstd, hipStream_t s);
int rmsnorm_bwd_blocks(int Mmax);
hipError_t launch_rmsnorm_bwd(int d, int Mmax, const int* Mdev, const float* dN, const float* H,
                              const float* rstd, const float* g, float* dH, float* dg_part,
                              hipStream_t s);
int loss_head_blocks(int B);
// part: [blocks][2h + 4] = dW2 (h) | db1 (h) | db2 | mse_t | mse_l | total.
// With ds_in (dL/ds [B]) and loss_in ({total, term_t, term_y}) the score
// gradient and the loss come from elsewhere (the ranking objective) and the
// MSE terms are not used.
hipError_t launch_loss_head_bwd(int B, int d, int h, const float* s, const float* t, const float* y,
                                const float* a1, const float* W1, const float* W2, float* da1,
                                float* dpooled, float* part, hipStream_t st, const float* ds_in = nullptr,
                                const float* loss_in = nullptr);

// ---------------------------------------------------------------- ranking objectives
// LambdaRank (Eq. (6)) of scores s [B] against label set l0 (nsets == 1) or
// against l0 and l1 weighted w0, w1 (nsets == 2). ds [B] (may be null)
// receives d/ds of (w0 L(s; l0) + w1 L(s; l1)) (nsets == 1: of L(s; l0));
// out receives {L} (nsets == 1) or {w0 L0 + w1 L1, L1, L0}. ws: a scratch
// of rank_workspace_floats(B, nsets) floats. key [B] (may be null: s) holds
// the values the score ranks D_i are counted from (descending, equal keys
// in index order); w1_scale (may be null: 1) is a device value that
// multiplies w1 (the teacher gate of the batch).
size_t rank_workspace_floats(int B, int nsets);
hipError_t launch_lambdarank(int B, int nsets, const float* s, const float* l0, const float* l1, float sigma,
                             float w0, float w1, float* ws, float* ds, float* out, hipStream_t st,
                             const float* key = nullptr, const float* w1_scale = nullptr);
// The teacher-loss gate of Eq. (10)-(11): phi[j] = 1 - (e[j] - min e) /
// (max e - min e) over n batch losses (all ones when they are equal).
hipError_t launch_teacher_gate(int n, const float* e, float* phi, hipStream_t st);
// ---------------------------------------------------------------- score consumers
// Per-segment top-K: out [n_seg][K] global indices of each segment's K best
// scores (best first, equal scores in index order, NaN last), -1 past a
// segment's end. offs [n_seg + 1]. K in [1, 1024].
hipError_t launch_topk(int n_seg, const int* offs, const float* s, int K, int* out, hipStream_t st);
// Eq. (12): out[0..2] = Top-k, numerator, denominator (fp64). ws holds
// topk_score_workspace_bytes(n_seg, k) bytes, 256-byte aligned.
size_t topk_score_workspace_bytes(int n_seg, int k);
hipError_t launch_topk_score(int n_seg, const int* offs, const float* s, const float* lat, const float* w,
                             int k, double* out, void* ws, hipStream_t st);
// RDU selection (Alg. 1, Eq. (1)-(3)) of up to n_select programs from a pool
// of N: out [n_select] in selection order (-1 past the end), count [1].
// op [N] in [0, n_ops) (others are never selected), n_ops <= 4096;
// init [n_init] the initial labeled programs (distinct, in [0, N)).
size_t rdu_workspace_bytes(int N, int n_ops);
hipError_t launch_rdu_select(int N, const float* s, const int* op, int n_ops, const int* init, int n_init,
                             int n_select, int* out, int* count, void* ws, hipStream_t st);

// EWC penalty (Eq. (9)): grad += lam F (theta - prev); loss[3] =
// lam/2 sum F (theta - prev)^2 and loss[0] += loss[3]. part: ewc_part_floats().
int ewc_part_floats();
hipError_t launch_ewc(int64_t n, const float* theta, const float* prev, const float* fisher, float lam,
                      float* grad, float* part, float* loss, hipStream_t st);
// dg_part: [B][d]
hipError_t launch_normf_pool_bwd(int B, int d, const int* offs, const float* H, const float* g_f,
                                 int final_norm, float eps, const float* dpooled, float* dH,
                                 float* dg_part, hipStream_t s);
size_t scan_bwd_ckpt_floats(int B, int E, int L, int N);
// ckpt: the forward scan's checkpoints of this layer (launch_scan's ckpt).
// dA_part: [B][E][N] (already d/dA_log), dD_part: [B][E]
hipError_t launch_scan_bwd(int B, int E, int L, int N, int R, const int* offs, const uint16_t* u,
                           const float* xdbl, const uint16_t* xz, const uint16_t* ysave,
                           const float* dyg, const float* W_dt, const float* b_dt,
                           const float* A_log, const float* D, const float* ckpt, float* dv, float* du,
                           float* dxz, float* dxdbl, float* dA_part, float* dD_part, float* dbc_part,
                           hipStream_t s, const int* ord = nullptr);
// dbc_part (scratch for launch_scan_bwd; null: one block per program)
size_t scan_bwd_part_floats(int B, int L, int N);
// part: [B][K+1][E] = dw (K rows) | db
hipError_t launch_conv_bwd(int B, int E, int K, const int* offs, const uint16_t* x, int ldx,
                           const float* w, const float* b, const float* du, float* dx, int lddx,
                           float* part, hipStream_t s);
int colsum_splits(int Mmax);
hipError_t launch_colsum(const int* Mdev, int Mmax, const float* A, int64_t lda, int C, int splits,
                         float* part, hipStream_t s);
// d_step: the steps taken before this one (device), for the bias correction
hipError_t launch_adam(int64_t n, float* p, float* m, float* v, const float* g, float lr, float b1,
                       float b2, float eps, const int64_t* d_step, hipStream_t s);

}  // namespace tcl
