// Host-side model state shared by the scoring and training entry points
// (internal to libtcl).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdarg>
#include <cstdio>
#include <string>
#include <vector>

#include "kernels.h"
#include "tcl.h"

namespace tcl {

tcl_status fail(tcl_status st, const char* fmt, ...);
const char* last_error();

#define TCL_HIP(call)                                                                          \
  do {                                                                                         \
    hipError_t e_ = (call);                                                                    \
    if (e_ != hipSuccess) return ::tcl::fail(TCL_ERR_HIP, "%s: %s", #call, hipGetErrorString(e_)); \
  } while (0)

inline size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

// Offsets (in floats) of every tensor of the canonical parameter blob.
struct BlobLayout {
  size_t W0, b0, g_f, W1, b1, W2, b2, total;
  // multi-layer encoder: layers 1 and 2 after W0, b0 (n_enc Linear layers in
  // all); three-layer decoder: W3, b3 after W2 [h2,h], b2 [h2]
  int n_enc = 1;
  int enc_dims[4] = {0, 0, 0, 0};  // F, hidden widths, d_model
  size_t We[3] = {0, 0, 0}, be[3] = {0, 0, 0};
  size_t W3 = 0, b3 = 0;
  struct L {
    size_t g, W_in, conv_w, conv_b, W_x, W_dt, b_dt, A_log, D, W_out;
  };
  std::vector<L> layers;
};
BlobLayout blob_layout(const tcl_config& c);

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
  int category(const char* n);
  hipError_t event(hipEvent_t* e);
  hipError_t flush();
  void release();
};

// Launch CALL (a hipError_t expression) on stream `s`; with timing enabled,
// bracket it by events on that stream under category NAME.
#define TCL_LAUNCH(TIMING, NAME, CALL)                                                \
  do {                                                                                \
    hipEvent_t ea_ = nullptr, eb_ = nullptr;                                          \
    if ((TIMING).on) {                                                                \
      TCL_HIP((TIMING).event(&ea_));                                                  \
      TCL_HIP(hipEventRecord(ea_, s));                                                \
    }                                                                                 \
    TCL_HIP(CALL);                                                                    \
    if ((TIMING).on) {                                                                \
      TCL_HIP((TIMING).event(&eb_));                                                  \
      TCL_HIP(hipEventRecord(eb_, s));                                                \
      (TIMING).pending.push_back({(TIMING).category(NAME), ea_, eb_});                \
    }                                                                                 \
  } while (0)

}  // namespace tcl

// Device-side state of a model: one allocation holding every derived weight
// layout, the fp32 master blob, and the table of derivation jobs.
struct tcl_model {
  tcl_config cfg{};
  int device = 0;
  // tcl_score's two half-batch streams and their fork/join events (null
  // when they could not be created: the batch then runs as one)
  hipStream_t aux[2] = {nullptr, nullptr};
  hipEvent_t ev[3] = {nullptr, nullptr, nullptr};
  int score_streams = 2;  // tcl_set_score_streams
  size_t n_params = 0;
  void* dev = nullptr;
  size_t dev_bytes = 0;
  float* master = nullptr;                 // canonical fp32 blob (device)
  tcl::DeriveJob* jobs = nullptr;          // derivation table (device)
  int njobs = 0;
  int64_t derive_total = 0;
  struct Layer {
    // fp32 (bf16-rounded for bf16 models)
    float *W_in_fold, *g, *conv_w, *conv_b, *W_x, *W_dt, *b_dt, *A_log, *D, *W_out;
    // transposed fp32 copies for the backward pass
    float *W_outT, *W_xT, *W_inT, *W_dtT;
    // bf16 copies (bf16 models)
    uint16_t *W_in_h, *W_x_h, *W_out_h;
    // transposed bf16 copies for the backward pass's data gradients (bf16 models)
    uint16_t *W_outT_h, *W_xT_h, *W_inT_h;
    // three-way bf16 splits, [3][rows][cols] (fp32 models on the split path):
    // W_in with the gain folded, W_x, W_out
    uint16_t *W_in_s, *W_x_s, *W_out_s;
    // two-part fp16 splits of W_in (gain folded) and W_out, [2][rows][cols]
    // (fp32 models on the split path), and whether their ranges allow them
    uint16_t *W_in_h2, *W_out_h2;
    bool in_h2_ok, out_h2_ok;
  };
  float *W0 = nullptr, *b0 = nullptr, *g_f = nullptr, *W1 = nullptr, *W1T = nullptr,
        *b1 = nullptr, *W2 = nullptr, *b2 = nullptr;
  int ldw0 = 0;  // leading dimension of the fp32 W0: F rounded up to 4, zero-padded
  // encoder layers 1.. of a multi-layer encoder (fp32 [out][in], bias, and
  // the three-way split [3][out][ld] on the split path, ld = in rounded to 8)
  float *We[3] = {nullptr, nullptr, nullptr}, *be[3] = {nullptr, nullptr, nullptr};
  uint16_t* We_s[3] = {nullptr, nullptr, nullptr};
  uint16_t* We_h2[3] = {nullptr, nullptr, nullptr};  // two-part fp16 splits, [2][out][ld]
  bool We_h2_ok[3] = {false, false, false};
  // three-layer decoder: W2 [h2][h] and transposed [h][h2], W3 [h2], b3 [1]
  float *W2T = nullptr, *W3 = nullptr, *b3 = nullptr;
  uint16_t* W0_h = nullptr;  // bf16 [d, ldw0_h], K zero-padded to a multiple of 8
  int ldw0_h = 0;
  uint16_t* W0_s = nullptr;  // three-way bf16 split of W0, [3][d][ldw0_h] (split path)
  uint16_t* W0_h2 = nullptr;  // two-part fp16 split of W0, [2][d][ldw0_h] (split path)
  bool W0_h2_ok = false;
  bool split = false;        // fp32 model whose projections run on the split path
  std::vector<Layer> layers;
  tcl::Timing timing;
};

namespace tcl {

// Workspace plan of one scoring call (byte offsets, 256-aligned).
struct ScorePlan {
  size_t offs, ord, tpos, H, xz, u, xdbl, feats, enc1, enc2, total;
};
ScorePlan score_plan(const tcl_config& c, int64_t B, int64_t L);

// The model's GEMM: the split path where it has a kernel for the shape,
// the fp32 MFMA path otherwise.
hipError_t model_gemm(const tcl_model* m, const GemmArgs& a, const uint16_t* Ws, int ldws, int flags,
                      hipStream_t s);
// fp32 models: encoder Linear layer i (0 = the gathered input Linear; A is
// then the [B, L, ldw0] padded input) from A to C, ReLU when `act`; and
// Mamba block l in place on the residual stream H [tokens, d]. Launches are
// timed under tag + kernel name.
// tpos_out (layer 0 only, optional): where the split path's gathered input
// Linear also writes the token positions; *tpos_written tells whether it did.
tcl_status enqueue_encoder_layer_f32(tcl_model* m, Timing& T, const std::string& tag, int i, int B, int L,
                                     const int* offs, const float* A, float* C, bool act, hipStream_t s,
                                     uint8_t* tpos_out = nullptr, bool* tpos_written = nullptr);
// tpos (per packed row, its position in its program; launch_token_pos) lets
// the split path fuse the conv into x_proj; null: the conv runs on its own.
tcl_status enqueue_block_f32(tcl_model* m, Timing& T, const std::string& tag, int l, int B, int L,
                             const int* offs, const uint8_t* tpos, float* H, float* xz, float* u, float* xdbl,
                             hipStream_t s, const int* ord = nullptr);

// Enqueue the scoring pass (no argument checks): its parts in order.
tcl_status run_score(tcl_model* m, int B, int L, const float* d_feats, const int* d_lengths,
                     float* d_scores, char* ws, hipStream_t s);
// One part of the scoring pass: 0 the front (token offsets, the encoder),
// 1 .. n_layers the Mamba block part - 1, n_layers + 1 the tail (pool and
// head). The parts of one batch run in order on one stream.
tcl_status run_score_part(tcl_model* m, int B, int L, const float* d_feats, const int* d_lengths,
                          float* d_scores, char* ws, hipStream_t s, int part);

// Re-derive every weight layout from the device master blob (stream-ordered).
tcl_status derive_weights(tcl_model* m, hipStream_t s);

tcl_status check_config(const tcl_config* c);

}  // namespace tcl
