// Host-side launch descriptors shared between the C-ABI layer and the kernel
// translation units. Every pointer is a device pointer; the ABI layer has
// validated sizes and carved the workspace before filling these.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>

namespace fpo {

constexpr int kMaxMats = 64;

// Vocabulary chunk c of a plan: the first nwide chunks are cw + cq wide, the
// others cw, and the last one runs to V. Sets its first entry and width.
inline void chunk_span(int64_t V, int nchunk, int64_t cw, int64_t cq, int nwide, int c, int64_t* v0,
                       int64_t* w) {
  *v0 = (int64_t)c * cw + (int64_t)std::min(c, nwide) * cq;
  *w = c == nchunk - 1 ? V - *v0 : cw + (c < nwide ? cq : 0);
}

struct OeLaunch {
  bool bf16;
  int64_t T, d, V, Vc;  // Vc: widest chunk, rounded up to 256
  int64_t ldp;          // row pitch of the staged p~ (elements, >= Vc)
  int nchunk, nwide;    // chunk layout (chunk_span)
  int64_t cw, cq;
  int nsplit;
  float eps, min_rms;
  const void* h_final;
  const void* gamma;
  const void* W_U;
  const int32_t* targets;
  float* g_tilde;
  void* g_tilde_lp;
  float* g_pre;
  float* lse;
  float* loss;
  int32_t* argmax;
  int32_t* bad_targets;
  // workspace
  void* y;
  void* P;
  float* blk_m;
  float* blk_s;
  int32_t* blk_i;
  float* fout;   // [T] exp(Ref - M_new) of the current chunk
  float* alpha;  // [T] exp(M_old - M_new)
  float* ref;    // [T] staging reference of the current chunk
  float* zt;     // [T] target logit <y_t, W_U[y_t]> (from the stored y)
  float* runM;
  float* runS;
  int32_t* runA;
  float* G;
  void* stream;
};
hipError_t launch_output_error(const OeLaunch& a);

struct PgLaunch {
  bool bf16;
  bool full_mlp;
  int64_t T, d, d_ff, Tp;
  int L;
  float scale;
  const void* g_lp;                 // [T, d]
  const void* a[kMaxMats];          // [T, d_ff]
  const void* W3i[kMaxMats];        // [d, d_ff]
  const void* q[kMaxMats];
  const void* u[kMaxMats];
  const void* x_in[kMaxMats];       // [T, d]
  float* dW3[kMaxMats];
  uint16_t* dW3_bf16[kMaxMats];     // staged bf16 pseudogradient (instead of dW3), or null
  float* dW1[kMaxMats];
  float* dW2[kMaxMats];
  const float* ref[kMaxMats];
  // norm chain: per layer, g_l = VJP_pre(VJP_post(g~ fp32; mlp_out_l, gamma_l); pre_in_l, gamma_pre_l),
  // either factor optional
  bool pffn;
  const float* g_f32;               // [T, d]
  const void* mlp_out[kMaxMats];    // [T, d]
  const void* gamma_pffn[kMaxMats]; // [d]
  float pffn_eps, pffn_min_rms;
  bool pre;
  const void* pre_in[kMaxMats];     // [T, d] cached pre-MLP norm input
  const void* gamma_pre[kMaxMats];  // [d]
  float pre_eps, pre_min_rms;
  double* sumsq;                    // [n_mats] or null
  double* ref_dot;
  double* ref_sumsq;
  float* ref_cos;
  // workspace
  void* gT;                         // [d, Tp] transposed signal
  void* g_row;                      // [T, d] per-layer signal (post-FFN composition, full-MLP)
  float* chain_stats;               // [T, 4] per-token norm-chain statistics
  void* dq_T;                       // [d_ff, Tp] full-MLP gate error (transposed)
  void* du_T;                       // [d_ff, Tp] full-MLP up error (transposed)
  double* part;                     // per-tile partials
  void* stream;
};
hipError_t launch_pseudograd(const PgLaunch& a);
int64_t pseudograd_tiles(bool bf16, int64_t M, int64_t N);

constexpr int kOptAdamW = 1;  // fpo_opt_kind FPO_OPT_ADAMW

struct UpdLaunch {
  int kind;
  double lr, momentum, beta1, beta2, adam_eps, weight_decay, clip_frac;
  int64_t step;
  int n;
  int64_t numel[kMaxMats];
  const void* grad[kMaxMats];       // float32, or bf16 when grad_bf16
  bool grad_bf16;
  float* W[kMaxMats];
  void* W_lp[kMaxMats];
  bool lp_bf16;
  float* s1[kMaxMats];
  float* s2[kMaxMats];
  const double* grad_sumsq;
  double* W_sumsq;
  float* clip_scale;
  double* part;
  // clip-the-update mode: the clip bounds ||W' - W|| instead of ||dW|| (two
  // passes; dsq: [n] ||delta||^2 scratch)
  bool clip_update;
  double* dsq;
  void* stream;
};
// blocks = false: only the per-matrix reductions (||W'||^2, clip factors) of
// blocks already applied (by the fused pseudogradient launch).
hipError_t launch_update(const UpdLaunch& a, bool blocks = true);
// The update blocks of matrix m of `a` on `stream` (partials at part + blk_base);
// grid > 0: that many workgroups visit the blocks grid-stride.
hipError_t launch_update_blocks(const UpdLaunch& a, int m, int64_t blk_base, void* stream, int grid = 0);
// Caller-owned side stream and events of the overlapped path.
struct OverlapLaunch {
  void* side;
  void* ready;
  void* done;
};
// W3-only bf16 pseudogradients with the optimizer step overlapped (u: the
// update of the same matrices, grad = the dW3 outputs, grad_sumsq = a.sumsq);
// ov: the caller's side stream and events, or null for the library's own.
hipError_t launch_pseudograd_update(const PgLaunch& a, const UpdLaunch& u, const OverlapLaunch* ov);
int64_t update_blocks(int64_t numel);

struct CosLaunch {
  int n;
  int64_t numel[kMaxMats];
  const float* A[kMaxMats];
  const void* B[kMaxMats];
  bool b_bf16;
  double* dot;
  double* sa;
  double* sb;
  float* cos;
  double* part;
  void* stream;
};
hipError_t launch_cosine(const CosLaunch& a);
int64_t cosine_blocks(int64_t numel);

}  // namespace fpo
