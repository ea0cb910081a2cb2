/*
 * fpo.h - C ABI of the MI355X (gfx950) FPO hot path.
 *
 * Forward-Pass-Only MLP training derives every update from one forward pass:
 * the output-layer error e = softmax(z) - onehot(y) over the full vocabulary
 * (Sec. 3.1 step 2), its projection g = e W_U through the unembedding
 * (eq. gproj), the closed-form final-RMSNorm VJP with the min-RMS clamp
 * (Sec. 3.2, App. E eq. rmsnorm-vjp), and for every target layer the
 * token-summed outer product of that signal with the cached MLP activation
 * (eq. w3update), followed by a relatively clipped optimizer step on fp32
 * master weights (App. A). The layer-viability diagnostic compares the
 * pseudogradient with a reference gradient by cosine (eq. cosine).
 *
 * Conventions shared by every call
 *  - Pointers are DEVICE pointers unless marked [host]. Arrays of pointers
 *    ("const T* const* x") are [host] arrays whose entries are device
 *    pointers.
 *  - Every call validates its arguments on the host, enqueues work on
 *    `stream` (a hipStream_t; NULL = the default stream) and returns without
 *    synchronising. Results are valid once the stream has reached them.
 *  - The calls allocate nothing, never synchronise the host and issue no
 *    memset, so they can be captured into a HIP graph (stream capture); the
 *    overlapped optimizer path's side stream joins a capture through its
 *    events. Scalars passed by value (the optimizer step number, hence the
 *    first-step and AdamW bias-correction terms) are fixed at capture.
 *  - Library state: a thread-local error string; the static scratch array of
 *    fpo_apply_update_noalloc; and, for fpo_pseudograd's overlapped optimizer
 *    path when the caller passes no fpo_overlap, one side stream and two
 *    events per device, created by the first such call on the device (make it
 *    before any capture), kept until the process ends, and shared by every
 *    such call on that device under a lock: such calls from several threads
 *    are serialised while they enqueue, and one issued while another thread's
 *    capture holds the shared side stream joins that capture. Passing an
 *    fpo_overlap of the caller's own avoids all of this.
 *  - The caller owns every buffer. The library allocates no device memory;
 *    scratch space comes from the caller's workspace, whose size the
 *    matching *_workspace query returns (fpo_apply_update_noalloc instead
 *    uses a fixed device array inside the library, see there). Workspace pointers must be 256-byte
 *    aligned; every tensor operand (activations, weights, gradients,
 *    optimizer state, reference gradients) must be 16-byte aligned (the
 *    kernels move 16 bytes per lane; a bf16 W_lp: 8). Per-token and
 *    per-matrix outputs
 *    (lse, loss, argmax, sums of squares, dot products, cosines) need only
 *    their element alignment.
 *  - Inputs are read only. Outputs are fully overwritten (never accumulated
 *    into) and must not alias inputs, except where a buffer is documented as
 *    in/out.
 *  - Row-major layouts throughout: activations [T, features]; W_U [V, d];
 *    W3 (down projection) [d, d_ff]; W1 (gate), W2 (up) [d_ff, d].
 *  - Dtypes: FPO_F32 means every tensor is float32. FPO_BF16 means
 *    h_final, gamma, W_U, activations, g_tilde_lp, W3_init, gate, up, x_in
 *    and W_lp are bfloat16 (raw 16-bit patterns); everything else is
 *    float32 (g_tilde, dW, masters, optimizer state, reference gradients)
 *    or float64 (sums of squares, dot products).
 *  - d, d_ff and V must be multiples of 8; T, d, d_ff, V, L >= 1; at most
 *    2^23 tokens per call, and d <= 2^22 for fpo_pseudograd (launch-grid
 *    limits).
 *  - Errors: calls return 0 (FPO_OK) or a positive fpo_status. Problems a
 *    host can detect (NULL, non-positive or misaligned sizes, unknown
 *    enum, negative eps / min_rms / lr, small workspace) return before any
 *    launch. A failed launch returns FPO_ERR_HIP. fpo_last_error() gives a
 *    thread-local message for the last non-OK return. Data errors only the
 *    device can see (a target outside [0, V)) are counted, not returned.
 */
#ifndef FPO_H
#define FPO_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define FPO_ABI_VERSION 7

typedef enum {
  FPO_OK = 0,
  FPO_ERR_NULL = 1,        /* a required pointer is NULL */
  FPO_ERR_SHAPE = 2,       /* a size is non-positive, breaks the multiple-of-8 rule or exceeds a limit */
  FPO_ERR_DTYPE = 3,       /* unknown dtype */
  FPO_ERR_ARG = 4,         /* bad scalar argument or enum */
  FPO_ERR_WORKSPACE = 5,   /* workspace NULL, misaligned or smaller than the query */
  FPO_ERR_UNSUPPORTED = 6, /* valid request the library does not implement */
  FPO_ERR_HIP = 7          /* a HIP runtime call or kernel launch failed */
} fpo_status;

typedef enum { FPO_F32 = 0, FPO_BF16 = 1 } fpo_dtype;
typedef enum {
  FPO_MODE_W3 = 0,
  FPO_MODE_FULL_MLP = 1,
  FPO_MODE_POST_FFN = 2,
  FPO_MODE_GRAD_BF16 = 4,
  FPO_MODE_PRE_MLP = 8
} fpo_mode; /* bit flags */
typedef enum { FPO_OPT_SGD = 0, FPO_OPT_ADAMW = 1 } fpo_opt_kind;
typedef enum { FPO_CLIP_GRADIENT = 0, FPO_CLIP_UPDATE = 1 } fpo_clip_target;

/* Output-error call description.
 *   eps         inside rho = sqrt(mean x^2 + eps), forward and VJP (Sec. 3.2)
 *   min_rms     floor on rho inside the VJP only (App. E "Min-RMS clamp"; 0.5)
 *   vocab_chunk vocabulary columns staged per pass; 0 = library default.
 *               Rounded up to a multiple of 256. Affects scratch size and
 *               rounding order only, never the definition. */
typedef struct {
  int64_t T, d, V;
  int32_t dtype; /* fpo_dtype */
  float eps;
  float min_rms;
  int64_t vocab_chunk;
} fpo_oe_desc;

/* Pseudogradient call description.
 *   L      number of target layers in this call (<= 64)
 *   mode   FPO_MODE_W3 (0): down projection only; FPO_MODE_FULL_MLP (bit 0):
 *          also the gate (W1) and up (W2) signals through the fixed feedback
 *          W3_init (eq. errh); FPO_MODE_POST_FFN (bit 1): compose each layer's
 *          post-FFN RMSNorm VJP (the call's post_ffn argument is then
 *          required; the workspace holds every layer's composed signal);
 *          FPO_MODE_PRE_MLP (bit 3): compose each layer's pre-MLP RMSNorm
 *          VJP after it (pre_mlp argument; see fpo_pre_mlp);
 *          FPO_MODE_GRAD_BF16 (bit 2, FPO_BF16 W3-only path with the
 *          fused update): each dW3 tile is rounded once to bf16 (RNE) into
 *          the workspace and the update reads that (the precision of the
 *          paper's bf16 einsum); sumsq is then of the rounded values and dW3
 *          must be NULL
 *   scale  multiplier of the token sum; the paper divides by the token count
 *          (App. A pseudocode), so callers pass 1/T */
typedef struct {
  int64_t T, d, d_ff, L;
  int32_t dtype; /* fpo_dtype */
  int32_t mode;  /* fpo_mode */
  float scale;
} fpo_pg_desc;

/* Optimizer step on fp32 masters (Sec. 3.1 end; App. A).
 *   SGD:   momentum (0.9 in the paper), no dampening, no Nesterov; the first
 *          step (step == 1) stores the clipped gradient as the buffer.
 *   AdamW: beta1, beta2, adam_eps, decoupled weight_decay (0.01 in the
 *          paper), bias correction with the 1-based `step`.
 *   clip_frac  relative clip, 0.01 in the paper; <= 0 disables it.
 *   clip_target  what the clip bounds. FPO_CLIP_GRADIENT (0, the App. A
 *          pseudocode): ||s*dW||_F <= clip_frac * ||W||_F applied to the
 *          gradient before the step. FPO_CLIP_UPDATE (1, the App. A prose
 *          "clip each step's weight update"): the optimizer runs on the
 *          unclipped gradient and its state advances unclipped; only the
 *          step applied to W is scaled, ||W' - W||_F <= clip_frac * ||W||_F,
 *          with delta = -lr * b' (SGD) or -lr*wd*W - lr*m_hat/(sqrt(v_hat)+eps)
 *          (AdamW). Two streaming passes instead of one.
 * Hyperparameters are double; the derived factors (1 - beta, 1 - lr * wd,
 * bias corrections) are formed in double on the host and rounded once to
 * float32 for the device arithmetic. AdamW moments must be zero before step 1;
 * SGD ignores the buffer's content at step 1. */
typedef struct {
  int32_t kind; /* fpo_opt_kind */
  double lr, momentum, beta1, beta2, adam_eps, weight_decay, clip_frac;
  int64_t step;
  int32_t clip_target; /* fpo_clip_target */
} fpo_opt;

/* Buffers an update writes in place. Every member is a [host] array of
 * n_mats entries, except W_sumsq and clip_scale, which are device arrays.
 *   W_master  fp32 master weights, in/out
 *   W_lp      low-precision copy written after the step (bf16 RNE of the new
 *             master; fp32 copy when the call's dtype is FPO_F32); the array
 *             or any entry may be NULL to skip it
 *   state1    SGD momentum buffer | AdamW first moment, in/out. May be NULL
 *             (the array or an entry) for SGD with momentum 0: plain SGD
 *             keeps no state (b = s * dW each step; 14 bytes per parameter
 *             of HBM traffic instead of 22)
 *   state2    AdamW second moment, in/out (NULL for SGD)
 *   W_sumsq   device double[n_mats]: in ||W||_F^2 of the current masters
 *             (the clip's reference), out ||W'||_F^2 of the new masters
 *   clip_scale device float[n_mats], out: the clip factor s used (nullable;
 *             in FPO_CLIP_UPDATE mode the factor applied to the update) */
typedef struct {
  float* const* W_master;
  void* const* W_lp;
  float* const* state1;
  float* const* state2;
  double* W_sumsq;
  float* clip_scale;
} fpo_update_bufs;

int fpo_abi_version(void);

/* Thread-local message describing the last non-OK return on this thread. */
const char* fpo_last_error(void);

/* ---------------------------------------------------------------------------
 * fpo_output_error - output error, projection through W_U^T and the clamped
 * final-RMSNorm VJP (Sec. 3.1 steps 2-4; eq. gproj; App. E eq. rmsnorm-vjp).
 *
 * For each token t: rho_t = sqrt(mean_k x_tk^2 + eps); y_t = gamma * x_t / rho_t;
 * z_tv = <y_t, W_U[v]> for every v in [0, V); e_t = softmax(z_t) - onehot(y_t);
 * g_t = sum_v e_tv W_U[v]; then with rho~ = max(rho_t, min_rms), x^ = x_t / rho~,
 * c = (1/d) <x^, gamma * g_t>: g~_t = (gamma * g_t - c x^) / rho~.
 * The T x V logits are never stored: the vocabulary is processed in chunks
 * with a running maximum and partition function per token.
 *
 *   h_final    [T, d]  cached final-norm input (dtype)
 *   gamma      [d]     final-norm gain (dtype)
 *   W_U        [V, d]  unembedding (dtype)
 *   targets    int32 [T] next-token ids. An id outside [0, V) is counted in
 *              *bad_targets and its token gets e = 0, g = g~ = 0, loss = 0.
 *   g_tilde    float [T, d] out: the VJP output
 *   g_tilde_lp [T, d] out (dtype), nullable: g~ rounded to the operand dtype
 *   g_pre      float [T, d] out, nullable: g before the VJP
 *   lse, loss  float [T] out, nullable: log-sum-exp of z_t; lse - z_{t,y_t}
 *   argmax     int32 [T] out, nullable: lowest index of max_v z_tv
 *   bad_targets int32 [1] out, nullable: number of out-of-range targets
 *   ws, ws_bytes  workspace of at least fpo_output_error_workspace(desc) bytes
 * Returns FPO_OK or an fpo_status. */
size_t fpo_output_error_workspace(const fpo_oe_desc* desc);
int fpo_output_error(const fpo_oe_desc* desc, const void* h_final, const void* gamma,
                     const void* W_U, const int32_t* targets, float* g_tilde, void* g_tilde_lp,
                     float* g_pre, float* lse, float* loss, int32_t* argmax,
                     int32_t* bad_targets, void* ws, size_t ws_bytes, void* stream);

/* Post-feedforward RMSNorm composition (Sec. 3.2 "Post-feedforward RMSNorm";
 * App. A pseudocode; OLMo-2 and Gemma 3 layouts): each target layer's left
 * operand becomes g_l = the clamped RMSNorm VJP of that layer's post-FFN norm
 * (input: the cached MLP output, gain: the layer's post-FFN gain) applied to
 * the fp32 g~:
 *   rho~ = max(sqrt(mean mlp_out_t^2 + eps), min_rms); x^ = mlp_out_t / rho~;
 *   c = (1/d) <x^, gamma * g~_t>;  g_l,t = (gamma * g~_t - c x^) / rho~
 * rounded to the operand dtype, then used for dW3_l and (full-MLP mode) E_l.
 *   g_tilde   float [T, d]: fpo_output_error's g_tilde
 *   mlp_out   [host] L pointers to [T, d] (dtype): cached MLP outputs
 *   gamma     [host] L pointers to [d] (dtype): post-FFN norm gains
 *   eps, min_rms  as in fpo_oe_desc (the paper uses min_rms 0.5) */
typedef struct {
  const float* g_tilde;
  const void* const* mlp_out;
  const void* const* gamma;
  float eps;
  float min_rms;
} fpo_post_ffn;

/* Pre-MLP RMSNorm composition (Sec. 3.2 "Pre-MLP RMSNorm (Qwen3, Gemma 3)";
 * the per-architecture composition appendix and its table). The paper says
 * these families also compose "the pre-MLP RMSNorm Jacobian at each target
 * layer" without placing it on the W3 path; the library applies it as the
 * App. A pseudocode applies the post-FFN norm's: the clamped RMSNorm VJP at
 * the norm's cached input x (the residual stream entering the layer's MLP
 * sub-block) and gain, after the post-FFN VJP when both are composed (Gemma 3):
 *   rho~ = max(sqrt(mean x_t^2 + eps), min_rms); x^ = x_t / rho~;
 *   c = (1/d) <x^, gamma * v_t>;  g_l,t = (gamma * v_t - c x^) / rho~
 * with v the fp32 g~ (or its post-FFN composition), rounded once to the
 * operand dtype, then used for dW3_l and (full-MLP mode) E_l.
 *   g_tilde  float [T, d]: fpo_output_error's g_tilde (the same pointer as
 *            post_ffn->g_tilde when both are given)
 *   x        [host] L pointers to [T, d] (dtype): cached pre-MLP norm inputs
 *   gamma    [host] L pointers to [d] (dtype): pre-MLP norm gains */
typedef struct {
  const float* g_tilde;
  const void* const* x;
  const void* const* gamma;
  float eps;
  float min_rms;
} fpo_pre_mlp;

/* Caller-owned side stream and events for fpo_pseudograd's overlapped
 * optimizer path (each matrix's update runs on side_stream beside the GEMM
 * launches that follow its outer products). All three are hipStream_t / hipEvent_t handles of
 * the current device; the events should be created with
 * hipEventDisableTiming. The library only records, waits on and launches into
 * them; a set must not be used by two calls that run concurrently. */
typedef struct {
  void* side_stream;
  void* ready_event;
  void* done_event;
} fpo_overlap;

/* ---------------------------------------------------------------------------
 * fpo_pseudograd - per-layer token-summed outer products (eq. w3update, with
 * the App. A divisor supplied as desc->scale) and, in full-MLP mode, the
 * W1/W2 signals through the fixed feedback W3_init (eq. errh) with exact
 * SwiGLU derivatives:
 *   dW3_l = scale * g~^T a_l                                  [d, d_ff]
 *   E_l = g~ W3_init_l; du = E_l * SiLU(q_l); dq = E_l * u_l * SiLU'(q_l)
 *   dW1_l = scale * dq^T x_in_l,  dW2_l = scale * du^T x_in_l  [d_ff, d]
 *
 *   g_tilde_lp [T, d] (dtype): the pseudogradient signal (fpo_output_error's
 *              g_tilde_lp, or g_tilde on the FPO_F32 path)
 *   a          [host] L pointers to [T, d_ff] cached MLP activations (dtype)
 *   W3_init, gate (q), up (u), x_in: [host] L pointers each, FULL_MLP only
 *              (NULL otherwise): W3_init [d, d_ff], q and u [T, d_ff],
 *              x_in [T, d], all dtype
 *   dW3        [host] L pointers to float [d, d_ff] out. May be NULL only
 *              when `ref` is given (fused diagnostic: no dW3 is stored), and
 *              must be NULL in FPO_MODE_GRAD_BF16
 *   dW1, dW2   [host] L pointers to float [d_ff, d] out (FULL_MLP only)
 *   sumsq      double out, nullable: ||dW||_F^2 per matrix, in the order
 *              W3(0..L-1) then, in FULL_MLP mode, W1(0..L-1), W2(0..L-1)
 *   ref        [host] L pointers to float [d, d_ff] reference gradients,
 *              nullable (layer-viability diagnostic, eq. cosine)
 *   ref_dot, ref_sumsq  double [L] out (required when ref is given):
 *              <dW3_l, R_l> and ||R_l||_F^2
 *   ref_cos    float [L] out, nullable (only with ref): the layer-viability
 *              cosine <dW3_l, R_l> / (||dW3_l|| ||R_l||), 0 when either norm
 *              is 0 (eq. cosine), from the same float64 sums
 *   post_ffn   required iff desc->mode has FPO_MODE_POST_FFN: compose each
 *              layer's post-FFN norm VJP (see fpo_post_ffn); g_tilde_lp is
 *              then unused and may be NULL
 *   pre_mlp    required iff desc->mode has FPO_MODE_PRE_MLP: compose each
 *              layer's pre-MLP norm VJP (see fpo_pre_mlp); g_tilde_lp is
 *              then unused and may be NULL
 *   opt, upd   both NULL, or both given: the call then also applies
 *              fpo_apply_update to the matrices in `sumsq` order, with the
 *              same result bit for bit as calling it separately
 *   overlap    nullable: the side stream and events of the overlapped
 *              optimizer path (see fpo_overlap); NULL uses the library's own
 *              (see "Library state" above)
 *   stream     the work is ordered on this stream. With opt given on the
 *              FPO_BF16 path with the gradient clip (W3 only or FULL_MLP),
 *              each matrix's norm reduction and update run on the side
 *              stream once its outer products are done, overlapping the GEMM
 *              launches that follow (the next layer's outer products; with
 *              FULL_MLP the W1/W2 launches too), and are joined back to
 *              `stream` with an event before the call's last kernel.
 * Returns FPO_OK or an fpo_status. */
size_t fpo_pseudograd_workspace(const fpo_pg_desc* desc);
int fpo_pseudograd(const fpo_pg_desc* desc, const void* g_tilde_lp, const void* const* a,
                   const void* const* W3_init, const void* const* gate, const void* const* up,
                   const void* const* x_in, float* const* dW3, float* const* dW1,
                   float* const* dW2, double* sumsq, const float* const* ref, double* ref_dot,
                   double* ref_sumsq, float* ref_cos, const fpo_post_ffn* post_ffn,
                   const fpo_pre_mlp* pre_mlp, const fpo_opt* opt, const fpo_update_bufs* upd,
                   const fpo_overlap* overlap, void* ws, size_t ws_bytes, void* stream);

/* ---------------------------------------------------------------------------
 * fpo_apply_update - relative clip and optimizer step on fp32 masters
 * (App. A: clip_rel_norm then the fp32-master step; Sec. 3.1 optimizers).
 * For each matrix m: s_m = 1 if clip_frac <= 0 or grad_sumsq[m] == 0, else
 * min(1, clip_frac * sqrt(W_sumsq[m]) / sqrt(grad_sumsq[m])); G = s_m * grad;
 * then the SGD-momentum or AdamW step on W_master, the optional low-precision
 * copy, and W_sumsq[m] <- ||W'||_F^2. The scale is computed on the device.
 * With opt->clip_target == FPO_CLIP_UPDATE the same s formula takes
 * ||delta||^2 of the unclipped step instead of grad_sumsq (see fpo_opt).
 *
 *   n_mats       number of matrices (<= 64 per call)
 *   numel        [host] int64 [n_mats]: elements per matrix (multiple of 4)
 *   grad         [host] n_mats pointers to float gradients
 *   grad_sumsq   double [n_mats]: ||grad||_F^2 (fpo_pseudograd's sumsq)
 *   lp_dtype     dtype of upd->W_lp entries (FPO_BF16 or FPO_F32)
 * Returns FPO_OK or an fpo_status. */
size_t fpo_apply_update_workspace(int64_t n_mats, const int64_t* numel);
int fpo_apply_update(const fpo_opt* opt, int64_t n_mats, const int64_t* numel,
                     const float* const* grad, const double* grad_sumsq,
                     const fpo_update_bufs* upd, int32_t lp_dtype, void* ws, size_t ws_bytes,
                     void* stream);

/* ---------------------------------------------------------------------------
 * fpo_apply_update_noalloc - fpo_apply_update for callers that cannot
 * allocate device memory or pass a workspace: code being captured into a HIP
 * graph, tight serving loops, harnesses that forbid allocation. Same
 * arguments (minus the workspace), same kernels and the same results bit for
 * bit as fpo_apply_update.
 *
 * Its scratch (one double per 4096 parameters of every matrix, plus one per
 * matrix) lives in a device array inside the library, FPO_NOALLOC_SCRATCH_BYTES
 * (8 MiB) on every GPU the library runs on, held until the process ends: at
 * most about 4.2e9 parameters per call. A call needing more returns
 * FPO_ERR_WORKSPACE before any launch. Nothing in the array has to start at
 * zero (every word a call reads was written earlier in the same call), so the
 * previous call's contents are harmless; but every call on one GPU shares the
 * array, so calls that overlap on one GPU (two streams, or two host threads
 * enqueueing concurrently) race on it and must be serialised by the caller.
 * The first call on a device resolves that device's copy of the array
 * (hipGetSymbolAddress): make it before any graph capture starts.
 * No hipMalloc, hipFree or allocating library routine is called.
 * Returns FPO_OK or an fpo_status. */
#define FPO_NOALLOC_SCRATCH_BYTES (8u << 20)
int fpo_apply_update_noalloc(const fpo_opt* opt, int64_t n_mats, const int64_t* numel,
                             const float* const* grad, const double* grad_sumsq,
                             const fpo_update_bufs* upd, int32_t lp_dtype, void* stream);

/* ---------------------------------------------------------------------------
 * fpo_cosine - per-pair dot product, squared norms and cosine (eq. cosine):
 * cos = <A, B> / (||A|| ||B||), 0 when either norm is 0.
 *   numel     [host] int64 [n_pairs] elements per pair (multiple of 4)
 *   A         [host] n_pairs pointers to float
 *   B         [host] n_pairs pointers (dtype_B), or NULL for norms of A only
 *   dot, sumsq_A, sumsq_B  double [n_pairs] out, each nullable
 *   cos       float [n_pairs] out, nullable
 * Returns FPO_OK or an fpo_status. */
size_t fpo_cosine_workspace(int64_t n_pairs, const int64_t* numel);
int fpo_cosine(int64_t n_pairs, const int64_t* numel, const float* const* A,
               const void* const* B, int32_t dtype_B, double* dot, double* sumsq_A,
               double* sumsq_B, float* cos, void* ws, size_t ws_bytes, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* FPO_H */
