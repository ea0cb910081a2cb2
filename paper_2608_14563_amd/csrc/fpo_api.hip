// C-ABI layer of libfpo: argument validation, workspace planning and carving,
// and the launch sequence of each call on the caller's stream. No device
// memory is allocated here and nothing synchronises with the host.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <mutex>
#include <string>

#include "../../include/fpo.h"
#include "launch.hpp"

// Scratch of fpo_apply_update_noalloc: a file-scope device array (one copy
// per GPU, held until the process ends). Host code never passes `scratch`
// itself to a kernel (its host-side name is not a device address): each
// device's copy is resolved once with hipGetSymbolAddress, on that device,
// and only that address is used.
static __device__ __align__(256) unsigned char scratch[FPO_NOALLOC_SCRATCH_BYTES];

namespace {

thread_local std::string g_err;

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

int hip_fail(hipError_t e, const char* where) {
  return fail(FPO_ERR_HIP, "%s: %s (%d)", where, hipGetErrorString(e), (int)e);
}

inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }
inline int64_t round_up(int64_t a, int64_t b) { return ceil_div(a, b) * b; }
inline bool aligned(const void* p, uintptr_t a) { return ((uintptr_t)p % a) == 0; }

constexpr int64_t kIntMax = 0x7fffffff;
// Launch geometry: the per-token kernels use one workgroup (256 lanes) per
// token in a 1-D grid, whose lane count must stay below 2^32; the signal
// transpose tiles d in 64-row steps along a grid dimension capped at 65536.
constexpr int64_t kMaxTokens = (int64_t)1 << 23;
constexpr int64_t kMaxHidden = (int64_t)1 << 22;
constexpr size_t kAlign = 256;

struct Carver {
  char* base;
  size_t off = 0;
  explicit Carver(void* b) : base((char*)b) {}
  template <typename T>
  T* take(int64_t n) {
    T* p = base ? (T*)(base + off) : nullptr;
    off += round_up((int64_t)(n * sizeof(T)), kAlign);
    return p;
  }
};

// A rows x cols band of 2-byte elements addressable through 32-bit buffer
// offsets with 2^31 reserved as the out-of-range offset.
bool band_fits(int64_t rows, int64_t cols) { return rows * cols <= ((int64_t)1 << 30); }

// ------------------------------------------------------------------ plans
// Vocabulary chunks: the first `nwide` chunks are cw + cq wide, the others cw,
// and the last one takes what remains of V (see fpo::chunk_span). Vc, the
// widest chunk rounded up to 256, sizes the staged p~.
struct OePlan {
  int64_t Vc = 0, ldp = 0, nb = 0;
  int64_t cw = 0, cq = 0;
  int nchunk = 1, nwide = 0;
  int nsplit = 1;
};

// Workgroups one wave of the MI355X grid holds (one 256 x 256 tile per CU).
constexpr int64_t kWaveSlots = 256;
// The staged p~ rows are padded by 256 bytes so that the row pitch is an odd
// multiple of 256 bytes: with a power-of-two pitch (V = 131072: 256 KiB) the
// 256 rows of one tile share an L2 set and its stores are written back to HBM
// several times over (measured: 3.3 GB written for a 1.1 GB p~).
constexpr int64_t kPadBytes = 256;
// Default bytes of staged p~ per vocabulary chunk (see plan_oe).
constexpr int64_t kStageBytes = (int64_t)128 << 20;

OePlan plan_oe(const fpo_oe_desc& d) {
  const bool bf16 = d.dtype == FPO_BF16;
  const int64_t BM = bf16 ? 256 : 128, BN = BM, WTN = bf16 ? 128 : 64;
  const int64_t pad = kPadBytes / (bf16 ? 2 : 4);
  const int64_t esz = bf16 ? 2 : 4;
  // widest chunk allowed: the caller's width, or by default kStageBytes of
  // staged p~ (half of the 256 MB Infinity Cache, so that a chunk's p~ is
  // written by the logits launch and read back by the projection from the
  // cache rather than HBM; the T x V logits never exist in memory as a whole)
  int64_t wmax = d.vocab_chunk > 0 ? round_up(d.vocab_chunk, 256)
                                   : std::max<int64_t>(256, kStageBytes / esz / d.T / 256 * 256);
  // a chunk of W_U ([Vc, d]) and the staged p~ ([T, Vc + pad]) are copied
  // through 32-bit offsets
  if (bf16) {
    const int64_t lim = std::min(((int64_t)1 << 30) / d.d, ((int64_t)1 << 30) / d.T - pad);
    wmax = std::min(wmax, std::max<int64_t>(256, lim / 256 * 256));
  }
  OePlan p;
  const int64_t V256 = round_up(d.V, 256);
  if (V256 <= wmax) {
    p.cw = V256;
  } else {
    const int64_t n0 = ceil_div(d.V, wmax);
    p.nchunk = (int)n0;
    p.cw = round_up(ceil_div(d.V, n0), 256);  // equal widths (the caller's choice)
    // Default plan: widths in whole logits waves. A chunk's logits launch has
    // ceil(T / BM) token tiles per 256-wide vocabulary tile, so a multiple of
    // q vocabulary entries fills whole waves of 256 workgroups; the last chunk
    // alone carries the remainder, and the total number of waves is that of
    // one launch over the whole vocabulary. (Equal widths left a nearly empty
    // last wave in every chunk: T = 2048, V = 100352 in four chunks of 25088
    // ran the logits 19% slower than one launch.)
    const int64_t q = round_up(std::max<int64_t>(1, kWaveSlots / ceil_div(d.T, BM)) * BN, 256);
    if (d.vocab_chunk <= 0 && q <= wmax) {
      for (int64_t n = n0;; ++n) {
        const int64_t base = d.V / (n * q) * q;
        if (base == 0) break;                       // keep equal widths
        const int64_t extra = d.V - n * base;       // < n q
        const int64_t k = std::min<int64_t>(n - 1, extra / q);
        const int64_t last = d.V - (n - 1) * base - k * q;
        const int64_t widest = std::max(k > 0 ? base + q : base, last);
        if (round_up(widest, 256) > wmax) continue;  // one chunk more
        p.nchunk = (int)n;
        p.cw = base;
        p.cq = q;
        p.nwide = (int)k;
        break;
      }
    }
  }
  // widest chunk
  int64_t widest = 0;
  for (int c = 0; c < p.nchunk; ++c) {
    int64_t v0, w;
    fpo::chunk_span(d.V, p.nchunk, p.cw, p.cq, p.nwide, c, &v0, &w);
    widest = std::max(widest, w);
  }
  p.Vc = round_up(widest, 256);
  p.ldp = p.Vc + pad;
  p.nb = p.Vc / WTN;
  // Split the projection's K range so that its launch fills whole waves: the
  // smallest split count (at most 8, at least two blocks per split) that gives
  // at least one wave and the best filled last wave. (T = 4096, d = 3072: 192
  // tiles, two splits leave the second wave half empty, four fill three.)
  const int64_t tiles = ceil_div(d.T, BM) * ceil_div(d.d, BN);
  const int64_t nsmax = std::min<int64_t>(8, std::max<int64_t>(1, p.nb / 2));
  const int64_t ns0 = std::min(nsmax, ceil_div(kWaveSlots, tiles));
  int64_t best = ns0;
  double best_fill = 0.0;
  for (int64_t ns = ns0; ns <= nsmax; ++ns) {
    const int64_t wg = tiles * ns;
    const double fill = (double)wg / (double)(ceil_div(wg, kWaveSlots) * kWaveSlots);
    if (fill > best_fill + 1e-9) {
      best = ns;
      best_fill = fill;
    }
  }
  p.nsplit = (int)best;
  return p;
}

size_t carve_oe(const fpo_oe_desc& d, const OePlan& p, void* ws, fpo::OeLaunch* L) {
  const int64_t esz = d.dtype == FPO_BF16 ? 2 : 4;
  Carver c(ws);
  void* y = c.take<char>(d.T * d.d * esz);
  void* P = c.take<char>(d.T * p.ldp * esz);
  float* blk_m = c.take<float>(d.T * p.nb);
  float* blk_s = c.take<float>(d.T * p.nb);
  int32_t* blk_i = c.take<int32_t>(d.T * p.nb);
  float* fout = c.take<float>(d.T);
  float* alpha = c.take<float>(d.T);
  float* ref = c.take<float>(d.T);
  float* zt = c.take<float>(d.T);
  float* runM = c.take<float>(d.T);
  float* runS = c.take<float>(d.T);
  int32_t* runA = c.take<int32_t>(d.T);
  float* G = c.take<float>((int64_t)p.nsplit * d.T * d.d);
  if (L) {
    L->y = y;
    L->P = P;
    L->blk_m = blk_m;
    L->blk_s = blk_s;
    L->blk_i = blk_i;
    L->fout = fout;
    L->alpha = alpha;
    L->ref = ref;
    L->zt = zt;
    L->runM = runM;
    L->runS = runS;
    L->runA = runA;
    L->G = G;
  }
  return c.off;
}

int check_oe_desc(const fpo_oe_desc* d) {
  if (!d) return fail(FPO_ERR_NULL, "fpo_output_error: desc is NULL");
  if (d->dtype != FPO_F32 && d->dtype != FPO_BF16)
    return fail(FPO_ERR_DTYPE, "fpo_output_error: unknown dtype %d", (int)d->dtype);
  if (d->T <= 0 || d->d <= 0 || d->V <= 0 || d->T > kIntMax || d->d > kIntMax || d->V > kIntMax)
    return fail(FPO_ERR_SHAPE, "fpo_output_error: sizes must be in [1, 2^31): T=%lld d=%lld V=%lld",
                (long long)d->T, (long long)d->d, (long long)d->V);
  if (d->d % 8 || d->V % 8)
    return fail(FPO_ERR_SHAPE, "fpo_output_error: d and V must be multiples of 8 (d=%lld V=%lld)",
                (long long)d->d, (long long)d->V);
  if (d->T > kMaxTokens)
    return fail(FPO_ERR_SHAPE, "fpo_output_error: at most %lld tokens per call (T=%lld)", (long long)kMaxTokens,
                (long long)d->T);
  if (!(d->eps >= 0.f) || !std::isfinite(d->eps))
    return fail(FPO_ERR_ARG, "fpo_output_error: eps must be finite and >= 0");
  if (!(d->min_rms >= 0.f) || !std::isfinite(d->min_rms))
    return fail(FPO_ERR_ARG, "fpo_output_error: min_rms must be finite and >= 0");
  if (d->vocab_chunk < 0) return fail(FPO_ERR_ARG, "fpo_output_error: vocab_chunk must be >= 0");
  // bf16 operands are copied through 32-bit buffer offsets: every operand band
  // (y, a W_U chunk of at least 256 rows, the staged p~) must fit in 2^31 bytes
  if (d->dtype == FPO_BF16 && (!band_fits(d->T, d->d) || !band_fits(256, d->d) || !band_fits(d->T, 256 + 128)))
    return fail(FPO_ERR_UNSUPPORTED,
                "fpo_output_error: bf16 operand bands must stay below 2^31 bytes (T*d, 256*d and 384*T "
                "elements <= 2^30; T=%lld d=%lld)",
                (long long)d->T, (long long)d->d);
  return FPO_OK;
}

struct PgPlan {
  int64_t Tp = 0, ntiles = 0, upd_blocks = 0;
  int nmats = 0;
};

PgPlan plan_pg(const fpo_pg_desc& d) {
  PgPlan p;
  const bool bf16 = d.dtype == FPO_BF16;
  p.Tp = round_up(d.T, 64);
  p.ntiles = fpo::pseudograd_tiles(bf16, d.d, d.d_ff);
  const bool full = (d.mode & FPO_MODE_FULL_MLP) != 0;
  p.nmats = (int)(full ? 3 * d.L : d.L);
  p.upd_blocks = p.nmats * fpo::update_blocks(d.d * d.d_ff);
  return p;
}

size_t carve_pg(const fpo_pg_desc& d, const PgPlan& p, void* ws, fpo::PgLaunch* L,
                double** upd_part, double** upd_dsq = nullptr) {
  const int64_t esz = d.dtype == FPO_BF16 ? 2 : 4;
  const bool full = (d.mode & FPO_MODE_FULL_MLP) != 0;
  const bool chain = (d.mode & (FPO_MODE_POST_FFN | FPO_MODE_PRE_MLP)) != 0;
  Carver c(ws);
  // token-contiguous left operand(s): shared, or one per layer (norm chain)
  void* gT = c.take<char>((chain ? d.L : 1) * d.d * p.Tp * esz);
  // norm chain + full-MLP: each layer's signal row-major too (error GEMM operand)
  void* grow = (chain && full) ? c.take<char>(d.L * d.T * d.d * esz) : nullptr;
  float* pstats = chain ? c.take<float>(4 * d.T) : nullptr;  // per-token norm-chain statistics
  void* dq = full ? c.take<char>(d.d_ff * p.Tp * esz) : nullptr;
  void* du = full ? c.take<char>(d.d_ff * p.Tp * esz) : nullptr;
  // tile partials: a region per matrix (3 L with the full MLP: the overlapped
  // update reduces each matrix's partials while later launches run)
  double* part = c.take<double>((full ? 3 * d.L : std::max<int64_t>(d.L, 2)) * p.ntiles * 3);
  double* up = c.take<double>(p.upd_blocks);
  double* dsq = c.take<double>(p.nmats);  // ||delta||^2 per matrix (clip-the-update mode)
  // staged bf16 pseudogradients (FPO_MODE_GRAD_BF16), one 256-aligned matrix per layer
  const bool stage = (d.mode & FPO_MODE_GRAD_BF16) != 0;
  for (int64_t l = 0; l < (stage ? d.L : 0); ++l) {
    uint16_t* sl = c.take<uint16_t>(d.d * d.d_ff);
    if (L) L->dW3_bf16[l] = sl;
  }
  if (L) {
    L->gT = gT;
    L->g_row = grow;
    L->chain_stats = pstats;
    L->dq_T = dq;
    L->du_T = du;
    L->part = part;
  }
  if (upd_part) *upd_part = up;
  if (upd_dsq) *upd_dsq = dsq;
  return c.off;
}

int check_pg_desc(const fpo_pg_desc* d) {
  if (!d) return fail(FPO_ERR_NULL, "fpo_pseudograd: desc is NULL");
  if (d->dtype != FPO_F32 && d->dtype != FPO_BF16)
    return fail(FPO_ERR_DTYPE, "fpo_pseudograd: unknown dtype %d", (int)d->dtype);
  if (d->mode < 0 || d->mode > (FPO_MODE_FULL_MLP | FPO_MODE_POST_FFN | FPO_MODE_GRAD_BF16 | FPO_MODE_PRE_MLP))
    return fail(FPO_ERR_ARG, "fpo_pseudograd: unknown mode %d", (int)d->mode);
  if ((d->mode & FPO_MODE_GRAD_BF16) && (d->dtype != FPO_BF16 || (d->mode & FPO_MODE_FULL_MLP)))
    return fail(FPO_ERR_UNSUPPORTED,
                "fpo_pseudograd: FPO_MODE_GRAD_BF16 is implemented for the W3-only FPO_BF16 path");
  if (d->T <= 0 || d->d <= 0 || d->d_ff <= 0 || d->L <= 0 || d->T > kIntMax || d->d > kIntMax ||
      d->d_ff > kIntMax)
    return fail(FPO_ERR_SHAPE, "fpo_pseudograd: sizes must be in [1, 2^31): T=%lld d=%lld d_ff=%lld L=%lld",
                (long long)d->T, (long long)d->d, (long long)d->d_ff, (long long)d->L);
  if (d->L > fpo::kMaxMats)
    return fail(FPO_ERR_SHAPE, "fpo_pseudograd: at most %d layers per call (L=%lld)", fpo::kMaxMats,
                (long long)d->L);
  if (d->d % 8 || d->d_ff % 8)
    return fail(FPO_ERR_SHAPE, "fpo_pseudograd: d and d_ff must be multiples of 8");
  if (d->T > kMaxTokens || d->d > kMaxHidden)
    return fail(FPO_ERR_SHAPE, "fpo_pseudograd: at most %lld tokens and d <= %lld per call (T=%lld d=%lld)",
                (long long)kMaxTokens, (long long)kMaxHidden, (long long)d->T, (long long)d->d);
  if (!std::isfinite(d->scale)) return fail(FPO_ERR_ARG, "fpo_pseudograd: scale must be finite");
  if (d->dtype == FPO_BF16) {
    // operand bands copied through 32-bit buffer offsets must fit in 2^31 bytes
    const int64_t Tp = round_up(d->T, 64);
    bool ok = band_fits(d->d, Tp) && band_fits(d->T, d->d_ff);
    if (d->mode & FPO_MODE_FULL_MLP)
      ok = ok && band_fits(d->T, d->d) && band_fits(d->d, d->d_ff) && band_fits(d->d_ff, Tp);
    if (!ok)
      return fail(FPO_ERR_UNSUPPORTED,
                  "fpo_pseudograd: bf16 operand bands must stay below 2^31 bytes (T=%lld d=%lld d_ff=%lld)",
                  (long long)d->T, (long long)d->d, (long long)d->d_ff);
  }
  return FPO_OK;
}

int check_opt(const fpo_opt* o) {
  if (!o) return fail(FPO_ERR_NULL, "optimizer description is NULL");
  if (o->kind != FPO_OPT_SGD && o->kind != FPO_OPT_ADAMW)
    return fail(FPO_ERR_ARG, "unknown optimizer kind %d", (int)o->kind);
  if (!(o->lr >= 0.0) || !std::isfinite(o->lr)) return fail(FPO_ERR_ARG, "lr must be finite and >= 0");
  if (o->step < 1) return fail(FPO_ERR_ARG, "step is 1-based (got %lld)", (long long)o->step);
  if (o->clip_target != FPO_CLIP_GRADIENT && o->clip_target != FPO_CLIP_UPDATE)
    return fail(FPO_ERR_ARG, "unknown clip_target %d", (int)o->clip_target);
  if (!std::isfinite(o->clip_frac)) return fail(FPO_ERR_ARG, "clip_frac must be finite");
  if (o->kind == FPO_OPT_SGD && !(o->momentum >= 0.0 && o->momentum <= 1.0))
    return fail(FPO_ERR_ARG, "momentum must be in [0, 1]");
  if (o->kind == FPO_OPT_ADAMW) {
    if (!(o->beta1 >= 0.0 && o->beta1 < 1.0) || !(o->beta2 >= 0.0 && o->beta2 < 1.0))
      return fail(FPO_ERR_ARG, "AdamW betas must be in [0, 1)");
    if (!(o->adam_eps > 0.0)) return fail(FPO_ERR_ARG, "AdamW eps must be > 0");
    if (!(o->weight_decay >= 0.0)) return fail(FPO_ERR_ARG, "weight_decay must be >= 0");
  }
  return FPO_OK;
}

int check_ws(void* ws, size_t have, size_t need, const char* who) {
  if (need == 0) return FPO_OK;
  if (!ws) return fail(FPO_ERR_WORKSPACE, "%s: workspace is NULL (%zu bytes needed)", who, need);
  if (!aligned(ws, kAlign)) return fail(FPO_ERR_WORKSPACE, "%s: workspace not 256-byte aligned", who);
  if (have < need)
    return fail(FPO_ERR_WORKSPACE, "%s: workspace %zu bytes < %zu needed", who, have, need);
  return FPO_OK;
}

int fill_update(const fpo_opt* opt, int64_t n, const int64_t* numel, const void* const* grad,
                const double* grad_sumsq, const fpo_update_bufs* upd, int32_t lp_dtype,
                fpo::UpdLaunch* U) {
  if (int e = check_opt(opt)) return e;
  if (!upd) return fail(FPO_ERR_NULL, "update buffers are NULL");
  if (n <= 0 || n > fpo::kMaxMats) return fail(FPO_ERR_SHAPE, "n_mats must be in [1, %d]", fpo::kMaxMats);
  // state1 may be absent only for plain SGD (momentum 0): no state is kept
  const bool stateless_ok = opt->kind == FPO_OPT_SGD && opt->momentum == 0.0;
  if (!numel || !grad || !grad_sumsq || !upd->W_master || !upd->W_sumsq || (!upd->state1 && !stateless_ok))
    return fail(FPO_ERR_NULL,
                "update: numel, grad, grad_sumsq, W_master, W_sumsq and state1 (unless SGD with momentum 0) "
                "are required");
  if (opt->kind == FPO_OPT_ADAMW && !upd->state2)
    return fail(FPO_ERR_NULL, "update: AdamW needs state2");
  if (lp_dtype != FPO_F32 && lp_dtype != FPO_BF16)
    return fail(FPO_ERR_DTYPE, "update: unknown low-precision dtype %d", (int)lp_dtype);
  U->kind = opt->kind;
  U->lr = opt->lr;
  U->momentum = opt->momentum;
  U->beta1 = opt->beta1;
  U->beta2 = opt->beta2;
  U->adam_eps = opt->adam_eps;
  U->weight_decay = opt->weight_decay;
  U->clip_frac = opt->clip_frac;
  U->step = opt->step;
  U->clip_update = opt->clip_target == FPO_CLIP_UPDATE;
  U->n = (int)n;
  U->lp_bf16 = lp_dtype == FPO_BF16;
  for (int64_t m = 0; m < n; ++m) {
    if (numel[m] <= 0 || numel[m] % 4)
      return fail(FPO_ERR_SHAPE, "update: numel[%lld]=%lld must be a positive multiple of 4",
                  (long long)m, (long long)numel[m]);
    float* s1m = upd->state1 ? upd->state1[m] : nullptr;
    if (!grad[m] || !upd->W_master[m] || (!s1m && !stateless_ok) ||
        (opt->kind == FPO_OPT_ADAMW && !upd->state2[m]))
      return fail(FPO_ERR_NULL, "update: NULL buffer for matrix %lld", (long long)m);
    const void* lpm = upd->W_lp ? upd->W_lp[m] : nullptr;
    const float* s2m = upd->state2 ? upd->state2[m] : nullptr;
    if (!aligned(grad[m], 16) || !aligned(upd->W_master[m], 16) || (s1m && !aligned(s1m, 16)) ||
        (s2m && !aligned(s2m, 16)) || (lpm && !aligned(lpm, U->lp_bf16 ? 8 : 16)))
      return fail(FPO_ERR_ARG, "update: buffers of matrix %lld must be 16-byte aligned (bf16 W_lp: 8)",
                  (long long)m);
    U->numel[m] = numel[m];
    U->grad[m] = grad[m];
    U->W[m] = upd->W_master[m];
    U->W_lp[m] = upd->W_lp ? upd->W_lp[m] : nullptr;
    U->s1[m] = s1m;
    U->s2[m] = upd->state2 ? upd->state2[m] : nullptr;
  }
  U->grad_sumsq = grad_sumsq;
  U->W_sumsq = upd->W_sumsq;
  U->clip_scale = upd->clip_scale;
  return FPO_OK;
}

// per-block partials, then n doubles of ||delta||^2 (clip-the-update mode)
size_t update_ws(int64_t n, const int64_t* numel) {
  int64_t blocks = 0;
  for (int64_t m = 0; m < n; ++m) blocks += fpo::update_blocks(numel[m]);
  return (size_t)(round_up(blocks * 8, kAlign) + round_up(n * 8, kAlign));
}

constexpr int kMaxScratchDevices = 64;
struct DeviceScratch {
  std::once_flag once;
  hipError_t err = hipSuccess;
  void* ptr = nullptr;
};
DeviceScratch g_scratch[kMaxScratchDevices];

// Address of the current device's copy of `scratch` (resolved on the first
// call on that device), or an error.
hipError_t scratch_address(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxScratchDevices) return hipErrorInvalidDevice;
  DeviceScratch& s = g_scratch[dev];
  std::call_once(s.once, [&s] { s.err = hipGetSymbolAddress(&s.ptr, HIP_SYMBOL(scratch)); });
  if (s.err != hipSuccess) return s.err;
  if (!s.ptr) return hipErrorInvalidSymbol;
  *out = s.ptr;
  return hipSuccess;
}

}  // namespace

extern "C" {

int fpo_abi_version(void) { return FPO_ABI_VERSION; }

const char* fpo_last_error(void) { return g_err.c_str(); }

size_t fpo_output_error_workspace(const fpo_oe_desc* desc) {
  if (check_oe_desc(desc)) return 0;
  return carve_oe(*desc, plan_oe(*desc), nullptr, nullptr);
}

int fpo_output_error(const fpo_oe_desc* desc, const void* h_final, const void* gamma,
                     const void* W_U, const int32_t* targets, float* g_tilde, void* g_tilde_lp,
                     float* g_pre, float* lse, float* loss, int32_t* argmax, int32_t* bad_targets,
                     void* ws, size_t ws_bytes, void* stream) {
  if (int e = check_oe_desc(desc)) return e;
  if (!h_final || !gamma || !W_U || !targets || !g_tilde)
    return fail(FPO_ERR_NULL, "fpo_output_error: h_final, gamma, W_U, targets and g_tilde are required");
  const void* ptrs[] = {h_final, gamma, W_U, g_tilde, g_tilde_lp, g_pre};
  for (const void* p : ptrs)
    if (p && !aligned(p, 16)) return fail(FPO_ERR_ARG, "fpo_output_error: tensors must be 16-byte aligned");
  const OePlan p = plan_oe(*desc);
  const size_t need = carve_oe(*desc, p, nullptr, nullptr);
  if (int e = check_ws(ws, ws_bytes, need, "fpo_output_error")) return e;
  fpo::OeLaunch L{};
  L.bf16 = desc->dtype == FPO_BF16;
  L.T = desc->T;
  L.d = desc->d;
  L.V = desc->V;
  L.Vc = p.Vc;
  L.ldp = p.ldp;
  L.nchunk = p.nchunk;
  L.cw = p.cw;
  L.cq = p.cq;
  L.nwide = p.nwide;
  L.nsplit = p.nsplit;
  L.eps = desc->eps;
  L.min_rms = desc->min_rms;
  L.h_final = h_final;
  L.gamma = gamma;
  L.W_U = W_U;
  L.targets = targets;
  L.g_tilde = g_tilde;
  L.g_tilde_lp = g_tilde_lp;
  L.g_pre = g_pre;
  L.lse = lse;
  L.loss = loss;
  L.argmax = argmax;
  L.bad_targets = bad_targets;
  L.stream = stream;
  carve_oe(*desc, p, ws, &L);
  hipError_t e = fpo::launch_output_error(L);
  if (e != hipSuccess) return hip_fail(e, "fpo_output_error launch");
  return FPO_OK;
}

size_t fpo_pseudograd_workspace(const fpo_pg_desc* desc) {
  if (check_pg_desc(desc)) return 0;
  return carve_pg(*desc, plan_pg(*desc), nullptr, nullptr, nullptr);
}

int fpo_pseudograd(const fpo_pg_desc* desc, const void* g_tilde_lp, const void* const* a,
                   const void* const* W3_init, const void* const* gate, const void* const* up,
                   const void* const* x_in, float* const* dW3, float* const* dW1, float* const* dW2,
                   double* sumsq, const float* const* ref, double* ref_dot, double* ref_sumsq,
                   float* ref_cos, const fpo_post_ffn* post_ffn, const fpo_pre_mlp* pre_mlp,
                   const fpo_opt* opt, const fpo_update_bufs* upd, const fpo_overlap* overlap, void* ws,
                   size_t ws_bytes, void* stream) {
  if (int e = check_pg_desc(desc)) return e;
  const bool full = (desc->mode & FPO_MODE_FULL_MLP) != 0;
  const bool pffn = (desc->mode & FPO_MODE_POST_FFN) != 0;
  const bool pre = (desc->mode & FPO_MODE_PRE_MLP) != 0;
  const int L = (int)desc->L;
  if (!a) return fail(FPO_ERR_NULL, "fpo_pseudograd: a is required");
  if (pffn != (post_ffn != nullptr))
    return fail(FPO_ERR_ARG, "fpo_pseudograd: post_ffn must be given exactly when mode has FPO_MODE_POST_FFN");
  if (pre != (pre_mlp != nullptr))
    return fail(FPO_ERR_ARG, "fpo_pseudograd: pre_mlp must be given exactly when mode has FPO_MODE_PRE_MLP");
  if (!g_tilde_lp && !post_ffn && !pre_mlp)
    return fail(FPO_ERR_NULL, "fpo_pseudograd: g_tilde_lp is required (unless post_ffn or pre_mlp is given)");
  if (pre_mlp) {
    if (!pre_mlp->g_tilde || !pre_mlp->x || !pre_mlp->gamma)
      return fail(FPO_ERR_NULL, "fpo_pseudograd: pre_mlp needs g_tilde, x and gamma");
    if (post_ffn && post_ffn->g_tilde != pre_mlp->g_tilde)
      return fail(FPO_ERR_ARG, "fpo_pseudograd: post_ffn and pre_mlp must name the same g_tilde");
    if (!aligned(pre_mlp->g_tilde, 16)) return fail(FPO_ERR_ARG, "fpo_pseudograd: pre_mlp->g_tilde not aligned");
    if (!(pre_mlp->eps >= 0.f) || !std::isfinite(pre_mlp->eps) || !(pre_mlp->min_rms >= 0.f) ||
        !std::isfinite(pre_mlp->min_rms))
      return fail(FPO_ERR_ARG, "fpo_pseudograd: pre_mlp eps and min_rms must be finite and >= 0");
    for (int l = 0; l < L; ++l) {
      if (!pre_mlp->x[l] || !pre_mlp->gamma[l])
        return fail(FPO_ERR_NULL, "fpo_pseudograd: pre_mlp buffers of layer %d are NULL", l);
      if (!aligned(pre_mlp->x[l], 16) || !aligned(pre_mlp->gamma[l], 16))
        return fail(FPO_ERR_ARG, "fpo_pseudograd: pre_mlp buffers of layer %d not 16-byte aligned", l);
    }
  }
  if (post_ffn) {
    if (!post_ffn->g_tilde || !post_ffn->mlp_out || !post_ffn->gamma)
      return fail(FPO_ERR_NULL, "fpo_pseudograd: post_ffn needs g_tilde, mlp_out and gamma");
    if (!aligned(post_ffn->g_tilde, 16)) return fail(FPO_ERR_ARG, "fpo_pseudograd: post_ffn->g_tilde not aligned");
    if (!(post_ffn->eps >= 0.f) || !std::isfinite(post_ffn->eps) || !(post_ffn->min_rms >= 0.f) ||
        !std::isfinite(post_ffn->min_rms))
      return fail(FPO_ERR_ARG, "fpo_pseudograd: post_ffn eps and min_rms must be finite and >= 0");
    for (int l = 0; l < L; ++l) {
      if (!post_ffn->mlp_out[l] || !post_ffn->gamma[l])
        return fail(FPO_ERR_NULL, "fpo_pseudograd: post_ffn buffers of layer %d are NULL", l);
      if (!aligned(post_ffn->mlp_out[l], 16) || !aligned(post_ffn->gamma[l], 16))
        return fail(FPO_ERR_ARG, "fpo_pseudograd: post_ffn buffers of layer %d not 16-byte aligned", l);
    }
  }
  const bool stage = (desc->mode & FPO_MODE_GRAD_BF16) != 0;
  if (stage && (dW3 || !opt))
    return fail(FPO_ERR_ARG, "fpo_pseudograd: FPO_MODE_GRAD_BF16 needs dW3 == NULL and the fused update");
  if (!dW3 && !ref && !stage) return fail(FPO_ERR_NULL, "fpo_pseudograd: dW3 may be NULL only with ref");
  if (ref && (!ref_dot || !ref_sumsq))
    return fail(FPO_ERR_NULL, "fpo_pseudograd: ref needs ref_dot and ref_sumsq");
  if (ref_cos && !ref) return fail(FPO_ERR_ARG, "fpo_pseudograd: ref_cos needs ref");
  if (overlap && (!overlap->side_stream || !overlap->ready_event || !overlap->done_event))
    return fail(FPO_ERR_NULL, "fpo_pseudograd: overlap needs side_stream, ready_event and done_event");
  if (full && (!W3_init || !gate || !up || !x_in || !dW1 || !dW2))
    return fail(FPO_ERR_NULL, "fpo_pseudograd: full-MLP mode needs W3_init, gate, up, x_in, dW1, dW2");
  if ((opt == nullptr) != (upd == nullptr))
    return fail(FPO_ERR_ARG, "fpo_pseudograd: opt and upd must both be given or both be NULL");
  if (opt && ((!dW3 && !stage) || !sumsq))
    return fail(FPO_ERR_NULL, "fpo_pseudograd: the fused update needs dW3 (or FPO_MODE_GRAD_BF16) and sumsq");
  if (g_tilde_lp && !aligned(g_tilde_lp, 16))
    return fail(FPO_ERR_ARG, "fpo_pseudograd: g_tilde_lp must be 16-byte aligned");
  fpo::PgLaunch P{};
  P.bf16 = desc->dtype == FPO_BF16;
  P.full_mlp = full;
  P.T = desc->T;
  P.d = desc->d;
  P.d_ff = desc->d_ff;
  P.L = L;
  P.scale = desc->scale;
  P.g_lp = g_tilde_lp;
  for (int l = 0; l < L; ++l) {
    if (!a[l]) return fail(FPO_ERR_NULL, "fpo_pseudograd: a[%d] is NULL", l);
    if (!aligned(a[l], 16)) return fail(FPO_ERR_ARG, "fpo_pseudograd: a[%d] not 16-byte aligned", l);
    P.a[l] = a[l];
    P.dW3[l] = dW3 ? dW3[l] : nullptr;
    if (dW3 && !dW3[l]) return fail(FPO_ERR_NULL, "fpo_pseudograd: dW3[%d] is NULL", l);
    if (P.dW3[l] && !aligned(P.dW3[l], 16)) return fail(FPO_ERR_ARG, "fpo_pseudograd: dW3[%d] not aligned", l);
    P.ref[l] = ref ? ref[l] : nullptr;
    if (ref && !ref[l]) return fail(FPO_ERR_NULL, "fpo_pseudograd: ref[%d] is NULL", l);
    if (ref && !aligned(ref[l], 16)) return fail(FPO_ERR_ARG, "fpo_pseudograd: ref[%d] not 16-byte aligned", l);
    if (full) {
      if (!W3_init[l] || !gate[l] || !up[l] || !x_in[l] || !dW1[l] || !dW2[l])
        return fail(FPO_ERR_NULL, "fpo_pseudograd: full-MLP buffer of layer %d is NULL", l);
      if (!aligned(W3_init[l], 16) || !aligned(gate[l], 16) || !aligned(up[l], 16) || !aligned(x_in[l], 16) ||
          !aligned(dW1[l], 16) || !aligned(dW2[l], 16))
        return fail(FPO_ERR_ARG, "fpo_pseudograd: full-MLP buffers of layer %d must be 16-byte aligned", l);
      P.W3i[l] = W3_init[l];
      P.q[l] = gate[l];
      P.u[l] = up[l];
      P.x_in[l] = x_in[l];
      P.dW1[l] = dW1[l];
      P.dW2[l] = dW2[l];
    }
  }
  if (post_ffn) {
    P.pffn = true;
    P.g_f32 = post_ffn->g_tilde;
    P.pffn_eps = post_ffn->eps;
    P.pffn_min_rms = post_ffn->min_rms;
    for (int l = 0; l < L; ++l) {
      P.mlp_out[l] = post_ffn->mlp_out[l];
      P.gamma_pffn[l] = post_ffn->gamma[l];
    }
  }
  if (pre_mlp) {
    P.pre = true;
    P.g_f32 = pre_mlp->g_tilde;
    P.pre_eps = pre_mlp->eps;
    P.pre_min_rms = pre_mlp->min_rms;
    for (int l = 0; l < L; ++l) {
      P.pre_in[l] = pre_mlp->x[l];
      P.gamma_pre[l] = pre_mlp->gamma[l];
    }
  }
  P.sumsq = sumsq;
  P.ref_dot = ref_dot;
  P.ref_sumsq = ref_sumsq;
  P.ref_cos = ref_cos;
  P.stream = stream;
  const PgPlan pl = plan_pg(*desc);
  P.Tp = pl.Tp;
  const size_t need = carve_pg(*desc, pl, nullptr, nullptr, nullptr);
  if (int e = check_ws(ws, ws_bytes, need, "fpo_pseudograd")) return e;
  double* upart = nullptr;
  double* udsq = nullptr;
  carve_pg(*desc, pl, ws, &P, &upart, &udsq);
  fpo::UpdLaunch U{};
  if (opt) {
    const int n = pl.nmats;
    if (n > fpo::kMaxMats) return fail(FPO_ERR_SHAPE, "fpo_pseudograd: fused update limited to %d matrices", fpo::kMaxMats);
    int64_t numel[fpo::kMaxMats];
    const void* grads[fpo::kMaxMats];
    for (int m = 0; m < n; ++m) {
      const int l = m % L, kind = m / L;
      numel[m] = desc->d * desc->d_ff;
      grads[m] = stage ? (const void*)P.dW3_bf16[l] : kind == 0 ? dW3[l] : (kind == 1 ? dW1[l] : dW2[l]);
    }
    if (int e = fill_update(opt, n, numel, grads, sumsq, upd, desc->dtype, &U)) return e;
    U.grad_bf16 = stage;
    U.part = upart;
    U.dsq = udsq;
    U.stream = stream;
  }
  hipError_t e;
  if (opt && P.bf16 && !U.clip_update) {
    // bf16, gradient clip: each matrix's update overlaps the GEMM launches
    // that follow its outer products (clip-the-update needs every step's norm
    // first: two passes after the pseudogradient)
    fpo::OverlapLaunch ov{};
    if (overlap) ov = fpo::OverlapLaunch{overlap->side_stream, overlap->ready_event, overlap->done_event};
    e = fpo::launch_pseudograd_update(P, U, overlap ? &ov : nullptr);
    if (e != hipSuccess) return hip_fail(e, "fpo_pseudograd overlapped launch");
    return FPO_OK;
  }
  e = fpo::launch_pseudograd(P);
  if (e != hipSuccess) return hip_fail(e, "fpo_pseudograd launch");
  if (opt) {
    e = fpo::launch_update(U);
    if (e != hipSuccess) return hip_fail(e, "fpo_pseudograd update launch");
  }
  return FPO_OK;
}

size_t fpo_apply_update_workspace(int64_t n_mats, const int64_t* numel) {
  if (n_mats <= 0 || !numel) return 0;
  return update_ws(n_mats, numel);
}

int fpo_apply_update(const fpo_opt* opt, int64_t n_mats, const int64_t* numel,
                     const float* const* grad, const double* grad_sumsq,
                     const fpo_update_bufs* upd, int32_t lp_dtype, void* ws, size_t ws_bytes,
                     void* stream) {
  fpo::UpdLaunch U{};
  if (int e = fill_update(opt, n_mats, numel, (const void* const*)grad, grad_sumsq, upd, lp_dtype, &U))
    return e;
  if (int e = check_ws(ws, ws_bytes, update_ws(n_mats, numel), "fpo_apply_update")) return e;
  U.part = (double*)ws;
  int64_t blocks = 0;
  for (int64_t m = 0; m < n_mats; ++m) blocks += fpo::update_blocks(numel[m]);
  U.dsq = (double*)((char*)ws + round_up(blocks * 8, kAlign));
  U.stream = stream;
  hipError_t e = fpo::launch_update(U);
  if (e != hipSuccess) return hip_fail(e, "fpo_apply_update launch");
  return FPO_OK;
}

int fpo_apply_update_noalloc(const fpo_opt* opt, int64_t n_mats, const int64_t* numel,
                             const float* const* grad, const double* grad_sumsq,
                             const fpo_update_bufs* upd, int32_t lp_dtype, void* stream) {
  fpo::UpdLaunch U{};
  if (int e = fill_update(opt, n_mats, numel, (const void* const*)grad, grad_sumsq, upd, lp_dtype, &U))
    return e;
  // the same scratch layout as fpo_apply_update's workspace, bounded by the array
  const size_t need = update_ws(n_mats, numel);
  if (need > (size_t)FPO_NOALLOC_SCRATCH_BYTES)
    return fail(FPO_ERR_WORKSPACE,
                "fpo_apply_update_noalloc: these matrices need %zu bytes of scratch (8 per 4096 parameters), "
                "the library's static array holds %zu; split the call or use fpo_apply_update",
                need, (size_t)FPO_NOALLOC_SCRATCH_BYTES);
  void* ws = nullptr;
  if (hipError_t e = scratch_address(&ws)) return hip_fail(e, "fpo_apply_update_noalloc scratch address");
  U.part = (double*)ws;
  int64_t blocks = 0;
  for (int64_t m = 0; m < n_mats; ++m) blocks += fpo::update_blocks(numel[m]);
  U.dsq = (double*)((char*)ws + round_up(blocks * 8, kAlign));
  U.stream = stream;
  hipError_t e = fpo::launch_update(U);
  if (e != hipSuccess) return hip_fail(e, "fpo_apply_update_noalloc launch");
  return FPO_OK;
}

size_t fpo_cosine_workspace(int64_t n_pairs, const int64_t* numel) {
  if (n_pairs <= 0 || !numel) return 0;
  int64_t blocks = 0;
  for (int64_t m = 0; m < n_pairs; ++m) blocks += fpo::cosine_blocks(numel[m]);
  return (size_t)round_up(blocks * 3 * 8, kAlign);
}

int fpo_cosine(int64_t n_pairs, const int64_t* numel, const float* const* A, const void* const* B,
               int32_t dtype_B, double* dot, double* sumsq_A, double* sumsq_B, float* cos,
               void* ws, size_t ws_bytes, void* stream) {
  if (n_pairs <= 0 || n_pairs > fpo::kMaxMats)
    return fail(FPO_ERR_SHAPE, "fpo_cosine: n_pairs must be in [1, %d]", fpo::kMaxMats);
  if (!numel || !A) return fail(FPO_ERR_NULL, "fpo_cosine: numel and A are required");
  if (dtype_B != FPO_F32 && dtype_B != FPO_BF16)
    return fail(FPO_ERR_DTYPE, "fpo_cosine: unknown dtype %d", (int)dtype_B);
  fpo::CosLaunch C{};
  C.n = (int)n_pairs;
  C.b_bf16 = dtype_B == FPO_BF16;
  for (int64_t m = 0; m < n_pairs; ++m) {
    if (numel[m] <= 0 || numel[m] % 4)
      return fail(FPO_ERR_SHAPE, "fpo_cosine: numel[%lld] must be a positive multiple of 4", (long long)m);
    if (!A[m] || (B && !B[m])) return fail(FPO_ERR_NULL, "fpo_cosine: NULL pointer for pair %lld", (long long)m);
    if (!aligned(A[m], 16) || (B && !aligned(B[m], 16)))
      return fail(FPO_ERR_ARG, "fpo_cosine: pair %lld not 16-byte aligned", (long long)m);
    C.numel[m] = numel[m];
    C.A[m] = A[m];
    C.B[m] = B ? B[m] : nullptr;
  }
  if (int e = check_ws(ws, ws_bytes, fpo_cosine_workspace(n_pairs, numel), "fpo_cosine")) return e;
  C.dot = dot;
  C.sa = sumsq_A;
  C.sb = sumsq_B;
  C.cos = cos;
  C.part = (double*)ws;
  C.stream = stream;
  hipError_t e = fpo::launch_cosine(C);
  if (e != hipSuccess) return hip_fail(e, "fpo_cosine launch");
  return FPO_OK;
}

}  // extern "C"
