// Relative clip + optimizer step on fp32 masters (App. A; Sec. 3.1 optimizers)
// and the cosine / norm reduction of the layer-viability diagnostic
// (eq. cosine). Both stream parameters once, are HBM bound, and reduce in a
// fixed order (per-workgroup float64 partials, then one workgroup per matrix)
// so results are bit-reproducible.
#include "common.hpp"
#include "launch.hpp"
#include "prof.hpp"
#include "upd.hpp"

namespace fpo {

constexpr int kUpdBatch = 32;        // matrices per launch (kernel-argument budget)

int64_t update_blocks(int64_t numel) { return (numel + kElemsPerBlock - 1) / kElemsPerBlock; }
int64_t cosine_blocks(int64_t numel) { return (numel + kElemsPerBlock - 1) / kElemsPerBlock; }

struct UpdArgs {
  const void* grad[kUpdBatch];  // float32, or bf16 (the kernels' GB16)
  float* W[kUpdBatch];
  void* W_lp[kUpdBatch];
  float* s1[kUpdBatch];
  float* s2[kUpdBatch];
  int64_t numel[kUpdBatch];
  int64_t blk0[kUpdBatch + 1];
};

__device__ __forceinline__ int find_mat(const int64_t* blk0, int n, int64_t b) {
  int m = 0;
  while (m + 1 < n && blk0[m + 1] <= b) ++m;
  return m;
}

template <bool GB16, bool ADAM>
__global__ __launch_bounds__(256) void update_kernel(UpdArgs a, int n, OptScalars o,
                                                     const double* __restrict__ grad_sumsq,
                                                     const double* __restrict__ W_sumsq,
                                                     double* __restrict__ part) {
  __shared__ double red[16];
  const int64_t b = blockIdx.x;
  const int m = find_mat(a.blk0, n, b);
  const float s = clip_factor(grad_sumsq[m], W_sumsq[m], o.clip_frac);
  update_visit<GB16, ADAM, 1>(a.grad[m], a.W[m], a.W_lp[m], a.s1[m], a.s2[m], a.numel[m], b - a.blk0[m], 1,
                               a.blk0[m + 1] - a.blk0[m], s, o, red, part + a.blk0[m]);
}

// The blocks of one matrix (a.blk0[1] of them) visited by a fixed number of
// workgroups, NB blocks per visit (block b and b + gridDim.x, ...): run beside
// the outer products, one workgroup per CU fits next to an outer-product
// workgroup (registers and LDS), so neither kernel waits for the other's waves
// to drain, and NB blocks' loads in flight per workgroup hide memory latency.
// Each block's result and partial are those of update_kernel, bit for bit.
template <bool GB16, bool ADAM, int NB>
__global__ __launch_bounds__(256) void update_loop_kernel(UpdArgs a, OptScalars o,
                                                          const double* __restrict__ grad_sumsq,
                                                          const double* __restrict__ W_sumsq,
                                                          double* __restrict__ part) {
  __shared__ double red[16];
  const int64_t nb = a.blk0[1];
  const float s = clip_factor(grad_sumsq[0], W_sumsq[0], o.clip_frac);
  for (int64_t b = blockIdx.x; b < nb; b += (int64_t)NB * gridDim.x)
    update_visit<GB16, ADAM, NB>(a.grad[0], a.W[0], a.W_lp[0], a.s1[0], a.s2[0], a.numel[0], b, gridDim.x, nb,
                                  s, o, red, part);
}

// Clip-the-update mode, pass 1 (one workgroup per block): new optimizer state
// and per-block ||delta||^2.
template <bool GB16, bool ADAM>
__global__ __launch_bounds__(256) void delta_kernel(UpdArgs a, int n, OptScalars o, double* __restrict__ part) {
  __shared__ double red[16];
  const int64_t b = blockIdx.x;
  const int m = find_mat(a.blk0, n, b);
  delta_block<GB16, ADAM>(a.grad[m], a.W[m], a.s1[m], a.s2[m], a.numel[m], b - a.blk0[m], o, red, part + b);
}

// Fixed-order sum of each matrix's block partials into out[m].
__global__ __launch_bounds__(256) void sum_parts_kernel(UpdArgs a, const double* __restrict__ part,
                                                        double* __restrict__ out) {
  __shared__ double red[16];
  const int m = blockIdx.x;
  const double acc = block_sum_d(strided_sum_d(part, a.blk0[m], a.blk0[m + 1]), red);
  if (threadIdx.x == 0) out[m] = acc;
}

// Clip-the-update mode, pass 2: W' = W + s * delta with
// s = min(1, clip_frac ||W|| / ||delta||), per-block ||W'||^2.
template <bool GB16, bool ADAM>
__global__ __launch_bounds__(256) void apply_kernel(UpdArgs a, int n, OptScalars o,
                                                    const double* __restrict__ dsq,
                                                    const double* __restrict__ W_sumsq,
                                                    double* __restrict__ part) {
  __shared__ double red[16];
  const int64_t b = blockIdx.x;
  const int m = find_mat(a.blk0, n, b);
  const float s = clip_factor(dsq[m], W_sumsq[m], o.clip_frac);
  apply_block<GB16, ADAM>(a.grad[m], a.W[m], a.W_lp[m], a.s1[m], a.s2[m], a.numel[m], b - a.blk0[m], s, o, red,
                          part + b);
}

__global__ __launch_bounds__(256) void update_reduce_kernel(UpdArgs a, OptScalars o,
                                                            const double* __restrict__ part,
                                                            const double* __restrict__ grad_sumsq,
                                                            double* __restrict__ W_sumsq,
                                                            float* __restrict__ clip_scale) {
  __shared__ double red[16];
  const int m = blockIdx.x;
  const double acc = block_sum_d(strided_sum_d(part, a.blk0[m], a.blk0[m + 1]), red);
  if (threadIdx.x == 0) {
    // the clip factor the update used, from the W_sumsq it read (grad_sumsq:
    // ||dW||^2, or ||delta||^2 in clip-the-update mode)
    if (clip_scale) clip_scale[m] = clip_factor(grad_sumsq[m], W_sumsq[m], o.clip_frac);
    W_sumsq[m] = acc;
  }
}

#define FPO_CHECK_LAUNCH()             \
  do {                                 \
    hipError_t e_ = hipGetLastError(); \
    if (e_ != hipSuccess) return e_;   \
  } while (0)

// update_kernel over nb blocks of the n matrices of ua, in the variant for the
// gradient dtype and optimizer.
static hipError_t launch_update_kernel(const UpdArgs& ua, int n, const OptScalars& o, bool gb16, bool adam,
                                       const double* gs, const double* ws, double* pt, unsigned nb,
                                       hipStream_t st) {
  const dim3 g(nb);
  if (gb16 && adam)
    FPO_LAUNCH("update", st, update_kernel<true, true><<<g, dim3(256), 0, st>>>(ua, n, o, gs, ws, pt));
  else if (gb16)
    FPO_LAUNCH("update", st, update_kernel<true, false><<<g, dim3(256), 0, st>>>(ua, n, o, gs, ws, pt));
  else if (adam)
    FPO_LAUNCH("update", st, update_kernel<false, true><<<g, dim3(256), 0, st>>>(ua, n, o, gs, ws, pt));
  else
    FPO_LAUNCH("update", st, update_kernel<false, false><<<g, dim3(256), 0, st>>>(ua, n, o, gs, ws, pt));
  FPO_CHECK_LAUNCH();
  return hipSuccess;
}

// The update blocks of matrix m alone (no reduction), on stream st; its
// partials start at part + blk_base, as in launch_update. grid > 0: that many
// workgroups visit the blocks grid-stride (update_loop_kernel).
hipError_t launch_update_blocks(const UpdLaunch& a, int m, int64_t blk_base, void* stream, int grid) {
  hipStream_t st = (hipStream_t)stream;
  const OptScalars o = make_opt_scalars(a);
  UpdArgs ua{};
  ua.grad[0] = a.grad[m];
  ua.W[0] = a.W[m];
  ua.W_lp[0] = a.W_lp[m];
  ua.s1[0] = a.s1[m];
  ua.s2[0] = a.s2[m];
  ua.numel[0] = a.numel[m];
  ua.blk0[0] = 0;
  ua.blk0[1] = update_blocks(a.numel[m]);
  const bool loop = grid > 0 && grid < ua.blk0[1];
  const double* gs = a.grad_sumsq + m;
  const double* ws = a.W_sumsq + m;
  double* pt = a.part + blk_base;
  const bool adam = a.kind == kOptAdamW;
  if (loop) {
    // SGD: two blocks per visit (128 VGPRs, still beside an outer-product
    // workgroup); AdamW's second moment leaves room for one
    const dim3 g((unsigned)grid);
    if (adam && a.grad_bf16)
      FPO_LAUNCH("update", st, update_loop_kernel<true, true, 1><<<g, dim3(256), 0, st>>>(ua, o, gs, ws, pt));
    else if (adam)
      FPO_LAUNCH("update", st, update_loop_kernel<false, true, 1><<<g, dim3(256), 0, st>>>(ua, o, gs, ws, pt));
    else if (a.grad_bf16)
      FPO_LAUNCH("update", st, update_loop_kernel<true, false, 2><<<g, dim3(256), 0, st>>>(ua, o, gs, ws, pt));
    else
      FPO_LAUNCH("update", st, update_loop_kernel<false, false, 2><<<g, dim3(256), 0, st>>>(ua, o, gs, ws, pt));
  } else {
    if (hipError_t e = launch_update_kernel(ua, 1, o, a.grad_bf16, adam, gs, ws, pt, (unsigned)ua.blk0[1], st))
      return e;
  }
  FPO_CHECK_LAUNCH();
  return hipSuccess;
}

hipError_t launch_update(const UpdLaunch& a, bool blocks) {
  hipStream_t st = (hipStream_t)a.stream;
  const OptScalars o = make_opt_scalars(a);
  int64_t part_off = 0;
  for (int m0 = 0; m0 < a.n; m0 += kUpdBatch) {
    const int n = std::min(kUpdBatch, a.n - m0);
    UpdArgs ua{};
    int64_t nb = 0;
    for (int k = 0; k < n; ++k) {
      const int m = m0 + k;
      ua.grad[k] = a.grad[m];
      ua.W[k] = a.W[m];
      ua.W_lp[k] = a.W_lp[m];
      ua.s1[k] = a.s1[m];
      ua.s2[k] = a.s2[m];
      ua.numel[k] = a.numel[m];
      ua.blk0[k] = nb;
      nb += update_blocks(a.numel[m]);
    }
    ua.blk0[n] = nb;
    const double* clip_ref = a.grad_sumsq + m0;
    if (a.clip_update) {
      const bool adam = a.kind == kOptAdamW, gb = a.grad_bf16;
      const dim3 g((unsigned)nb);
      double* pt = a.part + part_off;
      if (adam && gb) FPO_LAUNCH("update_delta", st, delta_kernel<true, true><<<g, dim3(256), 0, st>>>(ua, n, o, pt));
      else if (adam) FPO_LAUNCH("update_delta", st, delta_kernel<false, true><<<g, dim3(256), 0, st>>>(ua, n, o, pt));
      else if (gb) FPO_LAUNCH("update_delta", st, delta_kernel<true, false><<<g, dim3(256), 0, st>>>(ua, n, o, pt));
      else FPO_LAUNCH("update_delta", st, delta_kernel<false, false><<<g, dim3(256), 0, st>>>(ua, n, o, pt));
      FPO_CHECK_LAUNCH();
      FPO_LAUNCH("update_reduce", st, sum_parts_kernel<<<dim3(n), dim3(256), 0, st>>>(ua, pt, a.dsq + m0));
      FPO_CHECK_LAUNCH();
      const double* dq = a.dsq + m0;
      const double* ws = a.W_sumsq + m0;
      if (adam && gb) FPO_LAUNCH("update", st, apply_kernel<true, true><<<g, dim3(256), 0, st>>>(ua, n, o, dq, ws, pt));
      else if (adam) FPO_LAUNCH("update", st, apply_kernel<false, true><<<g, dim3(256), 0, st>>>(ua, n, o, dq, ws, pt));
      else if (gb) FPO_LAUNCH("update", st, apply_kernel<true, false><<<g, dim3(256), 0, st>>>(ua, n, o, dq, ws, pt));
      else FPO_LAUNCH("update", st, apply_kernel<false, false><<<g, dim3(256), 0, st>>>(ua, n, o, dq, ws, pt));
      FPO_CHECK_LAUNCH();
      clip_ref = a.dsq + m0;
    } else if (blocks) {
      if (hipError_t e = launch_update_kernel(ua, n, o, a.grad_bf16, a.kind == kOptAdamW,
                                              a.grad_sumsq + m0, a.W_sumsq + m0, a.part + part_off,
                                              (unsigned)nb, st))
        return e;
    }
    FPO_LAUNCH("update_reduce", st,
               update_reduce_kernel<<<dim3(n), dim3(256), 0, st>>>(ua, o, a.part + part_off, clip_ref,
                                                        a.W_sumsq + m0,
                                                        a.clip_scale ? a.clip_scale + m0 : nullptr));
    FPO_CHECK_LAUNCH();
    part_off += nb;
  }
  return hipSuccess;
}

// ------------------------------------------------------------------ cosine
struct CosArgs {
  const float* A[kUpdBatch];
  const void* B[kUpdBatch];
  int64_t numel[kUpdBatch];
  int64_t blk0[kUpdBatch + 1];
};

__global__ __launch_bounds__(256) void cosine_kernel(CosArgs a, int n, int b_bf16,
                                                     double* __restrict__ part) {
  __shared__ double red[16];
  const int64_t b = blockIdx.x;
  const int m = find_mat(a.blk0, n, b);
  const int64_t base = (b - a.blk0[m]) * kElemsPerBlock;
  const int64_t end = (a.numel[m] < base + kElemsPerBlock) ? a.numel[m] : base + kElemsPerBlock;
  const float* A = a.A[m];
  const void* B = a.B[m];
  constexpr int U = kElemsPerBlock / 1024;
  f32x4 xs[U], ys[U];
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int64_t i = base + threadIdx.x * 4 + u * 1024;
    xs[u] = ys[u] = f32x4{0.f, 0.f, 0.f, 0.f};
    if (i < end) {
      xs[u] = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(A + i));
      if (B) {
        if (b_bf16) {
          const u32x2 h = __builtin_nontemporal_load(reinterpret_cast<const u32x2*>((const uint16_t*)B + i));
          ys[u] = f32x4{bf16_lo(h.x), bf16_hi(h.x), bf16_lo(h.y), bf16_hi(h.y)};
        } else {
          ys[u] = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>((const float*)B + i));
        }
      }
    }
  }
  float dt = 0.f, sa = 0.f, sb = 0.f;
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const f32x4 x = xs[u], y = ys[u];  // zero outside the matrix
    sa += x.x * x.x + x.y * x.y + x.z * x.z + x.w * x.w;
    dt += x.x * y.x + x.y * y.y + x.z * y.z + x.w * y.w;
    sb += y.x * y.x + y.y * y.y + y.z * y.z + y.w * y.w;
  }
  const double d0 = block_sum_d((double)dt, red);
  const double d1 = block_sum_d((double)sa, red);
  const double d2 = block_sum_d((double)sb, red);
  if (threadIdx.x == 0) {
    part[3 * b] = d0;
    part[3 * b + 1] = d1;
    part[3 * b + 2] = d2;
  }
}

__global__ __launch_bounds__(256) void cosine_reduce_kernel(CosArgs a, const double* __restrict__ part,
                                                            double* __restrict__ dot,
                                                            double* __restrict__ sa,
                                                            double* __restrict__ sb,
                                                            float* __restrict__ cosv) {
  __shared__ double red[16];
  const int m = blockIdx.x;
  // two visits per iteration (six independent accumulators) keep loads in flight
  double x = 0.0, y = 0.0, z = 0.0, x1 = 0.0, y1 = 0.0, z1 = 0.0;
  int64_t b = a.blk0[m] + threadIdx.x;
  for (; b + 256 < a.blk0[m + 1]; b += 512) {
    x += part[3 * b];
    y += part[3 * b + 1];
    z += part[3 * b + 2];
    x1 += part[3 * (b + 256)];
    y1 += part[3 * (b + 256) + 1];
    z1 += part[3 * (b + 256) + 2];
  }
  for (; b < a.blk0[m + 1]; b += 256) {
    x += part[3 * b];
    y += part[3 * b + 1];
    z += part[3 * b + 2];
  }
  x += x1;
  y += y1;
  z += z1;
  x = block_sum_d(x, red);
  y = block_sum_d(y, red);
  z = block_sum_d(z, red);
  if (threadIdx.x == 0) {
    if (dot) dot[m] = x;
    if (sa) sa[m] = y;
    if (sb) sb[m] = z;
    if (cosv) cosv[m] = (y == 0.0 || z == 0.0) ? 0.f : (float)(x / sqrt(y * z));
  }
}

hipError_t launch_cosine(const CosLaunch& a) {
  hipStream_t st = (hipStream_t)a.stream;
  int64_t part_off = 0;
  for (int m0 = 0; m0 < a.n; m0 += kUpdBatch) {
    const int n = std::min(kUpdBatch, a.n - m0);
    CosArgs ca{};
    int64_t nb = 0;
    for (int k = 0; k < n; ++k) {
      ca.A[k] = a.A[m0 + k];
      ca.B[k] = a.B[m0 + k];
      ca.numel[k] = a.numel[m0 + k];
      ca.blk0[k] = nb;
      nb += cosine_blocks(a.numel[m0 + k]);
    }
    ca.blk0[n] = nb;
    FPO_LAUNCH("cosine", st,
               cosine_kernel<<<dim3((unsigned)nb), dim3(256), 0, st>>>(ca, n, a.b_bf16, a.part + 3 * part_off));
    FPO_CHECK_LAUNCH();
    FPO_LAUNCH("cosine_reduce", st,
               cosine_reduce_kernel<<<dim3(n), dim3(256), 0, st>>>(
        ca, a.part + 3 * part_off, a.dot ? a.dot + m0 : nullptr, a.sa ? a.sa + m0 : nullptr,
        a.sb ? a.sb + m0 : nullptr, a.cos ? a.cos + m0 : nullptr));
    FPO_CHECK_LAUNCH();
    part_off += nb;
  }
  return hipSuccess;
}

}  // namespace fpo
