// Relative clip + optimizer step on fp32 masters (App. A; Sec. 3.1 optimizers)
// and the cosine / norm reduction of the layer-viability diagnostic
// (eq. cosine). Both stream parameters once, are HBM bound, and reduce in a
// fixed order (per-workgroup float64 partials, then one workgroup per matrix)
// so results are bit-reproducible.
#include "common.hpp"
#include "launch.hpp"
#include "prof.hpp"

namespace fpo {

constexpr int kUpdBatch = 32;        // matrices per launch (kernel-argument budget)
constexpr int kElemsPerBlock = 4096;  // 256 threads x 4 x float4

int64_t update_blocks(int64_t numel) { return (numel + kElemsPerBlock - 1) / kElemsPerBlock; }
int64_t cosine_blocks(int64_t numel) { return (numel + kElemsPerBlock - 1) / kElemsPerBlock; }

struct UpdArgs {
  const float* grad[kUpdBatch];
  float* W[kUpdBatch];
  void* W_lp[kUpdBatch];
  float* s1[kUpdBatch];
  float* s2[kUpdBatch];
  int64_t numel[kUpdBatch];
  int64_t blk0[kUpdBatch + 1];
};

// Device copies of the hyperparameters: each derived factor is formed in double
// on the host and rounded once to float.
struct OptScalars {
  int kind, first, lp_bf16;
  float lr, momentum, beta1, one_m_beta1, beta2, one_m_beta2, adam_eps, decay;
  float inv_bc1, inv_sqrt_bc2;  // 1/(1-beta1^t), 1/sqrt(1-beta2^t)
  double clip_frac;
};

__device__ __forceinline__ int find_mat(const int64_t* blk0, int n, int64_t b) {
  int m = 0;
  while (m + 1 < n && blk0[m + 1] <= b) ++m;
  return m;
}

__device__ __forceinline__ float clip_factor(double gs, double ws, double frac) {
  if (frac <= 0.0 || gs == 0.0) return 1.0f;
  const double s = frac * sqrt(ws) / sqrt(gs);
  return (float)(s < 1.0 ? s : 1.0);
}

__global__ __launch_bounds__(256) void update_kernel(UpdArgs a, int n, OptScalars o,
                                                     const double* __restrict__ grad_sumsq,
                                                     const double* __restrict__ W_sumsq,
                                                     double* __restrict__ part) {
  __shared__ double red[16];
  const int64_t b = blockIdx.x;
  const int m = find_mat(a.blk0, n, b);
  const float s = clip_factor(grad_sumsq[m], W_sumsq[m], o.clip_frac);
  const int64_t base = (b - a.blk0[m]) * kElemsPerBlock;
  const int64_t end = (a.numel[m] < base + kElemsPerBlock) ? a.numel[m] : base + kElemsPerBlock;
  const float* g = a.grad[m];
  float* W = a.W[m];
  float* s1 = a.s1[m];
  float* s2 = a.s2[m];
  void* lp = a.W_lp[m];
  float ss = 0.f;
  for (int64_t i = base + threadIdx.x * 4; i < end; i += 1024) {
    f32x4 gv = *reinterpret_cast<const f32x4*>(g + i) * s;
    f32x4 w = *reinterpret_cast<const f32x4*>(W + i);
    if (o.kind == 0) {  // SGD with momentum
      f32x4 bv;
      if (o.first) {
        bv = gv;
      } else {
        f32x4 old = *reinterpret_cast<const f32x4*>(s1 + i);
        bv.x = fmaf(o.momentum, old.x, gv.x);
        bv.y = fmaf(o.momentum, old.y, gv.y);
        bv.z = fmaf(o.momentum, old.z, gv.z);
        bv.w = fmaf(o.momentum, old.w, gv.w);
      }
      *reinterpret_cast<f32x4*>(s1 + i) = bv;
      w.x = fmaf(-o.lr, bv.x, w.x);
      w.y = fmaf(-o.lr, bv.y, w.y);
      w.z = fmaf(-o.lr, bv.z, w.z);
      w.w = fmaf(-o.lr, bv.w, w.w);
    } else {  // AdamW, decoupled weight decay, bias corrected
      f32x4 mv = *reinterpret_cast<const f32x4*>(s1 + i);
      f32x4 vv = *reinterpret_cast<const f32x4*>(s2 + i);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float ge = gv[e];
        const float me = o.beta1 * mv[e] + o.one_m_beta1 * ge;
        const float ve = o.beta2 * vv[e] + o.one_m_beta2 * ge * ge;
        mv[e] = me;
        vv[e] = ve;
        const float denom = sqrtf(ve) * o.inv_sqrt_bc2 + o.adam_eps;
        w[e] = w[e] * o.decay - o.lr * (me * o.inv_bc1) / denom;
      }
      *reinterpret_cast<f32x4*>(s1 + i) = mv;
      *reinterpret_cast<f32x4*>(s2 + i) = vv;
    }
    *reinterpret_cast<f32x4*>(W + i) = w;
    if (lp) {
      if (o.lp_bf16)
        st4((uint16_t*)lp, i, w);
      else
        st4((float*)lp, i, w);
    }
    ss += w.x * w.x + w.y * w.y + w.z * w.z + w.w * w.w;
  }
  const double t = block_sum_d((double)ss, red);
  if (threadIdx.x == 0) part[b] = t;
}

__global__ __launch_bounds__(256) void update_reduce_kernel(UpdArgs a, OptScalars o,
                                                            const double* __restrict__ part,
                                                            const double* __restrict__ grad_sumsq,
                                                            double* __restrict__ W_sumsq,
                                                            float* __restrict__ clip_scale) {
  __shared__ double red[16];
  const int m = blockIdx.x;
  double acc = 0.0;
  for (int64_t b = a.blk0[m] + threadIdx.x; b < a.blk0[m + 1]; b += 256) acc += part[b];
  acc = block_sum_d(acc, red);
  if (threadIdx.x == 0) {
    // the clip factor used by update_kernel, from the W_sumsq it read
    if (clip_scale) clip_scale[m] = clip_factor(grad_sumsq[m], W_sumsq[m], o.clip_frac);
    W_sumsq[m] = acc;
  }
}

#define FPO_CHECK_LAUNCH()             \
  do {                                 \
    hipError_t e_ = hipGetLastError(); \
    if (e_ != hipSuccess) return e_;   \
  } while (0)

hipError_t launch_update(const UpdLaunch& a) {
  hipStream_t st = (hipStream_t)a.stream;
  OptScalars o{};
  o.kind = a.kind;
  o.first = a.step <= 1;
  o.lp_bf16 = a.lp_bf16;
  o.lr = (float)a.lr;
  o.momentum = (float)a.momentum;
  o.beta1 = (float)a.beta1;
  o.one_m_beta1 = (float)(1.0 - a.beta1);
  o.beta2 = (float)a.beta2;
  o.one_m_beta2 = (float)(1.0 - a.beta2);
  o.adam_eps = (float)a.adam_eps;
  o.decay = (float)(1.0 - a.lr * a.weight_decay);
  o.clip_frac = a.clip_frac;
  const double bc1 = 1.0 - pow(a.beta1, (double)a.step);
  const double bc2 = 1.0 - pow(a.beta2, (double)a.step);
  o.inv_bc1 = (float)(1.0 / bc1);
  o.inv_sqrt_bc2 = (float)(1.0 / sqrt(bc2));
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
    FPO_LAUNCH("update", st,
               update_kernel<<<dim3((unsigned)nb), dim3(256), 0, st>>>(ua, n, o, a.grad_sumsq + m0,
                                                          a.W_sumsq + m0, a.part + part_off));
    FPO_CHECK_LAUNCH();
    FPO_LAUNCH("update_reduce", st,
               update_reduce_kernel<<<dim3(n), dim3(256), 0, st>>>(ua, o, a.part + part_off,
                                                        a.grad_sumsq + m0, a.W_sumsq + m0,
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
  float dt = 0.f, sa = 0.f, sb = 0.f;
  for (int64_t i = base + threadIdx.x * 4; i < end; i += 1024) {
    f32x4 x = *reinterpret_cast<const f32x4*>(A + i);
    sa += x.x * x.x + x.y * x.y + x.z * x.z + x.w * x.w;
    if (B) {
      f32x4 y = b_bf16 ? ld4((const uint16_t*)B, i) : ld4((const float*)B, i);
      dt += x.x * y.x + x.y * y.y + x.z * y.z + x.w * y.w;
      sb += y.x * y.x + y.y * y.y + y.z * y.z + y.w * y.w;
    }
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
  double x = 0.0, y = 0.0, z = 0.0;
  for (int64_t b = a.blk0[m] + threadIdx.x; b < a.blk0[m + 1]; b += 256) {
    x += part[3 * b];
    y += part[3 * b + 1];
    z += part[3 * b + 2];
  }
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
