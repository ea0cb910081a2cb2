// Relative clip + optimizer step on fp32 masters (App. A; Sec. 3.1
// optimizers): the per-block device routine shared by the standalone update
// kernel and the fused outer-product + update kernel, and the host-side
// derivation of its scalars.
#pragma once

#include "common.hpp"
#include "launch.hpp"

#include <math.h>

namespace fpo {

constexpr int kElemsPerBlock = 4096;  // 256 threads x 4 x float4

// Device copies of the hyperparameters: each derived factor is formed in double
// on the host and rounded once to float.
struct OptScalars {
  int kind, first, lp_bf16;
  float lr, momentum, beta1, one_m_beta1, beta2, one_m_beta2, adam_eps, decay;
  float lr_wd;  // lr * weight_decay: AdamW's decay term of the update (clip-the-update mode)
  float inv_bc1, inv_sqrt_bc2;  // 1/(1-beta1^t), 1/sqrt(1-beta2^t)
  double clip_frac;
};

// Scalars of one optimizer step, each derived factor formed in double and
// rounded once to float.
inline OptScalars make_opt_scalars(const UpdLaunch& a) {
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
  o.lr_wd = (float)(a.lr * a.weight_decay);
  o.clip_frac = a.clip_frac;
  const double bc1 = 1.0 - pow(a.beta1, (double)a.step);
  const double bc2 = 1.0 - pow(a.beta2, (double)a.step);
  o.inv_bc1 = (float)(1.0 / bc1);
  o.inv_sqrt_bc2 = (float)(1.0 / sqrt(bc2));
  return o;
}

__device__ __forceinline__ float clip_factor(double gs, double ws, double frac) {
  if (frac <= 0.0 || gs == 0.0) return 1.0f;
  const double s = frac * sqrt(ws) / sqrt(gs);
  return (float)(s < 1.0 ? s : 1.0);
}

// Update of NB blocks (kElemsPerBlock elements each; block k starts at
// (b0 + k * bstride) * kElemsPerBlock, blocks at or past nb are skipped) of one
// matrix with clip factor s; writes each block's ||W'||^2 to part[block].
// Every thread of the 256-thread workgroup must call it (it reduces through
// `red`, 16 doubles of LDS). ADAM selects the optimizer at compile time so
// that SGD keeps no second-moment registers. The gradient is float32, or bf16
// when GB16 (the staged pseudogradient, widened exactly). A block's result
// and partial do not depend on NB or on which blocks share the call.
template <bool GB16, bool ADAM, int NB>
__device__ __forceinline__ void update_visit(const void* __restrict__ gp, float* __restrict__ W,
                                              void* lp, float* __restrict__ s1,
                                              float* __restrict__ s2, int64_t numel, int64_t b0,
                                              int64_t bstride, int64_t nb, float s,
                                              const OptScalars& o, double* red,
                                              double* __restrict__ part) {
  // Every operand is streamed once: all of a thread's loads (of all NB blocks)
  // are issued before any store, and loads and stores are non-temporal so the
  // stream does not evict cached data.
  constexpr int U = kElemsPerBlock / 1024;
  // plain SGD (momentum 0, no state buffer): b = s * dW each step
  const bool fresh = !ADAM && (o.first || s1 == nullptr);
  f32x4 gv[NB][U], w[NB][U], v1[NB][U];
  f32x4 v2[ADAM ? NB : 1][U];
#pragma unroll
  for (int k = 0; k < NB; ++k) {
    const int64_t base = (b0 + k * bstride) * kElemsPerBlock;
    const int64_t end = (b0 + k * bstride >= nb) ? 0 : (numel < base + kElemsPerBlock ? numel : base + kElemsPerBlock);
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t i = base + threadIdx.x * 4 + u * 1024;
      gv[k][u] = w[k][u] = v1[k][u] = f32x4{0.f, 0.f, 0.f, 0.f};
      if constexpr (ADAM) v2[k][u] = f32x4{0.f, 0.f, 0.f, 0.f};
      if (i < end) {
        if constexpr (GB16) {
          const u32x2 h = __builtin_nontemporal_load(reinterpret_cast<const u32x2*>((const uint16_t*)gp + i));
          gv[k][u] = f32x4{bf16_lo(h.x), bf16_hi(h.x), bf16_lo(h.y), bf16_hi(h.y)};
        } else {
          gv[k][u] = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>((const float*)gp + i));
        }
        w[k][u] = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(W + i));
        if (!fresh) v1[k][u] = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(s1 + i));
        if constexpr (ADAM) v2[k][u] = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(s2 + i));
      }
    }
  }
#pragma unroll
  for (int k = 0; k < NB; ++k) {
    const int64_t blk = b0 + k * bstride;
    const int64_t base = blk * kElemsPerBlock;
    const int64_t end = (blk >= nb) ? 0 : (numel < base + kElemsPerBlock ? numel : base + kElemsPerBlock);
    float ss = 0.f;
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t i = base + threadIdx.x * 4 + u * 1024;
      if (i >= end) continue;
      const f32x4 gs = gv[k][u] * s;
      f32x4 wv = w[k][u];
      if constexpr (!ADAM) {  // SGD with momentum
        f32x4 bv;
        if (fresh) {
          bv = gs;
        } else {
          bv.x = fmaf(o.momentum, v1[k][u].x, gs.x);
          bv.y = fmaf(o.momentum, v1[k][u].y, gs.y);
          bv.z = fmaf(o.momentum, v1[k][u].z, gs.z);
          bv.w = fmaf(o.momentum, v1[k][u].w, gs.w);
        }
        if (s1) __builtin_nontemporal_store(bv, reinterpret_cast<f32x4*>(s1 + i));
        wv.x = fmaf(-o.lr, bv.x, wv.x);
        wv.y = fmaf(-o.lr, bv.y, wv.y);
        wv.z = fmaf(-o.lr, bv.z, wv.z);
        wv.w = fmaf(-o.lr, bv.w, wv.w);
      } else {  // AdamW, decoupled weight decay, bias corrected
        f32x4 mv = v1[k][u], vv = v2[k][u];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float ge = gs[e];
          const float me = o.beta1 * mv[e] + o.one_m_beta1 * ge;
          const float ve = o.beta2 * vv[e] + o.one_m_beta2 * ge * ge;
          mv[e] = me;
          vv[e] = ve;
          const float denom = sqrtf(ve) * o.inv_sqrt_bc2 + o.adam_eps;
          wv[e] = wv[e] * o.decay - o.lr * (me * o.inv_bc1) / denom;
        }
        __builtin_nontemporal_store(mv, reinterpret_cast<f32x4*>(s1 + i));
        __builtin_nontemporal_store(vv, reinterpret_cast<f32x4*>(s2 + i));
      }
      __builtin_nontemporal_store(wv, reinterpret_cast<f32x4*>(W + i));
      if (lp) {
        if (o.lp_bf16)
          __builtin_nontemporal_store(u32x2{pack_bf16x2(wv.x, wv.y), pack_bf16x2(wv.z, wv.w)},
                                      reinterpret_cast<u32x2*>((uint16_t*)lp + i));
        else
          __builtin_nontemporal_store(wv, reinterpret_cast<f32x4*>((float*)lp + i));
      }
      ss += wv.x * wv.x + wv.y * wv.y + wv.z * wv.z + wv.w * wv.w;
    }
    const double t = block_sum_d((double)ss, red);
    if (threadIdx.x == 0 && blk < nb) part[blk] = t;
  }
}

// ---- clip-the-update mode (||W' - W|| <= clip_frac ||W||): two passes.
// The optimizer's update of one element, unclipped: delta = -lr * b' (SGD,
// b' = momentum * b + g, or g at the first step / without state), or
// delta = -lr_wd * W - lr * m_hat / (sqrt(v_hat) + eps) (AdamW) from the new
// moments. Pass 1 writes the new state and the block's ||delta||^2; pass 2
// recomputes delta from the stored state and applies W' = W + s * delta.
template <bool ADAM>
__device__ __forceinline__ float upd_delta(float w, float b_or_m, float v, const OptScalars& o) {
  if constexpr (ADAM) {
    const float denom = sqrtf(v) * o.inv_sqrt_bc2 + o.adam_eps;
    return -o.lr_wd * w - o.lr * (b_or_m * o.inv_bc1) / denom;
  } else {
    return -o.lr * b_or_m;
  }
}

template <bool GB16>
__device__ __forceinline__ f32x4 load_grad4(const void* gp, int64_t i) {
  if constexpr (GB16) {
    const u32x2 h = __builtin_nontemporal_load(reinterpret_cast<const u32x2*>((const uint16_t*)gp + i));
    return f32x4{bf16_lo(h.x), bf16_hi(h.x), bf16_lo(h.y), bf16_hi(h.y)};
  } else {
    return __builtin_nontemporal_load(reinterpret_cast<const f32x4*>((const float*)gp + i));
  }
}

// Pass 1 over block b: new optimizer state (written) and the block's
// ||delta||^2 (to *part_b).
template <bool GB16, bool ADAM>
__device__ __forceinline__ void delta_block(const void* __restrict__ gp, const float* __restrict__ W,
                                            float* __restrict__ s1, float* __restrict__ s2,
                                            int64_t numel, int64_t b, const OptScalars& o,
                                            double* red, double* part_b) {
  constexpr int U = kElemsPerBlock / 1024;
  const int64_t base = b * kElemsPerBlock;
  const int64_t end = numel < base + kElemsPerBlock ? numel : base + kElemsPerBlock;
  const bool fresh = !ADAM && (o.first || s1 == nullptr);
  f32x4 gv[U], w[U], v1[U], v2[U];
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int64_t i = base + threadIdx.x * 4 + u * 1024;
    gv[u] = w[u] = v1[u] = v2[u] = f32x4{0.f, 0.f, 0.f, 0.f};
    if (i < end) {
      gv[u] = load_grad4<GB16>(gp, i);
      if constexpr (ADAM) {
        w[u] = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(W + i));
        v2[u] = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(s2 + i));
      }
      if (!fresh) v1[u] = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(s1 + i));
    }
  }
  float ss = 0.f;
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int64_t i = base + threadIdx.x * 4 + u * 1024;
    if (i >= end) continue;
    f32x4 nb, nv = v2[u];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float ge = gv[u][e];
      if constexpr (ADAM) {
        nb[e] = o.beta1 * v1[u][e] + o.one_m_beta1 * ge;
        nv[e] = o.beta2 * v2[u][e] + o.one_m_beta2 * ge * ge;
      } else {
        nb[e] = fresh ? ge : fmaf(o.momentum, v1[u][e], ge);
      }
      const float dl = upd_delta<ADAM>(w[u][e], nb[e], nv[e], o);
      ss += dl * dl;
    }
    if (s1) __builtin_nontemporal_store(nb, reinterpret_cast<f32x4*>(s1 + i));
    if constexpr (ADAM) __builtin_nontemporal_store(nv, reinterpret_cast<f32x4*>(s2 + i));
  }
  const double t = block_sum_d((double)ss, red);
  if (threadIdx.x == 0) *part_b = t;
}

// Pass 2 over block b: W' = W + s * delta (delta from the stored new state, or
// from the gradient when SGD keeps none), the low-precision copy, and the
// block's ||W'||^2 (to *part_b).
template <bool GB16, bool ADAM>
__device__ __forceinline__ void apply_block(const void* __restrict__ gp, float* __restrict__ W, void* lp,
                                            const float* __restrict__ s1, const float* __restrict__ s2,
                                            int64_t numel, int64_t b, float s, const OptScalars& o,
                                            double* red, double* part_b) {
  constexpr int U = kElemsPerBlock / 1024;
  const int64_t base = b * kElemsPerBlock;
  const int64_t end = numel < base + kElemsPerBlock ? numel : base + kElemsPerBlock;
  f32x4 w[U], v1[U], v2[U];
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int64_t i = base + threadIdx.x * 4 + u * 1024;
    w[u] = v1[u] = v2[u] = f32x4{0.f, 0.f, 0.f, 0.f};
    if (i < end) {
      w[u] = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(W + i));
      v1[u] = s1 ? __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(s1 + i)) : load_grad4<GB16>(gp, i);
      if constexpr (ADAM) v2[u] = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(s2 + i));
    }
  }
  float ss = 0.f;
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int64_t i = base + threadIdx.x * 4 + u * 1024;
    if (i >= end) continue;
    f32x4 wv;
#pragma unroll
    for (int e = 0; e < 4; ++e) wv[e] = fmaf(s, upd_delta<ADAM>(w[u][e], v1[u][e], v2[u][e], o), w[u][e]);
    __builtin_nontemporal_store(wv, reinterpret_cast<f32x4*>(W + i));
    if (lp) {
      if (o.lp_bf16)
        __builtin_nontemporal_store(u32x2{pack_bf16x2(wv.x, wv.y), pack_bf16x2(wv.z, wv.w)},
                                    reinterpret_cast<u32x2*>((uint16_t*)lp + i));
      else
        __builtin_nontemporal_store(wv, reinterpret_cast<f32x4*>((float*)lp + i));
    }
    ss += wv.x * wv.x + wv.y * wv.y + wv.z * wv.z + wv.w * wv.w;
  }
  const double t = block_sum_d((double)ss, red);
  if (threadIdx.x == 0) *part_b = t;
}

}  // namespace fpo
