// Output-error path (Sec. 3.1 steps 2-4; eq. gproj; App. E eq. rmsnorm-vjp):
//   rms_forward  : rho_t, y_t = gamma * x_t / rho_t, and the first chunk's
//                  reference R_t = <y_t, W_U[y_t]> (the target logit)  (HBM bound)
//   logits_chunk : z = y W_c^T for one vocabulary chunk (MFMA), per-block
//                  row statistics, p~ = exp(z - R_t) staged            (MFMA bound)
//   chunk_stats  : running max / partition function / argmax per token; the
//                  next chunk's reference R_t <- running max; the rare rows
//                  with a block far above R_t rescaled in place
//   proj_chunk   : G_s <- rescale(G_s) + p~ W_c (MFMA), one partial per split
//   finalize_vjp : g = sum_s G_s / S - W_U[y], the loss (from rms_forward's
//                  target logit), the clamped RMSNorm VJP              (HBM bound)
// The T x V logits are never stored: only one vocabulary chunk of p~ (bf16,
// at most 2^26 entries by default, so it stays in the 256 MB Infinity Cache)
// is staged between the logits and projection launches of that chunk.
#include "gemm.hpp"
#include "gemm2.hpp"
#include "launch.hpp"
#include "prof.hpp"

namespace fpo {

// ------------------------------------------------------------------ forward
// Per-token row kernels (one 256-lane workgroup per token, 1024 entries per
// sweep) hold rows of up to this many sweeps in registers between passes.
constexpr int kRowRegIters = 8;

// The value of f after rounding to the storage type T.
template <typename T> __device__ __forceinline__ float round_to(float f);
template <> __device__ __forceinline__ float round_to<float>(float f) { return f; }
template <> __device__ __forceinline__ float round_to<uint16_t>(float f) { return bf16_to_f32(to_bf16(f)); }

// One workgroup per token: rho and y = gamma * x / rho (stored in the operand
// dtype), and the reference of the first vocabulary chunk, R = <y, W_U[v]>
// with v the token's target (entry 0 for a target outside [0, V)) from the
// stored (rounded) y: any logit is at most the row maximum, which is all the
// staging of p~ = exp(z - R) needs (see logits_epilogue).
template <typename T>
__global__ __launch_bounds__(256) void rms_forward_kernel(const T* __restrict__ x,
                                                          const T* __restrict__ gamma, int d,
                                                          float eps, T* __restrict__ y,
                                                          const T* __restrict__ W_U,
                                                          const int32_t* __restrict__ targets, int V,
                                                          float* __restrict__ ref,
                                                          float* __restrict__ zt,
                                                          int32_t* __restrict__ bad) {
  __shared__ float red[16];
  const int64_t row = blockIdx.x;
  const T* xr = x + row * d;
  // rows of up to kRowRegIters * 1024 entries are read once (held in registers)
  float ss = 0.f;
  f32x4 xk[kRowRegIters];
#pragma unroll
  for (int it = 0; it < kRowRegIters; ++it) {
    const int k = threadIdx.x * 4 + it * 1024;
    xk[it] = k < d ? ld4(xr, k) : f32x4{0.f, 0.f, 0.f, 0.f};
    ss += xk[it].x * xk[it].x + xk[it].y * xk[it].y + xk[it].z * xk[it].z + xk[it].w * xk[it].w;
  }
  for (int k = threadIdx.x * 4 + kRowRegIters * 1024; k < d; k += 1024) {
    const f32x4 v = ld4(xr, k);
    ss += v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
  }
  ss = block_sum(ss, red);
  const float inv = 1.0f / sqrtf(ss / (float)d + eps);
  const int tg = targets[row];
  const T* wr = W_U + (int64_t)((tg >= 0 && tg < V) ? tg : 0) * d;
  float zr = 0.f;
  auto out = [&](int k, f32x4 v) {
    const f32x4 g = ld4(gamma, k);
    const f32x4 o = {g.x * v.x * inv, g.y * v.y * inv, g.z * v.z * inv, g.w * v.w * inv};
    st4(y + row * d, k, o);
    const f32x4 w = ld4(wr, k);
    zr += round_to<T>(o.x) * w.x + round_to<T>(o.y) * w.y + round_to<T>(o.z) * w.z + round_to<T>(o.w) * w.w;
  };
#pragma unroll
  for (int it = 0; it < kRowRegIters; ++it) {
    const int k = threadIdx.x * 4 + it * 1024;
    if (k < d) out(k, xk[it]);
  }
  for (int k = threadIdx.x * 4 + kRowRegIters * 1024; k < d; k += 1024) out(k, ld4(xr, k));
  zr = block_sum(zr, red);
  if (threadIdx.x == 0) {
    ref[row] = zr;
    zt[row] = zr;  // the loss's target logit (valid targets), for finalize_vjp
  }
  if (bad && row == 0 && threadIdx.x == 0) *bad = 0;
}

// ------------------------------------------------------------------ logits
// Staging reference. A token's p~ entries are exp(z - R) with R its reference
// for the chunk (a logit of the first chunk, then the running maximum: never
// above the row maximum), so that every block of the chunk, and every chunk,
// shares one scale and the projection needs no per-block factor. Entries far
// below R (z < R - 87) underflow: relative to the sum, which holds an entry of
// at least exp(0), they weigh below 1e-33. A block whose maximum m exceeds
// R + kRefMargin would risk overflow in the projection's sums; it is staged as
// exp(z - m) instead, and the statistics kernel brings that token's row to one
// scale (base_b below is the scale of block b; both kernels take the same
// float decision).
constexpr float kRefMargin = 64.f;

__device__ __forceinline__ float block_base(float m, float R) { return m > R + kRefMargin ? m : R; }

// One workgroup: 256 (bf16) / 128 (fp32) tokens x as many vocabulary columns of
// the chunk; each wave's 128 / 64 columns form one statistics block b (block
// max m, sum of the staged p~, first arg-max). Columns at or beyond `vc_valid`
// are masked out; p~ = exp(z - base_b) is staged for the projection.
template <typename PT, bool CONTIG, class Map, class VA, int FM, int FN>
__device__ __forceinline__ void logits_epilogue(VA (&acc)[FM][FN], const Map& mp, int m0,
                                                int n0, int b, int T, int vc_valid, int v0,
                                                const float* __restrict__ ref,
                                                PT* __restrict__ P, int64_t ldp, int nb,
                                                float* __restrict__ blk_m,
                                                float* __restrict__ blk_s,
                                                int32_t* __restrict__ blk_i) {
  const int lr = threadIdx.x & (Map::LPR - 1);
#pragma unroll
  for (int f = 0; f < FM; ++f) {
#pragma unroll
    for (int r = 0; r < Map::R; ++r) {
      const int row = m0 + mp.row(f, r);
      float z[FN];
      float m = -INFINITY;
      int mi = 0x7fffffff;
#pragma unroll
      for (int i = 0; i < FN; ++i) {  // columns increase with i
        const int c = n0 + mp.col(i);
        z[i] = acc[f][i][r];
        if (c < vc_valid && z[i] > m) {
          m = z[i];
          mi = c;
        }
      }
      // lowest column among equal maxima across the lanes of the row
#pragma unroll
      for (int o = 1; o < Map::LPR; o <<= 1) {
        const float m2 = __shfl_xor(m, o, 64);
        const int i2 = __shfl_xor(mi, o, 64);
        if (m2 > m || (m2 == m && i2 < mi)) {
          m = m2;
          mi = i2;
        }
      }
      const float base = block_base(m, row < T ? ref[row] : 0.f);
      float p[FN];
      float s = 0.f;
#pragma unroll
      for (int i = 0; i < FN; ++i) {
        p[i] = (n0 + mp.col(i) < vc_valid) ? __expf(z[i] - base) : 0.f;
        s += p[i];
      }
      s = wave_sum<Map::LPR>(s);
      if (row < T) {
        PT* pr = P + (int64_t)row * ldp + n0;
        if constexpr (CONTIG) {
#pragma unroll
          for (int i = 0; i < FN; i += 4)
            st4(pr, mp.col(i), f32x4{p[i], p[i + 1], p[i + 2], p[i + 3]});
        } else {
#pragma unroll
          for (int i = 0; i < FN; ++i) st_from_f32(pr, mp.col(i), p[i]);
        }
        if (lr == 0 && b < nb) {
          const int64_t o = (int64_t)row * nb + b;
          blk_m[o] = m;
          blk_s[o] = s;
          blk_i[o] = (mi == 0x7fffffff) ? mi : v0 + mi;
        }
      }
    }
  }
}

// bf16: the tile is computed transposed, C^T = W_c y^T (rows: 256 vocabulary
// entries, columns: 256 tokens). Each lane then holds 64 logits of one token
// per accumulator column block i (vocabulary rows 32f + 8q + 4h + j, h = lane
// half, j < 4, in increasing order for increasing (f, q, j)); the lane pair
// (l, l ^ 32) covers the wave's 128 vocabulary entries of that token, so the
// block statistics need one cross-lane exchange. The bf16 p~ tile (256 tokens
// x 256 entries, 128 KB) is staged in the LDS ring, free after the main loop,
// as [token][32 chunks of 8 entries] with chunk c of token row r at position
// c ^ (r & 31) (the 32 token rows of one 8-byte write, and the 32 chunks of
// one row read back, fall in distinct 16-byte slots), then written out as
// whole 512-byte token rows: scattered 8-byte runs cost 7% of the kernel.
template <bool RAGGED>
__device__ __forceinline__ void logits_epilogue_vt(const f32x16 (&acc)[4][4], G2Smem& sm, int vt0,
                                                   int tt0, int T, int vc_valid, int v0,
                                                   const float* __restrict__ ref,
                                                   uint16_t* __restrict__ P, int64_t ldp, int nb,
                                                   float* __restrict__ blk_m,
                                                   float* __restrict__ blk_s,
                                                   int32_t* __restrict__ blk_i) {
  const int l = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int lc = l & 31, h = l >> 5;
  const int vw = vt0 + (w >> 1) * G2::WTM;  // chunk-relative first entry of the wave's block
  const int b = vw / G2::WTM;
  const int vl = vw + 4 * h;                // entry of offset 0 in this lane
  const int lim = vc_valid - vl;            // offset o is in range iff o < lim (RAGGED only)
  float R[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int t = tt0 + (w & 1) * G2::WTN + 32 * i + lc;
    R[i] = t < T ? ref[t] : 0.f;
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int t = tt0 + (w & 1) * G2::WTN + 32 * i + lc;
    // block maximum, then its first (lowest) entry; offsets o = 32f + 8q + j
    // increase with (f, r)
    float m = -INFINITY;
#pragma unroll
    for (int f = 0; f < 4; ++f)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int o = 32 * f + 8 * (r >> 2) + (r & 3);
        if (!RAGGED || o < lim) m = fmaxf(m, acc[f][i][r]);
      }
    int mo = 0x7fffffff;
#pragma unroll
    for (int f = 3; f >= 0; --f)
#pragma unroll
      for (int r = 15; r >= 0; --r) {
        const int o = 32 * f + 8 * (r >> 2) + (r & 3);
        if ((!RAGGED || o < lim) && acc[f][i][r] == m) mo = o;
      }
    int mi = mo == 0x7fffffff ? mo : vl + mo;
    {
      const float m2 = __shfl_xor(m, 32, 64);
      const int i2 = __shfl_xor(mi, 32, 64);
      if (m2 > m || (m2 == m && i2 < mi)) {
        m = m2;
        mi = i2;
      }
    }
    const float base = block_base(m, R[i]);
    // exp(z - base) as 2^(z log2 e - base log2 e): one fma ahead of the exp
    // instead of a subtract and a multiply (the staged value is bf16)
    const float nb2 = -base * 1.44269504088896341f;
    float s = 0.f;
    // LDS token row of this lane and the tile column of its entries at f = q = 0
    const int lrow = (w & 1) * G2::WTN + 32 * i + lc;
    const int col0 = vl - vt0;
    char* lds_row = reinterpret_cast<char*>(sm.s) + lrow * 512 + (col0 & 7) * 2;
#pragma unroll
    for (int f = 0; f < 4; ++f)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        float p[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int o = 32 * f + 8 * q + j;
          p[j] = (!RAGGED || o < lim) ? __builtin_amdgcn_exp2f(fmaf(acc[f][i][4 * q + j], 1.44269504088896341f, nb2))
                                      : 0.f;
          s += p[j];
        }
        const int chunk = ((col0 + 32 * f + 8 * q) >> 3) ^ lc;  // lrow & 31 == lc
        *reinterpret_cast<u32x2*>(lds_row + chunk * 16) = u32x2{pack_bf16x2(p[0], p[1]), pack_bf16x2(p[2], p[3])};
      }
    s += __shfl_xor(s, 32, 64);
    if (t < T && h == 0 && b < nb) {
      const int64_t ob = (int64_t)t * nb + b;
      blk_m[ob] = m;
      blk_s[ob] = s;
      blk_i[ob] = (mi == 0x7fffffff) ? mi : v0 + mi;
    }
  }
  __syncthreads();
  // whole token rows out: each half-wave one row, 16 bytes per lane (entries
  // past vc_valid were staged as zeros; the tile lies inside the chunk's Vc
  // columns)
  const int c = threadIdx.x & 31;
#pragma unroll 4
  for (int k = 0; k < 32; ++k) {
    const int r = (int)(threadIdx.x >> 5) + 8 * k;
    const int t = tt0 + r;
    if (t >= T) break;  // rows increase with k
    const u32x4 v = sm.s[r * 32 + (c ^ (r & 31))];
    *reinterpret_cast<u32x4*>(P + (int64_t)t * ldp + vt0 + 8 * c) = v;
  }
}

template <class E, bool FAST>
__global__ __launch_bounds__(256, 1) void logits_chunk_kernel(
    const typename E::T* __restrict__ y, const typename E::T* __restrict__ Wc, int T, int d,
    int vc_valid, int v0, const float* __restrict__ ref, typename E::T* __restrict__ P, int64_t ldp,
    int nb, float* __restrict__ blk_m, float* __restrict__ blk_s, int32_t* __restrict__ blk_i) {
  using TT = Tile<E>;
  const int ntm = (T + TT::BM - 1) / TT::BM, ntn = (vc_valid + TT::BN - 1) / TT::BN;
  int tm, tn;
  // consecutive workgroups share a vocabulary band and sweep the token tiles
  grouped_tile(xcd_remap(blockIdx.x, gridDim.x), ntm, ntn, 8, tm, tn);
  const int m0 = tm * TT::BM, n0 = tn * TT::BN;
  if constexpr (E::EPC == 8) {
    __shared__ G2Smem sm;
    f32x16 acc[4][4];
    zero_acc2(acc);
    const Operand A{Wc + (int64_t)n0 * d, d, band_bytes(vc_valid - n0, d)};
    const Operand B{y + (int64_t)m0 * d, d, band_bytes(T - m0, d)};
    gemm2_mainloop<false, FAST>(sm, acc, A, B, vc_valid - n0, T - m0, d, 0, (d + G2::BK - 1) / G2::BK);
    if (FAST || n0 + ((threadIdx.x >> 7) + 1) * G2::WTM <= vc_valid)  // wave-uniform; FAST: whole tiles
      logits_epilogue_vt<false>(acc, sm, n0, m0, T, vc_valid, v0, ref, P, ldp, nb, blk_m, blk_s, blk_i);
    else
      logits_epilogue_vt<true>(acc, sm, n0, m0, T, vc_valid, v0, ref, P, ldp, nb, blk_m, blk_s, blk_i);
  } else {
    __shared__ GemmSmem<E> sm;
    f32x4 acc[E::FM][E::FN];
    zero_acc<E>(acc);
    const int b = n0 / TT::WTN + ((threadIdx.x >> 6) & 1);  // this wave's block
    gemm_mainloop<E, false>(sm, acc, y, d, T, Wc, d, vc_valid, d, m0, n0, 0,
                            (d + TT::BK - 1) / TT::BK, NoHook{});
    logits_epilogue<typename E::T, true>(acc, AccMap<E>(), m0, n0, b, T, vc_valid, v0, ref, P, ldp, nb,
                                         blk_m, blk_s, blk_i);
  }
}

// ------------------------------------------------------------------ stats
// One wave per token. Folds the chunk's block statistics (block max m_b, sum
// s_b of the block's staged p~, which is in scale base_b, first arg-max) into
// the running max M, the partition function S (in scale M) and the argmax:
//   M_new = max(M_old, max_b m_b);  S <- S exp(M_old - M_new) + sum_b s_b exp(base_b - M_new).
// The chunk's p~ share the token's reference scale R unless a block was staged
// in its own (m_b > R + kRefMargin): this wave then brings the token's row to
// the chunk maximum in place (every factor <= 1). With Ref the row's final
// scale, the projection stores G_s <- acc exp(Ref - M_new) + G_s exp(M_old - M_new)
// (fout, alpha), and the next chunk's reference is M_new.
constexpr int kStatsRegs = 24;  // blocks per lane held in registers (chunks of up to 1536 blocks)

template <typename PT>
__global__ __launch_bounds__(256) void chunk_stats_kernel(
    int T, int nb, int first, const float* __restrict__ blk_m, const float* __restrict__ blk_s,
    const int32_t* __restrict__ blk_i, float* __restrict__ ref, float* __restrict__ runM,
    float* __restrict__ runS, int32_t* __restrict__ runA, float* __restrict__ fout,
    float* __restrict__ alpha, PT* __restrict__ P, int64_t ldp) {
  const int w = threadIdx.x >> 6, l = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + w;
  if (row >= T) return;  // whole wave exits together; no barrier below
  const float* bm = blk_m + (int64_t)row * nb;
  const float* bs = blk_s + (int64_t)row * nb;
  const int32_t* bi = blk_i + (int64_t)row * nb;
  const float R = ref[row];
  const float Mold = first ? -INFINITY : runM[row];
  float mc = -INFINITY, s = 0.f, Mnew;
  int ai = 0x7fffffff;
  bool own = false;  // a block of this lane was staged in its own scale
  if (nb <= 64 * kStatsRegs) {
    // each lane's block maxima and sums loaded once (blocks l + 64j)
    float vm[kStatsRegs], vs[kStatsRegs];
#pragma unroll
    for (int j = 0; j < kStatsRegs; ++j) {
      const int b = l + 64 * j;
      vm[j] = b < nb ? bm[b] : -INFINITY;
      vs[j] = b < nb ? bs[b] : 0.f;
    }
#pragma unroll
    for (int j = 0; j < kStatsRegs; ++j) mc = fmaxf(mc, vm[j]);
    mc = wave_max(mc);
#pragma unroll
    for (int j = 0; j < kStatsRegs; ++j) {
      const int b = l + 64 * j;
      if (b < nb && vm[j] == mc) ai = min(ai, bi[b]);
    }
    Mnew = fmaxf(Mold, mc);
#pragma unroll
    for (int j = 0; j < kStatsRegs; ++j)
      if (l + 64 * j < nb) {
        const float bb = block_base(vm[j], R);
        own |= bb != R;
        s += vs[j] * __expf(bb - Mnew);
      }
  } else {
    for (int b = l; b < nb; b += 64) mc = fmaxf(mc, bm[b]);
    mc = wave_max(mc);
    for (int b = l; b < nb; b += 64)
      if (bm[b] == mc) ai = min(ai, bi[b]);
    Mnew = fmaxf(Mold, mc);
    for (int b = l; b < nb; b += 64) {
      const float bb = block_base(bm[b], R);
      own |= bb != R;
      s += bs[b] * __expf(bb - Mnew);
    }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) ai = min(ai, __shfl_xor(ai, o, 64));
  s = wave_sum(s);
  const bool any_own = __ballot(own) != 0;  // wave-uniform
  // a block above R + kRefMargin makes the chunk maximum exceed every base_b
  const float Ref = any_own ? mc : R;
  if (any_own) {
    // the token's staged row, 16-byte runs; 16 runs per block for both
    // element types (128 bf16 or 64 fp32 entries)
    u32x4* pr = reinterpret_cast<u32x4*>(P + (int64_t)row * ldp);
    for (int c = l; c < nb * 16; c += 64) {
      const float bb = block_base(bm[c >> 4], R);
      if (bb == Ref) continue;
      const float f = __expf(bb - Ref);
      u32x4 v = pr[c];
      if constexpr (sizeof(PT) == 2) {
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = pack_bf16x2(bf16_lo(v[e]) * f, bf16_hi(v[e]) * f);
      } else {
        v = __builtin_bit_cast(u32x4, __builtin_bit_cast(f32x4, v) * f);
      }
      pr[c] = v;
    }
  }
  if (l == 0) {
    const float a = first ? 0.f : __expf(Mold - Mnew);
    runS[row] = (first ? 0.f : runS[row] * a) + s;
    runM[row] = Mnew;
    alpha[row] = a;
    if (first || mc > Mold) runA[row] = ai;
    fout[row] = __expf(Ref - Mnew);
    ref[row] = Mnew;
  }
}

// ------------------------------------------------------------------ projection
// G_s[t, :] (one partial per split s of the chunk's blocks) holds
// sum_v exp(z_tv - M_t) W_U[v, :] over its share of the vocabulary processed
// so far; the chunk's products are accumulated in the row's staging scale and
// merged in the epilogue with the per-token factors of chunk_stats.
template <class Map, class VA, int FM, int FN>
__device__ __forceinline__ void proj_epilogue(VA (&acc)[FM][FN], const Map& mp, int m0, int n0,
                                              int T, int d, int first,
                                              const float* __restrict__ fout,
                                              const float* __restrict__ alpha,
                                              float* __restrict__ Gs) {
#pragma unroll
  for (int f = 0; f < FM; ++f)
#pragma unroll
    for (int r = 0; r < Map::R; ++r) {
      const int row = m0 + mp.row(f, r);
      const int c = n0 + mp.col(0);  // FN consecutive columns
      if (row >= T || c >= d) continue;
      const float so = fout[row];
      const float sa = first ? 0.f : alpha[row];
#pragma unroll
      for (int i = 0; i < FN; i += 4) {
        float* gp = Gs + (int64_t)row * d + c + i;
        f32x4 o = {acc[f][i][r] * so, acc[f][i + 1][r] * so, acc[f][i + 2][r] * so,
                   acc[f][i + 3][r] * so};
        if (!first) o += *reinterpret_cast<const f32x4*>(gp) * sa;
        *reinterpret_cast<f32x4*>(gp) = o;
      }
    }
}

// bf16 form of the merge: the tile's per-row factors exp(Ref - M_new) and
// exp(M_old - M_new) are staged in LDS (the ring is free after the main loop)
// and each fragment's 16 partial rows are loaded together before use, so the
// row loads overlap instead of serialising on their latency.
__device__ __forceinline__ void proj_epilogue2(f32x16 (&acc)[4][4], G2Smem& sm, int m0, int n0,
                                               int T, int d, int first,
                                               const float* __restrict__ fout,
                                               const float* __restrict__ alpha,
                                               float* __restrict__ Gs) {
  float* sf = reinterpret_cast<float*>(sm.s);
  {
    const int rr = m0 + (int)threadIdx.x;
    sf[threadIdx.x] = rr < T ? fout[rr] : 0.f;
    sf[256 + threadIdx.x] = (!first && rr < T) ? alpha[rr] : 0.f;
  }
  __syncthreads();
  const AccMap2<true> mp;
  const int c = n0 + mp.col(0);  // 4 consecutive columns
  const bool cok = c < d;        // d % 4 == 0
#pragma unroll
  for (int f = 0; f < 4; ++f) {
    f32x4 old[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int row = m0 + mp.row(f, r);
      old[r] = f32x4{0.f, 0.f, 0.f, 0.f};
      if (!first && cok && row < T) old[r] = *reinterpret_cast<const f32x4*>(Gs + (int64_t)row * d + c);
    }
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int lr = mp.row(f, r);
      const int row = m0 + lr;
      if (!cok || row >= T) continue;
      const float so = sf[lr], sa = sf[256 + lr];
      const f32x4 o = f32x4{acc[f][0][r], acc[f][1][r], acc[f][2][r], acc[f][3][r]} * so + old[r] * sa;
      *reinterpret_cast<f32x4*>(Gs + (int64_t)row * d + c) = o;
    }
  }
}

template <class E, bool FAST>
__global__ __launch_bounds__(256, 1) void proj_chunk_kernel(
    const typename E::T* __restrict__ P, int64_t ldp, const typename E::T* __restrict__ Wc,
    int T, int d, int vc_valid, int nb, int bps, int blkw, int first, int nsplit,
    const float* __restrict__ fout, const float* __restrict__ alpha, float* __restrict__ G,
    int64_t split_stride) {
  using TT = Tile<E>;
  // tiles: (token rows) x (split, column); columns of one split are adjacent
  const int ntm = (T + TT::BM - 1) / TT::BM, ntn = (d + TT::BN - 1) / TT::BN;
  int tm, tsn;
  grouped_tile(xcd_remap(blockIdx.x, gridDim.x), ntm, ntn * nsplit, 8, tm, tsn);
  const int sp = tsn / ntn;
  const int m0 = tm * TT::BM, n0 = (tsn % ntn) * TT::BN;
  float* Gs = G + sp * split_stride;
  if constexpr (E::EPC == 8) {
    __shared__ G2Smem sm;
    f32x16 acc[4][4];
    zero_acc2(acc);
    const int tpb = blkw / G2::BK;
    const int nkt = (vc_valid + G2::BK - 1) / G2::BK;
    const int kt0 = min(sp * bps * tpb, nkt), kt1 = min(min(nb, (sp + 1) * bps) * tpb, nkt);
    const Operand A{P + (int64_t)m0 * ldp, ldp, band_bytes(T - m0, ldp)};
    const Operand B{Wc + n0, d, band_bytes(vc_valid, d, n0)};
    gemm2_mainloop<true, FAST>(sm, acc, A, B, T - m0, d - n0, vc_valid, kt0, kt1);
    proj_epilogue2(acc, sm, m0, n0, T, d, first, fout, alpha, Gs);
  } else {
    __shared__ GemmSmem<E> sm;
    f32x4 acc[E::FM][E::FN];
    zero_acc<E>(acc);
    const int tpb = blkw / TT::BK;
    const int nkt = (vc_valid + TT::BK - 1) / TT::BK;
    const int kt0 = min(sp * bps * tpb, nkt), kt1 = min(min(nb, (sp + 1) * bps) * tpb, nkt);
    gemm_mainloop<E, true>(sm, acc, P, ldp, T, Wc, d, d, vc_valid, m0, n0, kt0, kt1, NoHook{});
    proj_epilogue(acc, AccMap<E>(), m0, n0, T, d, first, fout, alpha, Gs);
  }
}

// ------------------------------------------------------------------ finalize
// One workgroup per token: g = sum_s G_s / S - W_U[y] (zero for a target
// outside [0, V)), then the clamped VJP
//   rho~ = max(sqrt(mean x^2 + eps), min_rms); x^ = x / rho~;
//   c = (1/d) <x^, gamma * g>;  g~ = (gamma * g - c x^) / rho~.
// The loss takes the target logit that rms_forward formed from the stored y
// (the same products and summation order as a second pass here would use),
// so the row of y is not read again.
template <typename T>
__global__ __launch_bounds__(256) void finalize_vjp_kernel(
    int d, int V, int nsplit, int64_t split_stride, const float* __restrict__ G,
    const float* __restrict__ runM, const float* __restrict__ runS,
    const int32_t* __restrict__ runA, const float* __restrict__ zt,
    const int32_t* __restrict__ targets, const T* __restrict__ W_U, const T* __restrict__ x,
    const T* __restrict__ gamma, float eps, float min_rms, float* __restrict__ g_tilde,
    T* __restrict__ g_tilde_lp, float* __restrict__ g_pre, float* __restrict__ lse,
    float* __restrict__ loss, int32_t* __restrict__ argmax, int32_t* __restrict__ bad) {
  __shared__ float red[32];
  const int64_t row = blockIdx.x;
  const int tg = targets[row];
  const bool valid = tg >= 0 && tg < V;
  const float S = runS[row];
  const float invS = 1.0f / S;
  const T* xr = x + row * d;
  float* gt = g_tilde + row * d;
  float ss = 0.f, cd = 0.f;
  // pass 1: g = sum_s G_s / S - W_U[y] and the row reductions. Rows of up to
  // kRowRegIters * 1024 entries keep g and x in registers for pass 2; longer
  // rows park the rest of g in the g~ row (rewritten in pass 2).
  f32x4 gk[kRowRegIters], xk[kRowRegIters];
  auto pass1 = [&](int k) -> f32x4 {
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    for (int s = 0; s < nsplit; ++s) acc += *reinterpret_cast<const f32x4*>(G + s * split_stride + row * d + k);
    f32x4 g = {0.f, 0.f, 0.f, 0.f};
    if (valid) g = acc * invS - ld4(W_U + (int64_t)tg * d, k);
    if (g_pre) *reinterpret_cast<f32x4*>(g_pre + row * d + k) = g;
    return g;
  };
  auto reduce = [&](f32x4 g, f32x4 xv, f32x4 gm) {
    ss += xv.x * xv.x + xv.y * xv.y + xv.z * xv.z + xv.w * xv.w;
    cd += xv.x * gm.x * g.x + xv.y * gm.y * g.y + xv.z * gm.z * g.z + xv.w * gm.w * g.w;
  };
#pragma unroll
  for (int it = 0; it < kRowRegIters; ++it) {
    const int k = threadIdx.x * 4 + it * 1024;
    gk[it] = xk[it] = f32x4{0.f, 0.f, 0.f, 0.f};
    if (k < d) {
      gk[it] = pass1(k);
      xk[it] = ld4(xr, k);
      reduce(gk[it], xk[it], ld4(gamma, k));
    }
  }
  for (int k = threadIdx.x * 4 + kRowRegIters * 1024; k < d; k += 1024) {
    const f32x4 g = pass1(k), xv = ld4(xr, k);
    *reinterpret_cast<f32x4*>(gt + k) = g;
    reduce(g, xv, ld4(gamma, k));
  }
  block_sum2(ss, cd, red);
  const float rho = sqrtf(ss / (float)d + eps);
  const float rt = fmaxf(rho, min_rms);
  const float irt = 1.0f / rt;
  const float c = cd * irt / (float)d;  // (1/d) <x / rho~, gamma * g>
  // pass 2: g~ = (gamma g - c x^) / rho~
  auto out = [&](int k, f32x4 g, f32x4 xv) {
    const f32x4 gm = ld4(gamma, k);
    f32x4 o;
    o.x = (gm.x * g.x - c * xv.x * irt) * irt;
    o.y = (gm.y * g.y - c * xv.y * irt) * irt;
    o.z = (gm.z * g.z - c * xv.z * irt) * irt;
    o.w = (gm.w * g.w - c * xv.w * irt) * irt;
    *reinterpret_cast<f32x4*>(gt + k) = o;
    if (g_tilde_lp) st4(g_tilde_lp + row * d, k, o);
  };
#pragma unroll
  for (int it = 0; it < kRowRegIters; ++it) {
    const int k = threadIdx.x * 4 + it * 1024;
    if (k < d) out(k, gk[it], xk[it]);
  }
  for (int k = threadIdx.x * 4 + kRowRegIters * 1024; k < d; k += 1024)
    out(k, *reinterpret_cast<const f32x4*>(gt + k), ld4(xr, k));
  if (threadIdx.x == 0) {
    const float l_se = runM[row] + logf(S);
    if (lse) lse[row] = l_se;
    if (loss) loss[row] = valid ? l_se - zt[row] : 0.f;  // target logit from rms_forward
    if (argmax) argmax[row] = runA[row];
    if (!valid && bad) atomicAdd(bad, 1);
  }
}

// ------------------------------------------------------------------ launchers
#define FPO_CHECK_LAUNCH()                       \
  do {                                           \
    hipError_t e_ = hipGetLastError();           \
    if (e_ != hipSuccess) return e_;             \
  } while (0)

template <class E>
static hipError_t run_output_error(const OeLaunch& a) {
  using T = typename E::T;
  using TT = Tile<E>;
  hipStream_t st = (hipStream_t)a.stream;
  const T* x = (const T*)a.h_final;
  const T* gamma = (const T*)a.gamma;
  const T* W = (const T*)a.W_U;
  T* y = (T*)a.y;
  T* P = (T*)a.P;
  FPO_LAUNCH("rms_forward", st,
             rms_forward_kernel<T><<<dim3((unsigned)a.T), dim3(256), 0, st>>>(
      x, gamma, (int)a.d, a.eps, y, W, a.targets, (int)a.V, a.ref, a.zt, a.bad_targets));
  FPO_CHECK_LAUNCH();
  const int gm = (int)((a.T + TT::BM - 1) / TT::BM);
  for (int c = 0; c < a.nchunk; ++c) {
    int64_t v0, width;
    chunk_span(a.V, a.nchunk, a.cw, a.cq, a.nwide, c, &v0, &width);
    const int vc_valid = (int)width;
    const int gn = (vc_valid + TT::BN - 1) / TT::BN;
    const int nbv = (vc_valid + TT::WTN - 1) / TT::WTN;  // blocks holding a valid column
    // whole 256 x 256 tiles and 64-deep K tiles: the copy form without bounds
    const bool fast_l = vc_valid % TT::BM == 0 && a.T % TT::BN == 0 && a.d % 64 == 0;
    if (fast_l)
      FPO_LAUNCH("logits_chunk", st,
                 logits_chunk_kernel<E, true><<<dim3(gm * gn), dim3(256), 0, st>>>(
          y, W + v0 * a.d, (int)a.T, (int)a.d, vc_valid, (int)v0, a.ref, P, a.ldp, nbv, a.blk_m, a.blk_s,
          a.blk_i));
    else
      FPO_LAUNCH("logits_chunk", st,
                 logits_chunk_kernel<E, false><<<dim3(gm * gn), dim3(256), 0, st>>>(
          y, W + v0 * a.d, (int)a.T, (int)a.d, vc_valid, (int)v0, a.ref, P, a.ldp, nbv, a.blk_m, a.blk_s,
          a.blk_i));
    FPO_CHECK_LAUNCH();
    FPO_LAUNCH("chunk_stats", st,
               chunk_stats_kernel<T><<<dim3((unsigned)((a.T + 3) / 4)), dim3(256), 0, st>>>(
        (int)a.T, nbv, c == 0, a.blk_m, a.blk_s, a.blk_i, a.ref, a.runM, a.runS, a.runA, a.fout, a.alpha,
        P, a.ldp));
    FPO_CHECK_LAUNCH();
    const int bps = (nbv + a.nsplit - 1) / a.nsplit;
    const bool fast_p = a.T % TT::BM == 0 && a.d % TT::BN == 0 && vc_valid % 64 == 0;
    const dim3 gp(gm * (unsigned)((a.d + TT::BN - 1) / TT::BN) * a.nsplit);
    if (fast_p)
      FPO_LAUNCH("proj_chunk", st,
                 proj_chunk_kernel<E, true><<<gp, dim3(256), 0, st>>>(
          P, a.ldp, W + v0 * a.d, (int)a.T, (int)a.d, vc_valid, nbv, bps, TT::WTN, c == 0, a.nsplit,
          a.fout, a.alpha, a.G, a.T * a.d));
    else
      FPO_LAUNCH("proj_chunk", st,
                 proj_chunk_kernel<E, false><<<gp, dim3(256), 0, st>>>(
          P, a.ldp, W + v0 * a.d, (int)a.T, (int)a.d, vc_valid, nbv, bps, TT::WTN, c == 0, a.nsplit,
          a.fout, a.alpha, a.G, a.T * a.d));
    FPO_CHECK_LAUNCH();
  }
  FPO_LAUNCH("finalize_vjp", st,
             finalize_vjp_kernel<T><<<dim3((unsigned)a.T), dim3(256), 0, st>>>(
      (int)a.d, (int)a.V, a.nsplit, a.T * a.d, a.G, a.runM, a.runS, a.runA, a.zt, a.targets, W,
      x, gamma, a.eps, a.min_rms, a.g_tilde, (T*)a.g_tilde_lp, a.g_pre, a.lse, a.loss, a.argmax,
      a.bad_targets));
  FPO_CHECK_LAUNCH();
  return hipSuccess;
}

hipError_t launch_output_error(const OeLaunch& a) {
  return a.bf16 ? run_output_error<TileBF16>(a) : run_output_error<TileF32>(a);
}

}  // namespace fpo
