// Per-layer outer products (eq. w3update; App. A divisor) and the full-MLP
// feedback path (eq. errh):
//   signal_transpose : g~ [T, d] -> g~^T [d, Tp] (zero columns t >= T) so that
//                   the token axis, the contraction axis, is contiguous; with
//                   the post-FFN composition it forms each layer's signal
//                   (pffn_stats: its per-token norm statistics) on the way
//   outer_kernel  : C_m = scale * A_m B_m for a list of matrices (MFMA),
//                   A_m [M, Tp] token-contiguous, B_m [T, N] row-major; epilogue
//                   writes C (fp32, or rounded to bf16 for the fused update) and
//                   per-tile ||C||^2 (and <C, R>, ||R||^2)
//   errh_kernel   : E = g~ W3_init (MFMA); du = E*SiLU(q), dq = E*u*SiLU'(q),
//                   stored token-contiguous for the W1/W2 outer products
//   reduce_parts  : fixed-order float64 sums of the tile partials
// With the optimizer fused (bf16), launch_pseudograd_update runs the outer
// products one layer per launch and each matrix's update on a side stream,
// overlapping the GEMM launches that follow.
#include "gemm.hpp"
#include "gemm2.hpp"
#include "launch.hpp"
#include "prof.hpp"

#include <mutex>

namespace fpo {

// Per-token statistics of a layer's norm chain (one workgroup per token),
// with g the fp32 signal g~:
//   post-FFN (POST): irt1 = 1 / max(sqrt(mean x1^2 + eps1), min_rms1),
//                    c1 = (1/d) <x1 irt1, gamma1 g>;  v1 = (gamma1 g - c1 x1 irt1) irt1
//   pre-MLP (PRE):   irt2, c2 the same with x2, gamma2 and v1 (g without POST)
// where x1 is the cached MLP output and x2 the cached pre-MLP norm input.
// stats[t] = {irt1, c1, irt2, c2}; signal_transpose forms the composed signal
// from them elementwise with the same float expressions.
template <typename T, bool POST, bool PRE>
__global__ __launch_bounds__(256) void chain_stats_kernel(int d, const float* __restrict__ g,
                                                          const T* __restrict__ x1,
                                                          const T* __restrict__ gamma1, float eps1,
                                                          float mr1, const T* __restrict__ x2,
                                                          const T* __restrict__ gamma2, float eps2,
                                                          float mr2, float4* __restrict__ stats) {
  __shared__ float red[16];
  const int64_t row = blockIdx.x;
  const float* gr = g + row * d;
  float irt1 = 1.f, c1 = 0.f, irt2 = 1.f, c2 = 0.f;
  if constexpr (POST) {
    const T* xr = x1 + row * d;
    float ss = 0.f, cd = 0.f;
    for (int k = threadIdx.x * 4; k < d; k += 1024) {
      const f32x4 xv = ld4(xr, k), gm = ld4(gamma1, k), gv = *reinterpret_cast<const f32x4*>(gr + k);
      ss += xv.x * xv.x + xv.y * xv.y + xv.z * xv.z + xv.w * xv.w;
      cd += xv.x * gm.x * gv.x + xv.y * gm.y * gv.y + xv.z * gm.z * gv.z + xv.w * gm.w * gv.w;
    }
    ss = block_sum(ss, red);
    cd = block_sum(cd, red);
    irt1 = 1.0f / fmaxf(sqrtf(ss / (float)d + eps1), mr1);
    c1 = cd * irt1 / (float)d;
  }
  if constexpr (PRE) {
    const T* x1r = x1 + row * d;
    const T* xr = x2 + row * d;
    float ss = 0.f, cd = 0.f;
    for (int k = threadIdx.x * 4; k < d; k += 1024) {
      f32x4 v = *reinterpret_cast<const f32x4*>(gr + k);
      if constexpr (POST) {
        const f32x4 xv = ld4(x1r, k), gm = ld4(gamma1, k);
        v.x = (gm.x * v.x - c1 * xv.x * irt1) * irt1;
        v.y = (gm.y * v.y - c1 * xv.y * irt1) * irt1;
        v.z = (gm.z * v.z - c1 * xv.z * irt1) * irt1;
        v.w = (gm.w * v.w - c1 * xv.w * irt1) * irt1;
      }
      const f32x4 xv = ld4(xr, k), gm = ld4(gamma2, k);
      ss += xv.x * xv.x + xv.y * xv.y + xv.z * xv.z + xv.w * xv.w;
      cd += xv.x * gm.x * v.x + xv.y * gm.y * v.y + xv.z * gm.z * v.z + xv.w * gm.w * v.w;
    }
    ss = block_sum(ss, red);
    cd = block_sum(cd, red);
    irt2 = 1.0f / fmaxf(sqrtf(ss / (float)d + eps2), mr2);
    c2 = cd * irt2 / (float)d;
  }
  if (threadIdx.x == 0) stats[row] = float4{irt1, c1, irt2, c2};
}

// The token-contiguous copy of a layer's left operand: dst [C, ldd] with
// dst[c, r] = v(r, c) for r < R and 0 for R <= r < Rp, where v is src[r, c]
// (the shared signal, CHAIN == 0) or the fp32 src passed through the layer's
// norm chain (CHAIN bit 0: post-FFN VJP, bit 1: pre-MLP VJP, in that order;
// statistics from chain_stats_kernel), in the operand dtype (also stored
// row-major to row_out when given). 64 x 64 tiles through LDS, 16-byte loads
// and 8- / 16-byte stores.
template <typename T, int CHAIN>
__global__ __launch_bounds__(256) void signal_transpose_kernel(
    const void* __restrict__ src, const T* __restrict__ x1, const T* __restrict__ gamma1,
    const T* __restrict__ x2, const T* __restrict__ gamma2, const float4* __restrict__ stats, int64_t R,
    int64_t C, T* __restrict__ dst, int64_t ldd, int64_t Rp, T* __restrict__ row_out) {
  __shared__ float tile[64][65];
  const int64_t r0 = (int64_t)blockIdx.x * 64, c0 = (int64_t)blockIdx.y * 64;
  // 64 rows x 16 column quads
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int q = threadIdx.x + 256 * k, rr = q >> 4, cq = (q & 15) * 4;
    const int64_t r = r0 + rr, c = c0 + cq;
    f32x4 v = {0.f, 0.f, 0.f, 0.f};
    if (r < R && c < C) {  // C % 8 == 0: a quad is all in or all out
      if constexpr (CHAIN != 0) {
        v = *reinterpret_cast<const f32x4*>((const float*)src + r * C + c);
        const float4 st = stats[r];
        if constexpr (CHAIN & 1) {
          const f32x4 xv = ld4(x1, r * C + c), gm = ld4(gamma1, c);
          v.x = (gm.x * v.x - st.y * xv.x * st.x) * st.x;
          v.y = (gm.y * v.y - st.y * xv.y * st.x) * st.x;
          v.z = (gm.z * v.z - st.y * xv.z * st.x) * st.x;
          v.w = (gm.w * v.w - st.y * xv.w * st.x) * st.x;
        }
        if constexpr (CHAIN & 2) {
          const f32x4 xv = ld4(x2, r * C + c), gm = ld4(gamma2, c);
          v.x = (gm.x * v.x - st.w * xv.x * st.z) * st.z;
          v.y = (gm.y * v.y - st.w * xv.y * st.z) * st.z;
          v.z = (gm.z * v.z - st.w * xv.z * st.z) * st.z;
          v.w = (gm.w * v.w - st.w * xv.w * st.z) * st.z;
        }
        if (row_out) st4(row_out, r * C + c, v);
      } else {
        v = ld4((const T*)src, r * C + c);
      }
    }
    tile[rr][cq] = v.x;
    tile[rr][cq + 1] = v.y;
    tile[rr][cq + 2] = v.z;
    tile[rr][cq + 3] = v.w;
  }
  __syncthreads();
  // 64 columns x 16 row quads
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int q = threadIdx.x + 256 * k, cc = q >> 4, rq = (q & 15) * 4;
    const int64_t r = r0 + rq, c = c0 + cc;
    if (c < C && r < Rp)  // Rp % 64 == 0
      st4(dst, c * ldd + r, f32x4{tile[rq][cc], tile[rq + 1][cc], tile[rq + 2][cc], tile[rq + 3][cc]});
  }
}

struct OuterArgs {
  const void* A[kMaxMats];
  const void* B[kMaxMats];
  float* C[kMaxMats];
  uint16_t* Cb[kMaxMats];  // bf16 output instead of C (bf16 tiles only), or null
  const float* R[kMaxMats];
};

template <class Map, class VA, int FM, int FN>
__device__ __forceinline__ void outer_epilogue(VA (&acc)[FM][FN], const Map& mp, int m0, int n0,
                                               int M, int N, float scale, float* __restrict__ C,
                                               const float* __restrict__ R, double* red,
                                               double* __restrict__ part_out) {
  float ss = 0.f, dt = 0.f, rr = 0.f;
#pragma unroll
  for (int f = 0; f < FM; ++f)
#pragma unroll
    for (int r = 0; r < Map::R; ++r) {
      const int row = m0 + mp.row(f, r);
      const int c = n0 + mp.col(0);  // FN consecutive columns
      if (row >= M || c >= N) continue;  // N % 8 == 0: a lane's columns are all in or all out
#pragma unroll
      for (int i = 0; i < FN; i += 4) {
        f32x4 v = {acc[f][i][r] * scale, acc[f][i + 1][r] * scale, acc[f][i + 2][r] * scale,
                   acc[f][i + 3][r] * scale};
        const int64_t o = (int64_t)row * N + c + i;
        if (C) *reinterpret_cast<f32x4*>(C + o) = v;
        ss += v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
        if (R) {
          f32x4 q = *reinterpret_cast<const f32x4*>(R + o);
          dt += v.x * q.x + v.y * q.y + v.z * q.z + v.w * q.w;
          rr += q.x * q.x + q.y * q.y + q.z * q.z + q.w * q.w;
        }
      }
    }
  double s0 = wave_sum_d((double)ss), s1 = wave_sum_d((double)dt), s2 = wave_sum_d((double)rr);
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) {
    red[w] = s0;
    red[4 + w] = s1;
    red[8 + w] = s2;
  }
  __syncthreads();
  if (threadIdx.x < 3) {
    const int k = threadIdx.x;
    part_out[k] = red[4 * k] + red[4 * k + 1] + red[4 * k + 2] + red[4 * k + 3];
  }
}

// bf16 form: 16 rows of a fragment are loaded (reference) before use, so
// the loads overlap; every lane's 4 columns are consecutive.
// With Cb the tile is stored rounded to bf16 (RNE) and the partial norms and
// dot products are of the rounded values.
__device__ __forceinline__ void outer_epilogue2(const f32x16 (&acc)[4][4], int m0, int n0, int M,
                                                int N, float scale, float* __restrict__ C,
                                                uint16_t* __restrict__ Cb,
                                                const float* __restrict__ R, double* red,
                                                double* __restrict__ part_out) {
  const AccMap2<true> mp;
  const int c = n0 + mp.col(0);
  const bool cok = c < N;  // N % 4 == 0: a lane's columns are all in or all out
  float ss = 0.f, dt = 0.f, rr = 0.f;
#pragma unroll
  for (int f = 0; f < 4; ++f) {
    f32x4 q[16];
    if (R) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = m0 + mp.row(f, r);
        q[r] = f32x4{0.f, 0.f, 0.f, 0.f};
        if (cok && row < M) q[r] = *reinterpret_cast<const f32x4*>(R + (int64_t)row * N + c);
      }
    }
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int row = m0 + mp.row(f, r);
      if (!cok || row >= M) continue;
      f32x4 v = f32x4{acc[f][0][r], acc[f][1][r], acc[f][2][r], acc[f][3][r]} * scale;
      if (Cb) {
        const u32x2 h = {pack_bf16x2(v.x, v.y), pack_bf16x2(v.z, v.w)};
        *reinterpret_cast<u32x2*>(Cb + (int64_t)row * N + c) = h;
        v = f32x4{bf16_lo(h.x), bf16_hi(h.x), bf16_lo(h.y), bf16_hi(h.y)};
      }
      if (C) *reinterpret_cast<f32x4*>(C + (int64_t)row * N + c) = v;
      ss += v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
      if (R) {
        dt += v.x * q[r].x + v.y * q[r].y + v.z * q[r].z + v.w * q[r].w;
        rr += q[r].x * q[r].x + q[r].y * q[r].y + q[r].z * q[r].z + q[r].w * q[r].w;
      }
    }
  }
  double s0 = wave_sum_d((double)ss), s1 = wave_sum_d((double)dt), s2 = wave_sum_d((double)rr);
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) {
    red[w] = s0;
    red[4 + w] = s1;
    red[8 + w] = s2;
  }
  __syncthreads();
  if (threadIdx.x < 3) {
    const int k = threadIdx.x;
    part_out[k] = red[4 * k] + red[4 * k + 1] + red[4 * k + 2] + red[4 * k + 3];
  }
}

template <class E, bool FAST>
__global__ __launch_bounds__(256, 1) void outer_kernel(OuterArgs args, int M, int N, int K,
                                                       int64_t lda, int64_t ldb, float scale,
                                                       double* __restrict__ part) {
  using TT = Tile<E>;
  using T = typename E::T;
  __shared__ double red[12];
  // one flat grid over (matrix, tile), matrix-major in dispatch order, each
  // matrix's tiles spread over the 8 XCDs (a contiguous group per XCD), so
  // that the XCDs tend to work on the same matrix at the same time rather
  // than on eight different ones (how closely depends on dispatch timing: the
  // 36-layer diagnostic launch reads 65-91 GB beyond L2 from run to run, for
  // 14.5 GB of operands, which the Infinity Cache serves)
  const int ntm = (M + TT::BM - 1) / TT::BM, ntn = (N + TT::BN - 1) / TT::BN;
  const int ntiles = ntm * ntn;
  const int mat = blockIdx.x / ntiles;
  const int tile = xcd_remap(blockIdx.x - mat * ntiles, ntiles);
  int tm, tn;
  grouped_tile(tile, ntm, ntn, 8, tm, tn);
  const int m0 = tm * TT::BM, n0 = tn * TT::BN;
  const T* Am = (const T*)args.A[mat];
  const T* Bm = (const T*)args.B[mat];
  double* po = part + ((int64_t)mat * ntiles + tm + (int64_t)tn * ntm) * 3;
  if constexpr (E::EPC == 8) {
    __shared__ G2Smem sm;
    f32x16 acc[4][4];
    zero_acc2(acc);
    const Operand A{Am + (int64_t)m0 * lda, lda, band_bytes(M - m0, lda)};
    const Operand B{Bm + n0, ldb, band_bytes(K, ldb, n0)};
    gemm2_mainloop<true, FAST>(sm, acc, A, B, M - m0, N - n0, K, 0, (K + G2::BK - 1) / G2::BK);
    outer_epilogue2(acc, m0, n0, M, N, scale, args.C[mat], args.Cb[mat], args.R[mat], red, po);
  } else {
    __shared__ GemmSmem<E> sm;
    f32x4 acc[E::FM][E::FN];
    zero_acc<E>(acc);
    gemm_mainloop<E, true>(sm, acc, Am, lda, M, Bm, ldb, N, K, m0, n0, 0, (K + TT::BK - 1) / TT::BK,
                           NoHook{});
    outer_epilogue(acc, AccMap<E>(), m0, n0, M, N, scale, args.C[mat], args.R[mat], red, po);
  }
}

// E = g~ W3_init for one layer; writes du^T and dq^T [d_ff, Tp] (rows t < Tp;
// t >= T give zero because the A rows load as zero and q, u are not read).
template <typename TE, class Map, class VA, int FM, int FN>
__device__ __forceinline__ void errh_epilogue(VA (&acc)[FM][FN], const Map& mp, int m0, int n0,
                                              const TE* __restrict__ q, const TE* __restrict__ u,
                                              int T, int Tp, int d_ff, TE* __restrict__ dq_T,
                                              TE* __restrict__ du_T) {
#pragma unroll
  for (int f = 0; f < FM; ++f)
#pragma unroll
  for (int rg = 0; rg < Map::R; rg += 4) {
    const int t0 = m0 + mp.row(f, rg);  // 4 consecutive tokens t0..t0+3
    if (t0 >= Tp) continue;             // Tp % 4 == 0
#pragma unroll
    for (int i = 0; i < FN; ++i) {
      const int j = n0 + mp.col(i);
      if (j >= d_ff) continue;
      float vq[4], vu[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int t = t0 + r;
        const float e = acc[f][i][rg + r];
        float dqv = 0.f, duv = 0.f;
        if (t < T) {
          const float qq = ld_as_f32(q, (int64_t)t * d_ff + j);
          const float uu = ld_as_f32(u, (int64_t)t * d_ff + j);
          const float sg = 1.0f / (1.0f + __expf(-qq));
          duv = e * qq * sg;
          dqv = e * uu * sg * (1.0f + qq * (1.0f - sg));
        }
        vq[r] = dqv;
        vu[r] = duv;
      }
      st4<TE>(dq_T + (int64_t)j * Tp + t0, 0, f32x4{vq[0], vq[1], vq[2], vq[3]});
      st4<TE>(du_T + (int64_t)j * Tp + t0, 0, f32x4{vu[0], vu[1], vu[2], vu[3]});
    }
  }
}

// bf16 form: per fragment and group of 4 consecutive tokens, the lane's 4
// consecutive columns of q and u are loaded as 8-byte runs (all 8 loads before
// use), and dq^T, du^T go out as 8-byte runs of 4 tokens.
__device__ __forceinline__ void errh_epilogue2(const f32x16 (&acc)[4][4], int m0, int n0,
                                               const uint16_t* __restrict__ q,
                                               const uint16_t* __restrict__ u, int T, int Tp,
                                               int d_ff, uint16_t* __restrict__ dq_T,
                                               uint16_t* __restrict__ du_T) {
  const AccMap2<true> mp;
  const int j0 = n0 + mp.col(0);
  if (j0 >= d_ff) return;  // d_ff % 4 == 0: the lane's 4 columns are all in or all out
#pragma unroll
  for (int f = 0; f < 4; ++f)
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const int t0 = m0 + mp.row(f, 4 * g);  // tokens t0..t0+3
      if (t0 >= Tp) continue;                // Tp % 4 == 0
      u32x2 qv[4], uv[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        qv[r] = u32x2{0u, 0u};
        uv[r] = u32x2{0u, 0u};
        if (t0 + r < T) {
          qv[r] = *reinterpret_cast<const u32x2*>(q + (int64_t)(t0 + r) * d_ff + j0);
          uv[r] = *reinterpret_cast<const u32x2*>(u + (int64_t)(t0 + r) * d_ff + j0);
        }
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        float vq[4], vu[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const uint32_t qw = qv[r][i >> 1], uw = uv[r][i >> 1];
          const float qq = (i & 1) ? bf16_hi(qw) : bf16_lo(qw);
          const float uu = (i & 1) ? bf16_hi(uw) : bf16_lo(uw);
          const float e = acc[f][i][4 * g + r];
          const float sg = 1.0f / (1.0f + __expf(-qq));
          const bool in = t0 + r < T;
          vu[r] = in ? e * qq * sg : 0.f;
          vq[r] = in ? e * uu * sg * (1.0f + qq * (1.0f - sg)) : 0.f;
        }
        st4<uint16_t>(dq_T + (int64_t)(j0 + i) * Tp + t0, 0, f32x4{vq[0], vq[1], vq[2], vq[3]});
        st4<uint16_t>(du_T + (int64_t)(j0 + i) * Tp + t0, 0, f32x4{vu[0], vu[1], vu[2], vu[3]});
      }
    }
}

// bf16 form for whole tiles (T and d_ff multiples of 256: no bounds), the
// transposed outputs staged through LDS one output per pass (pass 0: dq;
// pass 1: du, q loaded again; the accumulators are only read, so no register
// holds a second output): the lane's values for 4 consecutive tokens x 4
// consecutive columns go into the idle LDS ring as the 256 column x 256 token
// tile [column][32 chunks of 8 tokens] (chunk c of column j at position
// c ^ ((j >> 2) & 31)), then whole 512-byte token-contiguous rows of dq^T /
// du^T are stored. (Stored directly, each lane's 8-byte runs of 4 tokens land
// Tp apart: about 60 us of a 170 us tile at the OLMo-2 shapes; ragged tiles
// still take that form.) q and u are read as 8-byte runs of the lane's 4
// columns, one fragment group ahead of their use.
__device__ __forceinline__ void errh_epilogue_lds(f32x16 (&acc)[4][4], G2Smem& sm, int m0, int n0,
                                                  const uint16_t* __restrict__ q,
                                                  const uint16_t* __restrict__ u, int Tp,
                                                  int d_ff, uint16_t* __restrict__ dq_T,
                                                  uint16_t* __restrict__ du_T) {
  const AccMap2<true> mp;
  const int jl0 = mp.col(0);  // tile-relative first of the lane's 4 columns
  const int j0 = n0 + jl0;
  const int tr0 = mp.row(0, 0);  // tile-relative first token of the lane
  const int64_t lane_off = (int64_t)(m0 + tr0) * d_ff + j0;  // element (token m0 + tr0, column j0)
  char* lds = reinterpret_cast<char*>(sm.s);
#pragma unroll
  for (int pass = 0; pass < 2; ++pass) {
    // group k = 4 f + g: tokens m0 + tr0 + 32 f + 8 g .. + 3 (a uniform step from the lane's first)
    auto load = [&](int k, u32x2 (&qv)[4], u32x2 (&uv)[4]) {
      const int dt = 32 * (k >> 2) + 8 * (k & 3);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int64_t o = lane_off + (int64_t)(dt + r) * d_ff;
        qv[r] = *reinterpret_cast<const u32x2*>(q + o);
        uv[r] = pass == 0 ? *reinterpret_cast<const u32x2*>(u + o) : u32x2{0u, 0u};
      }
    };
    u32x2 qn[4], un[4];
    load(0, qn, un);
#pragma unroll
    for (int k = 0; k < 16; ++k) {
      const int f = k >> 2, g = k & 3;
      u32x2 qv[4], uv[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        qv[r] = qn[r];
        uv[r] = un[r];
      }
      if (k + 1 < 16) load(k + 1, qn, un);
      const int tl0 = mp.row(f, 4 * g);  // tile-relative tokens tl0 .. tl0 + 3
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        float v[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const uint32_t qw = qv[r][i >> 1], uw = uv[r][i >> 1];
          const float qq = (i & 1) ? bf16_hi(qw) : bf16_lo(qw);
          const float uu = (i & 1) ? bf16_hi(uw) : bf16_lo(uw);
          // read from its accumulator register at each use (both passes),
          // so no pass keeps a copy of the whole tile in vector registers
          float e;
          asm volatile("v_accvgpr_read_b32 %0, %1" : "=v"(e) : "a"(acc[f][i][4 * g + r]));
          // SiLU(q) = q sg, SiLU'(q) = sg (1 + q (1 - sg)); the reciprocal to
          // about 1 ulp (the values are rounded to bf16 next)
          const float sg = __builtin_amdgcn_rcpf(1.0f + __expf(-qq));
          v[r] = pass == 0 ? e * uu * sg * (1.0f + qq * (1.0f - sg)) : e * qq * sg;
        }
        const int jl = jl0 + i;
        const int pos = ((tl0 >> 3) ^ ((jl >> 2) & 31)) * 16 + ((tl0 >> 2) & 1) * 8;
        *reinterpret_cast<u32x2*>(lds + jl * 512 + pos) = u32x2{pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3])};
      }
    }
    __syncthreads();
    uint16_t* dst = pass == 0 ? dq_T : du_T;
    const int c = threadIdx.x & 31;
#pragma unroll 4
    for (int kk = 0; kk < 32; ++kk) {
      const int jl = (int)(threadIdx.x >> 5) + 8 * kk;
      const int t = m0 + 8 * c;
      *reinterpret_cast<u32x4*>(dst + (int64_t)(n0 + jl) * Tp + t) =
            *reinterpret_cast<const u32x4*>(lds + jl * 512 + ((c ^ ((jl >> 2) & 31)) * 16));
    }
    __syncthreads();
  }
}

template <class E, bool FAST>
__global__ __launch_bounds__(256, 1) void errh_kernel(const typename E::T* __restrict__ g,
                                                      const typename E::T* __restrict__ W3i,
                                                      const typename E::T* __restrict__ q,
                                                      const typename E::T* __restrict__ u, int T,
                                                      int Tp, int d, int d_ff,
                                                      typename E::T* __restrict__ dq_T,
                                                      typename E::T* __restrict__ du_T) {
  using TT = Tile<E>;
  const int ntm = (Tp + TT::BM - 1) / TT::BM, ntn = (d_ff + TT::BN - 1) / TT::BN;
  int tm, tn;
  grouped_tile(xcd_remap(blockIdx.x, gridDim.x), ntm, ntn, 8, tm, tn);
  const int m0 = tm * TT::BM, n0 = tn * TT::BN;
  if constexpr (E::EPC == 8) {
    __shared__ G2Smem sm;
    f32x16 acc[4][4];
    zero_acc2(acc);
    const Operand A{g + (int64_t)m0 * d, d, band_bytes(T - m0, d)};
    const Operand B{W3i + n0, d_ff, band_bytes(d, d_ff, n0)};
    gemm2_mainloop<true, FAST>(sm, acc, A, B, T - m0, d_ff - n0, d, 0, (d + G2::BK - 1) / G2::BK);
    if constexpr (FAST)
      errh_epilogue_lds(acc, sm, m0, n0, q, u, Tp, d_ff, dq_T, du_T);
    else
      errh_epilogue2(acc, m0, n0, q, u, T, Tp, d_ff, dq_T, du_T);
  } else {
    __shared__ GemmSmem<E> sm;
    f32x4 acc[E::FM][E::FN];
    zero_acc<E>(acc);
    gemm_mainloop<E, true>(sm, acc, g, d, T, W3i, d_ff, d_ff, d, m0, n0, 0,
                           (d + TT::BK - 1) / TT::BK, NoHook{});
    errh_epilogue<typename E::T>(acc, AccMap<E>(), m0, n0, q, u, T, Tp, d_ff, dq_T, du_T);
  }
}

// Fixed-order float64 sums of one matrix's tile partials per workgroup:
// ||C||^2 (into sumsq[mat_base + mat]) and, against a reference R, <C, R>,
// ||R||^2 and cos = <C, R> / (||C|| ||R||) (0 when either norm is 0; eq. cosine).
__global__ __launch_bounds__(256) void reduce_parts_kernel(const double* __restrict__ part,
                                                           int ntiles, int mat_base,
                                                           double* __restrict__ sumsq,
                                                           double* __restrict__ dot,
                                                           double* __restrict__ refsq,
                                                           float* __restrict__ cos) {
  __shared__ double red[16];
  const int mat = blockIdx.x;
  const double* p = part + (int64_t)mat * ntiles * 3;
  double a = 0.0, b = 0.0, c = 0.0;
  for (int t = threadIdx.x; t < ntiles; t += 256) {
    a += p[3 * t];
    b += p[3 * t + 1];
    c += p[3 * t + 2];
  }
  a = block_sum_d(a, red);
  b = block_sum_d(b, red);
  c = block_sum_d(c, red);
  if (threadIdx.x == 0) {
    if (sumsq) sumsq[mat_base + mat] = a;
    if (dot) dot[mat] = b;
    if (refsq) refsq[mat] = c;
    if (cos) cos[mat] = (a == 0.0 || c == 0.0) ? 0.f : (float)(b / sqrt(a * c));
  }
}

int64_t pseudograd_tiles(bool bf16, int64_t M, int64_t N) {
  const int BM = bf16 ? TileBF16::BM : TileF32::BM, BN = bf16 ? TileBF16::BN : TileF32::BN;
  return ((M + BM - 1) / BM) * ((N + BN - 1) / BN);
}

#define FPO_CHECK_LAUNCH()             \
  do {                                 \
    hipError_t e_ = hipGetLastError(); \
    if (e_ != hipSuccess) return e_;   \
  } while (0)

// Left operands of every layer, formed before any outer product (while HBM is
// otherwise idle): the shared signal's token-contiguous copy in a.gT, or, with
// a norm chain (post-FFN and / or pre-MLP composition), each layer's composed
// signal in a.gT + l * d * Tp (and row-major in a.g_row + l * T * d for the
// full-MLP error GEMM).
template <typename T, bool POST, bool PRE>
static hipError_t prepare_chain(const PgLaunch& a, hipStream_t st, dim3 grid) {
  constexpr int CHAIN = (POST ? 1 : 0) | (PRE ? 2 : 0);
  for (int l = 0; l < a.L; ++l) {
    const T* x1 = POST ? (const T*)a.mlp_out[l] : nullptr;
    const T* g1 = POST ? (const T*)a.gamma_pffn[l] : nullptr;
    const T* x2 = PRE ? (const T*)a.pre_in[l] : nullptr;
    const T* g2 = PRE ? (const T*)a.gamma_pre[l] : nullptr;
    FPO_LAUNCH("chain_stats", st,
               chain_stats_kernel<T, POST, PRE><<<dim3((unsigned)a.T), dim3(256), 0, st>>>(
        (int)a.d, a.g_f32, x1, g1, a.pffn_eps, a.pffn_min_rms, x2, g2, a.pre_eps, a.pre_min_rms,
        (float4*)a.chain_stats));
    FPO_CHECK_LAUNCH();
    T* row = a.full_mlp ? (T*)a.g_row + (int64_t)l * a.T * a.d : nullptr;
    FPO_LAUNCH("signal_transpose", st,
               signal_transpose_kernel<T, CHAIN><<<grid, dim3(256), 0, st>>>(
        a.g_f32, x1, g1, x2, g2, (const float4*)a.chain_stats, a.T, a.d, (T*)a.gT + (int64_t)l * a.d * a.Tp,
        a.Tp, a.Tp, row));
    FPO_CHECK_LAUNCH();
  }
  return hipSuccess;
}

template <typename T>
static hipError_t prepare_signals(const PgLaunch& a, hipStream_t st) {
  const dim3 grid((unsigned)(a.Tp / 64), (unsigned)((a.d + 63) / 64));
  if (a.pffn && a.pre) return prepare_chain<T, true, true>(a, st, grid);
  if (a.pffn) return prepare_chain<T, true, false>(a, st, grid);
  if (a.pre) return prepare_chain<T, false, true>(a, st, grid);
  FPO_LAUNCH("signal_transpose", st,
             signal_transpose_kernel<T, 0><<<grid, dim3(256), 0, st>>>(
      a.g_lp, nullptr, nullptr, nullptr, nullptr, nullptr, a.T, a.d, (T*)a.gT, a.Tp, a.Tp, nullptr));
  FPO_CHECK_LAUNCH();
  return hipSuccess;
}

// Layer l's token-contiguous left operand [d, Tp] and its row-major form [T, d].
template <typename T>
static const T* signal_T(const PgLaunch& a, int l) {
  return (const T*)a.gT + ((a.pffn || a.pre) ? (int64_t)l * a.d * a.Tp : 0);
}
template <typename T>
static const T* signal_rows(const PgLaunch& a, int l) {
  return (a.pffn || a.pre) ? (const T*)a.g_row + (int64_t)l * a.T * a.d : (const T*)a.g_lp;
}

// Whole 256 x 256 tiles and 64-deep K tiles (M, N multiples of 256, K of 64)
// take the GEMM core's copy form without bounds selects.
static bool whole_tiles(int64_t M, int64_t N, int64_t K) {
  return M % 256 == 0 && N % 256 == 0 && K % 64 == 0;
}

template <class E>
static void launch_outer(dim3 grid, hipStream_t st, const OuterArgs& oa, int M, int N, int K, int64_t lda,
                         int64_t ldb, float scale, double* part) {
  if (whole_tiles(M, N, K))
    outer_kernel<E, true><<<grid, dim3(256), 0, st>>>(oa, M, N, K, lda, ldb, scale, part);
  else
    outer_kernel<E, false><<<grid, dim3(256), 0, st>>>(oa, M, N, K, lda, ldb, scale, part);
}

template <class E>
static void launch_errh(dim3 grid, hipStream_t st, const typename E::T* g, const typename E::T* W3i,
                        const typename E::T* q, const typename E::T* u, int T, int Tp, int d, int d_ff,
                        typename E::T* dq_T, typename E::T* du_T) {
  if (whole_tiles(T, d_ff, d))
    errh_kernel<E, true><<<grid, dim3(256), 0, st>>>(g, W3i, q, u, T, Tp, d, d_ff, dq_T, du_T);
  else
    errh_kernel<E, false><<<grid, dim3(256), 0, st>>>(g, W3i, q, u, T, Tp, d, d_ff, dq_T, du_T);
}

template <class E>
static hipError_t run_pseudograd(const PgLaunch& a) {
  using T = typename E::T;
  using TT = Tile<E>;
  hipStream_t st = (hipStream_t)a.stream;
  const int ntiles = (int)pseudograd_tiles(a.bf16, a.d, a.d_ff);
  const int ntiles2 = (int)pseudograd_tiles(a.bf16, a.d_ff, a.d);
  hipError_t e;
  if ((e = prepare_signals<T>(a, st)) != hipSuccess) return e;
  // W3 outer products of every layer (M = d, N = d_ff, K = T) in one launch
  {
    OuterArgs oa{};
    for (int l = 0; l < a.L; ++l) {
      oa.A[l] = signal_T<T>(a, l);
      oa.B[l] = a.a[l];
      oa.C[l] = a.dW3[l];
      oa.Cb[l] = a.dW3_bf16[l];
      oa.R[l] = a.ref[l];
    }
    FPO_LAUNCH("outer", st,
               launch_outer<E>(dim3(ntiles * a.L), st, oa, (int)a.d, (int)a.d_ff, (int)a.T, a.Tp, a.d_ff,
                               a.scale, a.part));
    FPO_CHECK_LAUNCH();
    FPO_LAUNCH("reduce_parts", st,
               reduce_parts_kernel<<<dim3(a.L), dim3(256), 0, st>>>(a.part, ntiles, 0, a.sumsq, a.ref_dot,
                                                         a.ref_sumsq, a.ref_cos));
    FPO_CHECK_LAUNCH();
  }
  if (!a.full_mlp) return hipSuccess;
  // W1/W2 signals through W3_init (eq. errh), one layer at a time
  for (int l = 0; l < a.L; ++l) {
    FPO_LAUNCH("errh", st,
               launch_errh<E>(dim3((unsigned)(((a.Tp + TT::BM - 1) / TT::BM) * ((a.d_ff + TT::BN - 1) / TT::BN))),
                              st, signal_rows<T>(a, l), (const T*)a.W3i[l], (const T*)a.q[l],
                              (const T*)a.u[l], (int)a.T, (int)a.Tp, (int)a.d, (int)a.d_ff, (T*)a.dq_T,
                              (T*)a.du_T));
    FPO_CHECK_LAUNCH();
    OuterArgs oa{};
    oa.A[0] = a.dq_T;
    oa.B[0] = a.x_in[l];
    oa.C[0] = a.dW1[l];
    oa.A[1] = a.du_T;
    oa.B[1] = a.x_in[l];
    oa.C[1] = a.dW2[l];
    FPO_LAUNCH("outer", st,
               launch_outer<E>(dim3(ntiles2 * 2), st, oa, (int)a.d_ff, (int)a.d, (int)a.T, a.Tp, a.d, a.scale,
                               a.part));
    FPO_CHECK_LAUNCH();
    // matrices W1(l) and W2(l) sit at a.L + l and 2 a.L + l of sumsq
    if (a.sumsq) {
      FPO_LAUNCH("reduce_parts", st,
                 reduce_parts_kernel<<<dim3(1), dim3(256), 0, st>>>(a.part, ntiles2, a.L + l, a.sumsq,
                                                         nullptr, nullptr, nullptr));
      FPO_CHECK_LAUNCH();
      FPO_LAUNCH("reduce_parts", st,
                 reduce_parts_kernel<<<dim3(1), dim3(256), 0, st>>>(a.part + (int64_t)ntiles2 * 3, ntiles2,
                                                         2 * a.L + l, a.sumsq, nullptr, nullptr, nullptr));
      FPO_CHECK_LAUNCH();
    }
  }
  return hipSuccess;
}

// Side stream and events of one device for the overlapped pseudogradient +
// update (created on first use, kept until the process ends; one call's
// enqueue sequence holds the device's lock).
struct PgOverlap {
  std::mutex mu;
  bool ready = false;
  hipStream_t side = nullptr;
  hipEvent_t ready_l = nullptr, done = nullptr;
  int cus = 0;  // compute units: workgroups of an update that runs beside the outer products
};
constexpr int kMaxDevices = 64;
static PgOverlap g_pgo[kMaxDevices];

static hipError_t pg_overlap_init(PgOverlap& p, int dev) {
  if (p.ready) return hipSuccess;
  hipError_t e;
  if ((e = hipDeviceGetAttribute(&p.cus, hipDeviceAttributeMultiprocessorCount, dev)) != hipSuccess) return e;
  // default priority: both streams at the same priority
  if ((e = hipStreamCreateWithFlags(&p.side, hipStreamNonBlocking)) != hipSuccess) return e;
  if ((e = hipEventCreateWithFlags(&p.ready_l, hipEventDisableTiming)) != hipSuccess) return e;
  if ((e = hipEventCreateWithFlags(&p.done, hipEventDisableTiming)) != hipSuccess) return e;
  p.ready = true;
  return hipSuccess;
}

// bf16 pseudogradient with the optimizer step overlapped: the outer products
// run one layer per launch on the caller's stream; once a matrix's tiles are
// done, its norm and update (few registers and no LDS, so its workgroups sit
// beside an outer-product GEMM's on the same CUs) stream on a side stream while
// the following launches run, with one workgroup per CU so that each CU holds
// one GEMM workgroup and one update workgroup; the updates released by the last
// launch have the machine to itself. With the full MLP, the W3 launches come
// first, then per layer the W1/W2 signal GEMM (eq. errh: all registers, so an
// update workgroup and an errh workgroup take turns on a CU) and one launch of
// both W1/W2 outer products, which releases both updates. Same per-block arithmetic and reduction order as the
// separate calls, so results are bit-identical to them. The side stream and its
// two events are the caller's (ov) or, when ov is null, the device's
// library-owned set, whose enqueue sequence is serialised by a lock.
static hipError_t enqueue_pseudograd_update(const PgLaunch& a, const UpdLaunch& u, hipStream_t side,
                                            hipEvent_t ready_l, hipEvent_t done, int cus);

hipError_t launch_pseudograd_update(const PgLaunch& a, const UpdLaunch& u, const OverlapLaunch* ov) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  PgOverlap& po = g_pgo[dev];
  if (ov) {
    int cus = 0;
    if ((e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev)) != hipSuccess) return e;
    return enqueue_pseudograd_update(a, u, (hipStream_t)ov->side, (hipEvent_t)ov->ready, (hipEvent_t)ov->done,
                                     cus);
  }
  std::lock_guard<std::mutex> lock(po.mu);
  if ((e = pg_overlap_init(po, dev)) != hipSuccess) return e;
  return enqueue_pseudograd_update(a, u, po.side, po.ready_l, po.done, po.cus);
}

static hipError_t enqueue_pseudograd_update(const PgLaunch& a, const UpdLaunch& u, hipStream_t side,
                                            hipEvent_t ready_l, hipEvent_t done, int cus) {
  hipStream_t st = (hipStream_t)a.stream;
  hipError_t e;
  if ((e = prepare_signals<uint16_t>(a, st)) != hipSuccess) return e;
  const int ntiles = (int)pseudograd_tiles(true, a.d, a.d_ff);
  const int ntiles2 = (int)pseudograd_tiles(true, a.d_ff, a.d);
  // matrix m: W3 of layer m (m < L), then W1 and W2 of layer l at L + l and
  // 2 L + l; its update blocks start at the sum of the earlier matrices'
  // blocks. Tile partials have a region per matrix (the side stream reads them
  // while later launches run): slot l for W3 of layer l, slots L + 2l and
  // L + 2l + 1 for W1 and W2 of layer l (one launch writes both, the second
  // matrix's partials right after the first's).
  const int nm = a.full_mlp ? 3 * a.L : a.L;
  int64_t blk_base[kMaxMats + 1];
  blk_base[0] = 0;
  for (int m = 0; m < nm; ++m) blk_base[m + 1] = blk_base[m] + update_blocks(u.numel[m]);
  auto tpart = [&](int slot) { return a.part + (int64_t)slot * ntiles * 3; };
  // the norm reduction and the update of matrix m (partials in `slot`) on the
  // side stream, after the launch just enqueued on st; `alone`: no GEMM
  // follows to share the CUs
  auto release = [&](int m, int slot, int nt, bool ref, bool alone) -> hipError_t {
    FPO_LAUNCH("reduce_parts", side,
               reduce_parts_kernel<<<dim3(1), dim3(256), 0, side>>>(
        tpart(slot), nt, m, a.sumsq, ref && a.ref_dot ? a.ref_dot + m : nullptr,
        ref && a.ref_sumsq ? a.ref_sumsq + m : nullptr, ref && a.ref_cos ? a.ref_cos + m : nullptr));
    FPO_CHECK_LAUNCH();
    // one workgroup per CU beside the next GEMM launch; the last updates run
    // alone and take the whole machine
    return launch_update_blocks(u, m, blk_base[m], side, alone ? 0 : cus);
  };
  auto handoff = [&]() -> hipError_t {
    hipError_t r;
    if ((r = hipEventRecord(ready_l, st)) != hipSuccess) return r;
    return hipStreamWaitEvent(side, ready_l, 0);
  };
  for (int l = 0; l < a.L; ++l) {
    OuterArgs oa{};
    oa.A[0] = signal_T<uint16_t>(a, l);
    oa.B[0] = a.a[l];
    oa.C[0] = a.dW3[l];
    oa.Cb[0] = a.dW3_bf16[l];
    oa.R[0] = a.ref[l];
    FPO_LAUNCH("outer", st,
               launch_outer<TileBF16>(dim3(ntiles), st, oa, (int)a.d, (int)a.d_ff, (int)a.T, a.Tp, a.d_ff,
                                      a.scale, tpart(l)));
    FPO_CHECK_LAUNCH();
    // layer l's tiles are complete: its norm reduction and update follow on the
    // side stream, so the next layer's outer products start right away
    if ((e = handoff()) != hipSuccess) return e;
    if ((e = release(l, l, ntiles, true, !a.full_mlp && l + 1 == a.L)) != hipSuccess) return e;
  }
  // full MLP: W1/W2 signals through W3_init (eq. errh), then both outer
  // products of the layer in one launch, their updates released together
  for (int l = 0; a.full_mlp && l < a.L; ++l) {
    FPO_LAUNCH("errh", st,
               launch_errh<TileBF16>(dim3((unsigned)(((a.Tp + 255) / 256) * ((a.d_ff + 255) / 256))), st,
                                     signal_rows<uint16_t>(a, l), (const uint16_t*)a.W3i[l],
                                     (const uint16_t*)a.q[l], (const uint16_t*)a.u[l], (int)a.T, (int)a.Tp,
                                     (int)a.d, (int)a.d_ff, (uint16_t*)a.dq_T, (uint16_t*)a.du_T));
    FPO_CHECK_LAUNCH();
    const int m1 = a.L + l, m2 = 2 * a.L + l;
    OuterArgs oa{};
    oa.A[0] = a.dq_T;
    oa.B[0] = a.x_in[l];
    oa.C[0] = a.dW1[l];
    oa.A[1] = a.du_T;
    oa.B[1] = a.x_in[l];
    oa.C[1] = a.dW2[l];
    const int slot = a.L + 2 * l;  // ntiles2 == ntiles (256 x 256 tiles of d x d_ff or d_ff x d)
    FPO_LAUNCH("outer", st,
               launch_outer<TileBF16>(dim3(ntiles2 * 2), st, oa, (int)a.d_ff, (int)a.d, (int)a.T, a.Tp, a.d,
                                      a.scale, tpart(slot)));
    FPO_CHECK_LAUNCH();
    if ((e = handoff()) != hipSuccess) return e;
    const bool last = l + 1 == a.L;
    if ((e = release(m1, slot, ntiles2, false, last)) != hipSuccess) return e;
    if ((e = release(m2, slot + 1, ntiles2, false, last)) != hipSuccess) return e;
  }
  if ((e = hipEventRecord(done, side)) != hipSuccess) return e;
  if ((e = hipStreamWaitEvent(st, done, 0)) != hipSuccess) return e;
  // ||W'||^2 and the clip factors of every matrix
  return launch_update(u, false);
}

hipError_t launch_pseudograd(const PgLaunch& a) {
  return a.bf16 ? run_pseudograd<TileBF16>(a) : run_pseudograd<TileF32>(a);
}

}  // namespace fpo
