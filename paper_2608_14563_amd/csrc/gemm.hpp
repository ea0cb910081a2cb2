// fp32 MFMA tile core for the three contractions of the FPO hot path on
// gfx950 (the logits Y W_U^T, the projection P W_U and the per-layer outer
// product g~^T a) when the operands are fp32: one workgroup of 4 waves (2 x 2)
// computes a 128 x 128 tile of C = A B with v_mfma_f32_16x16x4_f32 (exact
// fp32 products, fp32 accumulation), A stored K-contiguous ([M][K]
// row-major) and B either K-contiguous ([N][K], "Bt") or N-contiguous
// ([K][N]); 32-deep K tiles, register-staged double buffering. bf16 operands
// run on the LDS-DMA core of gemm2.hpp; TileBF16 here only carries their tile
// constants.
//
// Lane layout. Within one 32-wide K step every lane l owns the eight K
// indices 8*(l>>4) + s, s = 0..7, for both operands (the K order inside the
// sum is a summation order only). Output columns are interleaved: the lane
// owns columns FN*(l&15) + i, i = 0..FN-1, of its wave's tile, so that its
// FN accumulator blocks hold FN consecutive output columns (16-byte epilogue
// stores) and an N-contiguous B tile is read with one 16-byte LDS load per K
// row.
//
// Accumulator acc[f][i][r] holds C[row, col] with
//   row = m0 + wm*WTM + 16*f + 4*(l>>4) + r,  col = n0 + wn*WTN + FN*(l&15) + i.
//
// K-contiguous LDS tiles are stored in 16-byte chunks, 8 chunks per row, with
// chunk index XOR-swizzled by (row ^ (row >> 3)) & 7 so that the lanes of a
// fragment read (consecutive rows, or rows 8 apart) hit distinct banks.
#pragma once

#include "common.hpp"

namespace fpo {

struct TileBF16 {
  using T = uint16_t;
  static constexpr int BM = 256, BN = 256, BK = 64, FM = 8, FN = 8, EPC = 8;
};
struct TileF32 {
  using T = float;
  static constexpr int BM = 128, BN = 128, BK = 32, FM = 4, FN = 4, EPC = 4;
};

template <class E>
struct Tile {
  using T = typename E::T;
  static constexpr int BM = E::BM, BN = E::BN, BK = E::BK, FM = E::FM, FN = E::FN, EPC = E::EPC;
  static constexpr int NT = 256;                 // threads per workgroup
  static constexpr int WTM = 16 * FM, WTN = 16 * FN;
  static constexpr int CPR = BK / EPC;           // chunks per K-contiguous row (8)
  static constexpr int KSTEPS = BK / 32;
  static constexpr int KC = 8 / EPC;             // chunks per lane per K step
  static constexpr int A_CHUNKS = BM * CPR;
  static constexpr int B_CHUNKS = BN * CPR;      // == BK * BN / EPC
  static constexpr int BN_CPR = BN / EPC;        // chunks per N-contiguous row (32)
  static constexpr int A_PT = A_CHUNKS / NT;
  static constexpr int BT_PT = B_CHUNKS / NT;
  static constexpr int BNC_PT = (BK * BN_CPR) / NT;
  static_assert(CPR == 8, "swizzle assumes 8 chunks per row");
  static_assert(BN_CPR == 32, "N-contiguous loader assumes 32 chunks per row");
};

template <class E>
struct GemmSmem {
  u32x4 a[2][Tile<E>::A_CHUNKS];
  u32x4 b[2][Tile<E>::B_CHUNKS];
};

__device__ __forceinline__ int swz(int row) { return (row ^ (row >> 3)) & 7; }

// ---------------------------------------------------------------- loaders
template <class E, bool BNC>
struct TileLoader {
  using TT = Tile<E>;
  using T = typename E::T;
  u32x4 ra[TT::A_PT];
  u32x4 rb[BNC ? TT::BNC_PT : TT::BT_PT];

  // A [M][lda] K-contiguous. Rows >= M and chunks >= K read as zero
  // (K is a multiple of EPC).
  __device__ __forceinline__ void load_a(const T* __restrict__ A, int64_t lda, int M, int K, int m0,
                                         int k0) {
    const int t = threadIdx.x;
#pragma unroll
    for (int j = 0; j < TT::A_PT; ++j) {
      const int row = (t >> 3) + 32 * j, c = t & 7;
      const int gm = m0 + row, gk = k0 + c * TT::EPC;
      u32x4 v = {0u, 0u, 0u, 0u};
      if (gm < M && gk < K) v = *reinterpret_cast<const u32x4*>(A + (int64_t)gm * lda + gk);
      ra[j] = v;
    }
  }
  __device__ __forceinline__ void store_a(u32x4* sa) {
    const int t = threadIdx.x;
#pragma unroll
    for (int j = 0; j < TT::A_PT; ++j) {
      const int row = (t >> 3) + 32 * j, c = t & 7;
      sa[row * 8 + (c ^ swz(row))] = ra[j];
    }
  }
  // B: N-contiguous [K][ldb] (BNC) or K-contiguous [N][ldb].
  __device__ __forceinline__ void load_b(const T* __restrict__ B, int64_t ldb, int N, int K, int n0,
                                         int k0) {
    const int t = threadIdx.x;
    if constexpr (BNC) {
#pragma unroll
      for (int j = 0; j < TT::BNC_PT; ++j) {
        const int row = (t >> 5) + 8 * j, c = t & 31;
        const int gk = k0 + row, gn = n0 + c * TT::EPC;
        u32x4 v = {0u, 0u, 0u, 0u};
        if (gk < K && gn < N) v = *reinterpret_cast<const u32x4*>(B + (int64_t)gk * ldb + gn);
        rb[j] = v;
      }
    } else {
#pragma unroll
      for (int j = 0; j < TT::BT_PT; ++j) {
        const int row = (t >> 3) + 32 * j, c = t & 7;
        const int gn = n0 + row, gk = k0 + c * TT::EPC;
        u32x4 v = {0u, 0u, 0u, 0u};
        if (gn < N && gk < K) v = *reinterpret_cast<const u32x4*>(B + (int64_t)gn * ldb + gk);
        rb[j] = v;
      }
    }
  }
  __device__ __forceinline__ void store_b(u32x4* sb) {
    const int t = threadIdx.x;
    if constexpr (BNC) {
#pragma unroll
      for (int j = 0; j < TT::BNC_PT; ++j) {
        const int row = (t >> 5) + 8 * j, c = t & 31;
        sb[row * 32 + c] = rb[j];
      }
    } else {
#pragma unroll
      for (int j = 0; j < TT::BT_PT; ++j) {
        const int row = (t >> 3) + 32 * j, c = t & 7;
        sb[row * 8 + (c ^ swz(row))] = rb[j];
      }
    }
  }
};

// ---------------------------------------------------------------- compute
template <bool BNC>
__device__ __forceinline__ void mma_tile_f32(const u32x4* __restrict__ sa,
                                             const u32x4* __restrict__ sb,
                                             f32x4 (&acc)[4][4], int wm, int wn) {
  using TT = Tile<TileF32>;
  const int l = threadIdx.x & 63;
  const int lr = l & 15, lg = l >> 4;
#pragma unroll
  for (int ks = 0; ks < TT::KSTEPS; ++ks) {
    float av[4][8];
#pragma unroll
    for (int f = 0; f < 4; ++f) {
      const int row = wm * TT::WTM + 16 * f + lr;
#pragma unroll
      for (int q = 0; q < 2; ++q) {
        u32x4 c = sa[row * 8 + ((ks * 8 + 2 * lg + q) ^ swz(row))];
#pragma unroll
        for (int e = 0; e < 4; ++e) av[f][4 * q + e] = __uint_as_float(c[e]);
      }
    }
    float bv[8][4];
    if constexpr (BNC) {
#pragma unroll
      for (int s = 0; s < 8; ++s) {
        const int k = ks * 32 + 8 * lg + s;
        u32x4 c = sb[k * 32 + wn * (TT::WTN / 4) + lr];
#pragma unroll
        for (int i = 0; i < 4; ++i) bv[s][i] = __uint_as_float(c[i]);
      }
    } else {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int row = wn * TT::WTN + 4 * lr + i;
#pragma unroll
        for (int q = 0; q < 2; ++q) {
          u32x4 c = sb[row * 8 + ((ks * 8 + 2 * lg + q) ^ swz(row))];
#pragma unroll
          for (int e = 0; e < 4; ++e) bv[4 * q + e][i] = __uint_as_float(c[e]);
        }
      }
    }
#pragma unroll
    for (int s = 0; s < 8; ++s)
#pragma unroll
      for (int f = 0; f < 4; ++f)
#pragma unroll
        for (int i = 0; i < 4; ++i)
          acc[f][i] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[f][s], bv[s][i], acc[f][i], 0, 0, 0);
  }
}

template <class E, bool BNC>
__device__ __forceinline__ void mma_tile(const u32x4* sa, const u32x4* sb,
                                         f32x4 (&acc)[E::FM][E::FN], int wm, int wn) {
  static_assert(E::EPC == 4, "this core computes fp32 tiles only");
  mma_tile_f32<BNC>(sa, sb, acc, wm, wn);
}

struct NoHook {
  template <class Acc>
  __device__ __forceinline__ void operator()(int, Acc&) const {}
};

// Main loop over K tiles [kt0, kt1) with LDS double buffering and register
// prefetch of the next tile. `hook(kt, acc)` runs before tile kt's products
// are accumulated. Ends with a barrier, so the caller may reuse LDS.
template <class E, bool BNC, class Hook>
__device__ __forceinline__ void gemm_mainloop(GemmSmem<E>& sm, f32x4 (&acc)[E::FM][E::FN],
                                              const typename E::T* __restrict__ A, int64_t lda,
                                              int M, const typename E::T* __restrict__ B,
                                              int64_t ldb, int N, int K, int m0, int n0, int kt0,
                                              int kt1, const Hook& hook) {
  using TT = Tile<E>;
  const int w = threadIdx.x >> 6;
  const int wm = w >> 1, wn = w & 1;
  TileLoader<E, BNC> ld;
  if (kt0 >= kt1) return;
  ld.load_a(A, lda, M, K, m0, kt0 * TT::BK);
  ld.load_b(B, ldb, N, K, n0, kt0 * TT::BK);
  ld.store_a(sm.a[0]);
  ld.store_b(sm.b[0]);
  __syncthreads();
  for (int kt = kt0; kt < kt1; ++kt) {
    const int cur = (kt - kt0) & 1;
    const bool more = kt + 1 < kt1;
    if (more) {
      ld.load_a(A, lda, M, K, m0, (kt + 1) * TT::BK);
      ld.load_b(B, ldb, N, K, n0, (kt + 1) * TT::BK);
    }
    hook(kt, acc);
    mma_tile<E, BNC>(sm.a[cur], sm.b[cur], acc, wm, wn);
    if (more) {
      ld.store_a(sm.a[cur ^ 1]);
      ld.store_b(sm.b[cur ^ 1]);
    }
    __syncthreads();
  }
}

template <class E>
__device__ __forceinline__ void zero_acc(f32x4 (&acc)[E::FM][E::FN]) {
#pragma unroll
  for (int f = 0; f < E::FM; ++f)
#pragma unroll
    for (int i = 0; i < E::FN; ++i) acc[f][i] = f32x4{0.f, 0.f, 0.f, 0.f};
}

// Workgroup -> tile mapping. Consecutive workgroup ids are dispatched
// round-robin over the 8 XCDs, each with its own L2. xcd_remap gives every
// XCD a contiguous range of logical tile ids; grouped_tile walks a range in
// groups of `gm` tile rows, so the workgroups resident on one XCD at a time
// cover a few tile rows x a few tile columns and share A rows and B columns
// in that XCD's L2 while they stream through K together.
constexpr int kXcds = 8;

__device__ __forceinline__ int xcd_remap(int bid, int nblk) {
  const int xcd = bid % kXcds, slot = bid / kXcds;
  const int per = nblk / kXcds, rem = nblk % kXcds;
  return xcd * per + (xcd < rem ? xcd : rem) + slot;
}

__device__ __forceinline__ void grouped_tile(int id, int ntm, int ntn, int gm, int& tm, int& tn) {
  const int width = gm * ntn;
  const int first = (id / width) * gm;
  const int rows = (ntm - first) < gm ? (ntm - first) : gm;
  const int r = id % width;
  tm = first + r % rows;
  tn = r / rows;
}

// Output coordinates of accumulator element [f][i][r] (relative to the tile).
template <class E>
struct AccMap {
  static constexpr int R = 4;     // accumulator elements per (f, i): rows 4 consecutive
  static constexpr int LPR = 16;  // lanes sharing one output row
  int row0, col0;  // tile-relative row of (f=0, r=0), col of i=0
  __device__ __forceinline__ AccMap() {
    const int l = threadIdx.x & 63, w = threadIdx.x >> 6;
    row0 = (w >> 1) * Tile<E>::WTM + 4 * (l >> 4);
    col0 = (w & 1) * Tile<E>::WTN + E::FN * (l & 15);
  }
  __device__ __forceinline__ int row(int f, int r) const { return row0 + 16 * f + r; }
  __device__ __forceinline__ int col(int i) const { return col0 + i; }
};

}  // namespace fpo
