// bf16 MFMA tile core with a 4-stage LDS ring fed by LDS-DMA buffer loads
// (gfx950 buffer_load_dwordx4 ... lds). One workgroup of 4 waves (2 x 2)
// computes a 256 x 256 tile of C = A B, A K-contiguous ([M][K]), B either
// N-contiguous ([K][N]) or K-contiguous ([N][K], "Bt"). K advances 32 per
// stage, one v_mfma_f32_16x16x32_bf16 K step.
//
// Pipeline: tiles kt+1..kt+3 are in flight while tile kt is multiplied; the
// global->LDS copies go straight into LDS (no register staging), each wave
// instruction filling 1 KB of LDS at base + 16 * lane. Out-of-range rows or
// K chunks are given a buffer offset beyond the resource and read as zero.
// One barrier per stage: a stage is refilled only after every wave has passed
// the barrier that follows its last use.
//
// LDS layouts (16-byte chunks):
//   K-contiguous tile: [rows][4 chunks], chunk c of row r stored at position
//     c ^ ((r >> 1) & 3) -- fragment reads of 16 consecutive rows are then
//     bank-conflict free on gfx950 (measured).
//   N-contiguous tile: [32 K rows][32 chunks] as in memory (conflict free).
// Lane layout of the MFMA operands as in gemm.hpp: lane l owns K indices
// 8*(l>>4) + s of the step. Output columns: for an N-contiguous B the lane owns
// 8 consecutive columns 8*(l&15) + i of its wave's 128; for a K-contiguous B
// it owns columns 16*i + (l&15).
#pragma once

#include "common.hpp"

namespace fpo {

struct G2 {
  static constexpr int BM = 256, BN = 256, BK = 32, NST = 4;
  static constexpr int WTM = 128, WTN = 128;
  static constexpr int A_CHUNKS = BM * 4;        // 16 KB
  static constexpr int B_CHUNKS = BN * 4;        // 16 KB
  static constexpr int STAGE_CHUNKS = A_CHUNKS + B_CHUNKS;
  static constexpr int LOADS_PER_STAGE = 8;      // DMA instructions per wave per stage
};

struct G2Smem {
  u32x4 s[G2::NST * G2::STAGE_CHUNKS];  // 128 KB
};

__device__ __forceinline__ int swz4(int row) { return (row >> 1) & 3; }

// One 16-byte-per-lane LDS-DMA copy: lane l's 16 bytes at rsrc + voff land at
// LDS byte address m0 + 16 * l. Issued as inline asm so that the compiler does
// not guard later LDS reads with vmcnt(0) (it cannot tell the ring stages
// apart); completion is tracked explicitly with wait_vmcnt. s_nop covers the
// M0 write -> LDS-DMA wait state.
__device__ __forceinline__ void dma16(u32x4 rsrc, uint32_t lds_addr, uint32_t voff) {
  asm volatile(
      "s_mov_b32 m0, %0\n\t"
      "s_nop 0\n\t"
      "buffer_load_dwordx4 %1, %2, 0 offen lds"
      :
      : "s"(lds_addr), "v"(voff), "s"(rsrc)
      : "memory", "m0");
}

__device__ __forceinline__ uint32_t lds_addr_of(const u32x4* p) {
  return __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)p);
}

// s_waitcnt vmcnt(n) leaving lgkmcnt / expcnt unconstrained (gfx9 encoding:
// vmcnt[3:0] at bits 3:0, vmcnt[5:4] at bits 15:14).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

constexpr uint32_t kOOB = 0x80000000u;  // beyond every resource: reads zero

// Workgroup barrier without the release fence of __syncthreads: the fence
// would make the compiler wait for every outstanding LDS-DMA copy (vmcnt(0)),
// i.e. for the tiles still in flight. Completion of the copies a stage needs
// is ensured by wait_vmcnt before the barrier; the empty asm statements keep
// the compiler from moving LDS accesses across it.
__device__ __forceinline__ void stage_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Operand view for the DMA loader.
struct Operand {
  const uint16_t* base;  // element (0, 0) of the workgroup's tile row/col band
  int64_t ld;            // row stride in elements
  uint32_t bytes;        // bytes addressable from base (resource size)
};

// Bytes from a band base covering `rows` rows of stride `ld` elements, less a
// leading column offset; 0 when the band is empty. Callers keep operand bands
// below 2^31 bytes (checked by the ABI layer), so every in-range offset is
// below kOOB.
__device__ __forceinline__ uint32_t band_bytes(int64_t rows, int64_t ld, int64_t col0 = 0) {
  const int64_t b = rows * ld * 2 - col0 * 2;
  return b > 0 ? (uint32_t)b : 0u;
}

// The resource must live in scalar registers; values derived from per-matrix
// kernel arguments are made provably uniform so the compiler does not wrap each
// copy in a waterfall loop.
// Buffer resource (base, stride 0, num_records = bytes, raw-buffer flags) in
// scalar registers.
__device__ __forceinline__ u32x4 make_rsrc(const Operand& o) {
  const uint64_t v = (uint64_t)(uintptr_t)o.base;
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(v >> 32)) & 0xffffu;
  const uint32_t nb = __builtin_amdgcn_readfirstlane(o.bytes);
  return u32x4{lo, hi, nb, 0x00020000u};
}

template <bool BNC>
struct Pipe2 {
  u32x4 ra, rb;
  int64_t lda, ldb;
  int M_rem, N_rem, K;  // rows of A / cols of B left from the band base; K total

  // Issue the DMA copies of K tile kt into ring stage st.
  __device__ __forceinline__ void issue(u32x4* smem, int st, int kt) const {
    const int w = threadIdx.x >> 6, l = threadIdx.x & 63;
    const int k0 = kt * G2::BK;
    u32x4* sa = smem + st * G2::STAGE_CHUNKS;
    u32x4* sb = sa + G2::A_CHUNKS;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int inst = w * 4 + j;
      const int row = 16 * inst + (l >> 2);
      const int c = (l & 3) ^ swz4(row);
      const int gk = k0 + 8 * c;
      const uint32_t off = (row < M_rem && gk < K) ? (uint32_t)(((int64_t)row * lda + gk) * 2) : kOOB;
      dma16(ra, lds_addr_of(sa + inst * 64), off);
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int inst = w * 4 + j;
      uint32_t off;
      if constexpr (BNC) {
        const int krow = 2 * inst + (l >> 5), c = l & 31;
        const int gk = k0 + krow;
        off = (gk < K && 8 * c < N_rem) ? (uint32_t)(((int64_t)gk * ldb + 8 * c) * 2) : kOOB;
      } else {
        const int row = 16 * inst + (l >> 2);
        const int c = (l & 3) ^ swz4(row);
        const int gk = k0 + 8 * c;
        off = (row < N_rem && gk < K) ? (uint32_t)(((int64_t)row * ldb + gk) * 2) : kOOB;
      }
      dma16(rb, lds_addr_of(sb + inst * 64), off);
    }
  }

  __device__ __forceinline__ static void compute(const u32x4* smem, int st, f32x4 (&acc)[8][8]) {
    const int w = threadIdx.x >> 6, l = threadIdx.x & 63;
    const int wm = w >> 1, wn = w & 1, lr = l & 15, lg = l >> 4;
    const u32x4* sa = smem + st * G2::STAGE_CHUNKS;
    const u32x4* sb = sa + G2::A_CHUNKS;
    u32x4 af[8];
#pragma unroll
    for (int f = 0; f < 8; ++f) {
      const int row = wm * G2::WTM + 16 * f + lr;
      af[f] = sa[row * 4 + (lg ^ swz4(row))];
    }
    u32x4 bo[8];
    if constexpr (BNC) {
      u32x4 raw[8];
#pragma unroll
      for (int s = 0; s < 8; ++s) raw[s] = sb[(8 * lg + s) * 32 + wn * 16 + lr];
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int q = i >> 1;
        const uint32_t sel = (i & 1) ? 0x07060302u : 0x05040100u;
        bo[i] = u32x4{__builtin_amdgcn_perm(raw[1][q], raw[0][q], sel),
                      __builtin_amdgcn_perm(raw[3][q], raw[2][q], sel),
                      __builtin_amdgcn_perm(raw[5][q], raw[4][q], sel),
                      __builtin_amdgcn_perm(raw[7][q], raw[6][q], sel)};
      }
    } else {
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int row = wn * G2::WTN + 16 * i + lr;
        bo[i] = sb[row * 4 + (lg ^ swz4(row))];
      }
    }
#pragma unroll
    for (int f = 0; f < 8; ++f)
#pragma unroll
      for (int i = 0; i < 8; ++i)
        acc[f][i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, af[f]),
                                                            __builtin_bit_cast(bf16x8, bo[i]),
                                                            acc[f][i], 0, 0, 0);
  }
};

// C tile (m0, n0) accumulated over K tiles [kt0, kt1). A_band / B_band point at
// row m0 of A and at the tile's first column (BNC: element (0, n0); Bt: row n0).
template <bool BNC>
__device__ __forceinline__ void gemm2_mainloop(G2Smem& sm, f32x4 (&acc)[8][8], const Operand& A,
                                               const Operand& B, int M_rem, int N_rem, int K,
                                               int kt0, int kt1) {
  Pipe2<BNC> p;
  p.ra = make_rsrc(A);
  p.rb = make_rsrc(B);
  p.lda = A.ld;
  p.ldb = B.ld;
  p.M_rem = M_rem;
  p.N_rem = N_rem;
  p.K = K;
  const int n = kt1 - kt0;
  if (n <= 0) return;
#pragma unroll
  for (int i = 0; i < G2::NST - 1; ++i)
    if (i < n) p.issue(sm.s, i, kt0 + i);
  for (int i = 0; i < n; ++i) {
    // tile i's copies are complete once at most the copies of tiles i+1, i+2
    // (issued after it) are outstanding
    const int ahead = n - 1 - i;
    if (ahead >= 2)
      wait_vmcnt<2 * G2::LOADS_PER_STAGE>();
    else if (ahead == 1)
      wait_vmcnt<G2::LOADS_PER_STAGE>();
    else
      wait_vmcnt<0>();
    stage_barrier();
    if (i + G2::NST - 1 < n) p.issue(sm.s, (i + G2::NST - 1) % G2::NST, kt0 + i + G2::NST - 1);
    Pipe2<BNC>::compute(sm.s, i % G2::NST, acc);
  }
  __syncthreads();
}

// Output coordinates of acc[f][i][r] relative to the tile.
template <bool BNC>
struct AccMap2 {
  int row0, colb, lr;
  __device__ __forceinline__ AccMap2() {
    const int l = threadIdx.x & 63, w = threadIdx.x >> 6;
    lr = l & 15;
    row0 = (w >> 1) * G2::WTM + 4 * (l >> 4);
    colb = (w & 1) * G2::WTN;
  }
  __device__ __forceinline__ int row(int f, int r) const { return row0 + 16 * f + r; }
  __device__ __forceinline__ int col(int i) const {
    return BNC ? colb + 8 * lr + i : colb + 16 * i + lr;
  }
};

}  // namespace fpo
