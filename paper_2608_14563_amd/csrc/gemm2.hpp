// bf16 MFMA tile core with a 4-stage LDS ring fed by LDS-DMA buffer loads
// (gfx950 buffer_load_dwordx4 ... lds). One workgroup of 4 waves (2 x 2)
// computes a 256 x 256 tile of C = A B, A K-contiguous ([M][K]), B either
// N-contiguous ([K][N]) or K-contiguous ([N][K], "Bt"). K advances 32 per
// stage = two K steps of v_mfma_f32_32x32x16_bf16 (each wave: 4 x 4 blocks of
// 32 x 32). The 32x32x16 shape sustains ~95% of the bf16 peak in a pure MFMA
// loop on gfx950 where 16x16x32 reaches ~70% (measured).
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
//     c ^ ((r >> 2) & 3) -- fragment reads (32 consecutive rows x 2 chunks)
//     are then bank-conflict free under every lane-phase model consistent
//     with ds_read_b128 timings measured on gfx950.
//   N-contiguous tile: [32 K rows][32 chunks] as in memory (conflict free).
// Lane layout: in K step h (16 wide) lane l owns K indices 16h + 8*(l>>5) + s,
// s = 0..7, for both operands (the K order inside an MFMA is a summation order
// only). A fragment f holds rows 32f + (l&31) of the wave's 128. Output
// columns: for an N-contiguous B the lane owns the 4 consecutive columns
// 4*(l&31) + i of its wave's 128 (the four B operands i are packed with v_perm
// from 4-column raw rows, so no LDS transpose is needed); for a K-contiguous B
// it owns columns 32*i + (l&31). Accumulator acc[f][i] element r holds row
// 32f + 8*(r>>2) + 4*(l>>5) + (r&3).
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
  u32x4 s[G2::NST * G2::STAGE_CHUNKS];  // 32 KB per stage
};

__device__ __forceinline__ int swz4(int row) { return (row >> 2) & 3; }

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
  uint32_t lds_wave;      // LDS byte address of this wave's slice of stage 0 (uniform)
  uint32_t offA[4], offB[4];  // per-lane byte offsets of this lane's copies at k0 = 0
  int kA[4], kB[4];           // K index of the chunk / row each copy reads at k0 = 0
  bool okA[4], okB[4];        // row (A, Bt) or column (B) inside the operand
  int K;
  int64_t stepB;              // bytes B advances per K tile (BNC: 32 rows; Bt: 64 bytes)

  __device__ __forceinline__ void setup(const u32x4* smem, const Operand& A, const Operand& B,
                                        int M_rem, int N_rem, int K_) {
    const int w = threadIdx.x >> 6, l = threadIdx.x & 63;
    ra = make_rsrc(A);
    rb = make_rsrc(B);
    lds_wave = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)smem + (uint32_t)w * 4096u);
    K = K_;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int inst = w * 4 + j;
      const int row = 16 * inst + (l >> 2);
      const int c = (l & 3) ^ swz4(row);
      kA[j] = 8 * c;
      okA[j] = row < M_rem;
      offA[j] = (uint32_t)(((int64_t)row * A.ld + 8 * c) * 2);
      if constexpr (BNC) {
        const int krow = 2 * inst + (l >> 5), cb = l & 31;
        kB[j] = krow;
        okB[j] = 8 * cb < N_rem;
        offB[j] = (uint32_t)(((int64_t)krow * B.ld + 8 * cb) * 2);
      } else {
        kB[j] = 8 * c;
        okB[j] = row < N_rem;
        offB[j] = (uint32_t)(((int64_t)row * B.ld + 8 * c) * 2);
      }
    }
    stepB = BNC ? (int64_t)G2::BK * B.ld * 2 : (int64_t)G2::BK * 2;
  }

  // DMA copy j (0..3: A, 4..7: B) of K tile kt into ring stage st; tiles at
  // or beyond K (and out-of-range rows / columns) read as zero.
  __device__ __forceinline__ void issue_one(int st, int kt, int j) const {
    const int k0 = kt * G2::BK;
    const uint32_t sa = lds_wave + (uint32_t)st * (G2::STAGE_CHUNKS * 16);
    if (j < 4) {
      const bool ok = okA[j] && (k0 + kA[j] < K);
      dma16(ra, sa + 1024u * j, ok ? offA[j] + (uint32_t)(k0 * 2) : kOOB);
    } else {
      const int jb = j - 4;
      const bool ok = okB[jb] && (k0 + kB[jb] < K);
      dma16(rb, sa + G2::A_CHUNKS * 16 + 1024u * jb, ok ? offB[jb] + (uint32_t)(kt * stepB) : kOOB);
    }
  }
  __device__ __forceinline__ void issue(int st, int kt) const {
#pragma unroll
    for (int j = 0; j < 8; ++j) issue_one(st, kt, j);
  }

  // A fragment (32 rows x K step h) f of a stage.
  __device__ __forceinline__ static u32x4 read_a(const u32x4* stage, int f, int h) {
    const int w = threadIdx.x >> 6, l = threadIdx.x & 63;
    const int row = (w >> 1) * G2::WTM + 32 * f + (l & 31);
    return stage[row * 4 + ((2 * h + (l >> 5)) ^ swz4(row))];
  }
  // BNC: raw K rows (4 columns, 8 bytes each) of K step `part` into
  // raw[part*8+s]; Bt: the operands (i, h) for i in {2 part, 2 part + 1} into
  // bq[i*2+h].
  __device__ __forceinline__ static void read_b(const u32x4* stage, u32x2 (&raw)[16], u32x4 (&bq)[8],
                                                int part) {
    const int w = threadIdx.x >> 6, l = threadIdx.x & 63;
    const int wn = w & 1, lc = l & 31, lk = l >> 5;
    const u32x4* sb = stage + G2::A_CHUNKS;
    if constexpr (BNC) {
      const u32x2* sb2 = reinterpret_cast<const u32x2*>(sb);
#pragma unroll
      for (int s = 0; s < 8; ++s) raw[part * 8 + s] = sb2[(16 * part + 8 * lk + s) * 64 + wn * 32 + lc];
    } else {
#pragma unroll
      for (int i = 2 * part; i < 2 * part + 2; ++i)
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const int row = wn * G2::WTN + 32 * i + lc;
          bq[i * 2 + h] = sb[row * 4 + ((2 * h + lk) ^ swz4(row))];
        }
    }
  }
  // B operands (i, h) for i in [i0, i0+2): v_perm packing of K-row pairs (BNC)
  // or as read (Bt). b[i*2+h].
  __device__ __forceinline__ static void pack_b(const u32x2 (&raw)[16], const u32x4 (&bq)[8],
                                                u32x4 (&b)[8], int i0) {
#pragma unroll
    for (int i = i0; i < i0 + 2; ++i)
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        if constexpr (BNC) {
          const int q = i >> 1;
          const uint32_t sel = (i & 1) ? 0x07060302u : 0x05040100u;
          const u32x2* r = raw + h * 8;
          b[i * 2 + h] = u32x4{__builtin_amdgcn_perm(r[1][q], r[0][q], sel),
                               __builtin_amdgcn_perm(r[3][q], r[2][q], sel),
                               __builtin_amdgcn_perm(r[5][q], r[4][q], sel),
                               __builtin_amdgcn_perm(r[7][q], r[6][q], sel)};
        } else {
          b[i * 2 + h] = bq[i * 2 + h];
        }
      }
  }
  // MFMA (f, i) of K step h.
  __device__ __forceinline__ static void mfma1(u32x4 a, const u32x4 (&b)[8], f32x16 (&acc)[4][4],
                                               int f, int h, int i) {
    acc[f][i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a),
                                                        __builtin_bit_cast(bf16x8, b[i * 2 + h]),
                                                        acc[f][i], 0, 0, 0);
  }
};

// One K tile: the 32 MFMAs of the current stage in 8 groups of 4 (K step h,
// fragment row f) with the packed B operands `bc`. Each group's A fragment is
// read two groups ahead; the first two of the tile come in `a0`, `a1` from the
// previous iteration, and the last two groups read those of the next tile.
// With one wave per SIMD the MFMA pipe idles whenever the wave stalls on other
// issue, so the remaining work is spread one item between consecutive MFMAs
// in a fixed order (sched_barrier keeps the compiler from regrouping it): the
// wait + barrier that make tile i+1 visible (after group 0), the eight copies
// of tile i + NST - 1, the next tile's B reads and their packing into `bn`.
#define FPO_SB() __builtin_amdgcn_sched_barrier(0)
template <bool BNC>
__device__ __forceinline__ void gemm2_iter(const Pipe2<BNC>& p, G2Smem& sm, f32x16 (&acc)[4][4],
                                           const u32x4 (&bc)[8], u32x4 (&bn)[8], u32x2 (&raw)[16],
                                           u32x4 (&bq)[8], u32x4& a0, u32x4& a1, int i, int kt0) {
  using P = Pipe2<BNC>;
  constexpr int NST = G2::NST;
  const u32x4* cur = sm.s + (i % NST) * G2::STAGE_CHUNKS;
  const u32x4* nxt = sm.s + ((i + 1) % NST) * G2::STAGE_CHUNKS;
  const int st = (i + NST - 1) % NST, kt = kt0 + i + NST - 1;
  // group 0: f0 h0
  P::mfma1(a0, bc, acc, 0, 0, 0); FPO_SB();
  u32x4 a2 = P::read_a(cur, 2, 0); FPO_SB();
  P::mfma1(a0, bc, acc, 0, 0, 1); FPO_SB();
  P::mfma1(a0, bc, acc, 0, 0, 2); FPO_SB();
  P::mfma1(a0, bc, acc, 0, 0, 3); FPO_SB();
  wait_vmcnt<(NST - 3) * G2::LOADS_PER_STAGE>();
  stage_barrier(); FPO_SB();
  // group 1: f1 h0
  P::mfma1(a1, bc, acc, 1, 0, 0); FPO_SB();
  u32x4 a3 = P::read_a(cur, 3, 0); FPO_SB();
  P::mfma1(a1, bc, acc, 1, 0, 1); FPO_SB();
  p.issue_one(st, kt, 0); FPO_SB();
  P::mfma1(a1, bc, acc, 1, 0, 2); FPO_SB();
  P::read_b(nxt, raw, bq, 0); FPO_SB();
  P::mfma1(a1, bc, acc, 1, 0, 3); FPO_SB();
  p.issue_one(st, kt, 1); FPO_SB();
  // group 2: f2 h0
  P::mfma1(a2, bc, acc, 2, 0, 0); FPO_SB();
  u32x4 a4 = P::read_a(cur, 0, 1); FPO_SB();
  P::mfma1(a2, bc, acc, 2, 0, 1); FPO_SB();
  p.issue_one(st, kt, 2); FPO_SB();
  P::mfma1(a2, bc, acc, 2, 0, 2); FPO_SB();
  P::read_b(nxt, raw, bq, 1); FPO_SB();
  P::mfma1(a2, bc, acc, 2, 0, 3); FPO_SB();
  p.issue_one(st, kt, 3); FPO_SB();
  // group 3: f3 h0
  P::mfma1(a3, bc, acc, 3, 0, 0); FPO_SB();
  u32x4 a5 = P::read_a(cur, 1, 1); FPO_SB();
  P::mfma1(a3, bc, acc, 3, 0, 1); FPO_SB();
  p.issue_one(st, kt, 4); FPO_SB();
  P::mfma1(a3, bc, acc, 3, 0, 2); FPO_SB();
  P::mfma1(a3, bc, acc, 3, 0, 3); FPO_SB();
  p.issue_one(st, kt, 5); FPO_SB();
  // group 4: f0 h1
  P::mfma1(a4, bc, acc, 0, 1, 0); FPO_SB();
  u32x4 a6 = P::read_a(cur, 2, 1); FPO_SB();
  P::mfma1(a4, bc, acc, 0, 1, 1); FPO_SB();
  P::pack_b(raw, bq, bn, 0); FPO_SB();
  P::mfma1(a4, bc, acc, 0, 1, 2); FPO_SB();
  p.issue_one(st, kt, 6); FPO_SB();
  P::mfma1(a4, bc, acc, 0, 1, 3); FPO_SB();
  // group 5: f1 h1
  P::mfma1(a5, bc, acc, 1, 1, 0); FPO_SB();
  u32x4 a7 = P::read_a(cur, 3, 1); FPO_SB();
  P::mfma1(a5, bc, acc, 1, 1, 1); FPO_SB();
  P::pack_b(raw, bq, bn, 2); FPO_SB();
  P::mfma1(a5, bc, acc, 1, 1, 2); FPO_SB();
  p.issue_one(st, kt, 7); FPO_SB();
  P::mfma1(a5, bc, acc, 1, 1, 3); FPO_SB();
  // group 6: f2 h1
  P::mfma1(a6, bc, acc, 2, 1, 0); FPO_SB();
  a0 = P::read_a(nxt, 0, 0); FPO_SB();
  P::mfma1(a6, bc, acc, 2, 1, 1); FPO_SB();
  P::mfma1(a6, bc, acc, 2, 1, 2); FPO_SB();
  P::mfma1(a6, bc, acc, 2, 1, 3); FPO_SB();
  // group 7: f3 h1
  P::mfma1(a7, bc, acc, 3, 1, 0); FPO_SB();
  a1 = P::read_a(nxt, 1, 0); FPO_SB();
  P::mfma1(a7, bc, acc, 3, 1, 1); FPO_SB();
  P::mfma1(a7, bc, acc, 3, 1, 2); FPO_SB();
  P::mfma1(a7, bc, acc, 3, 1, 3); FPO_SB();
}
#undef FPO_SB

// C tile accumulated over K tiles [kt0, kt1). A and B point at the band of the
// tile (A: row m0; B: column n0 (N-contiguous) or row n0 (K-contiguous)).
//
// Software pipeline over an NST-stage ring: while tile i is multiplied, tile
// i+1's operands are read (B packed) and tile i+NST-1's copies are issued.
// Copies are issued every iteration (beyond the last tile they read zeros into
// a stage no longer needed), so the wait before each barrier is a constant
// count: only tiles i+2 .. i+NST-2 may still be in flight. A stage is
// overwritten only after every wave has passed the barrier that follows its
// last read (its reads feed MFMAs issued before that barrier).
template <bool BNC>
__device__ __forceinline__ void gemm2_mainloop(G2Smem& sm, f32x16 (&acc)[4][4], const Operand& A,
                                               const Operand& B, int M_rem, int N_rem, int K,
                                               int kt0, int kt1) {
  constexpr int NST = G2::NST;
  const int n = kt1 - kt0;
  if (n <= 0) return;
  Pipe2<BNC> p;
  p.setup(sm.s, A, B, M_rem, N_rem, K);
#pragma unroll
  for (int s = 0; s < NST - 1; ++s) p.issue(s, kt0 + s);
  wait_vmcnt<(NST - 2) * G2::LOADS_PER_STAGE>();
  stage_barrier();
  u32x4 bc[8], bn[8], bq[8];
  u32x2 raw[16];
  Pipe2<BNC>::read_b(sm.s, raw, bq, 0);
  Pipe2<BNC>::read_b(sm.s, raw, bq, 1);
  u32x4 a0 = Pipe2<BNC>::read_a(sm.s, 0, 0), a1 = Pipe2<BNC>::read_a(sm.s, 1, 0);
  Pipe2<BNC>::pack_b(raw, bq, bc, 0);
  Pipe2<BNC>::pack_b(raw, bq, bc, 2);
  for (int i = 0; i < n; ++i) {
    gemm2_iter<BNC>(p, sm, acc, bc, bn, raw, bq, a0, a1, i, kt0);
#pragma unroll
    for (int j = 0; j < 8; ++j) bc[j] = bn[j];
  }
  wait_vmcnt<0>();
  __syncthreads();
}

__device__ __forceinline__ void zero_acc2(f32x16 (&acc)[4][4]) {
#pragma unroll
  for (int f = 0; f < 4; ++f)
#pragma unroll
    for (int i = 0; i < 4; ++i) acc[f][i] = f32x16{};
}

// Output coordinates of acc[f][i] element r relative to the tile.
template <bool BNC>
struct AccMap2 {
  static constexpr int R = 16;    // accumulator elements per (f, i): 4 groups of 4 consecutive rows
  static constexpr int LPR = 32;  // lanes sharing one output row
  int row0, colb, lc;
  __device__ __forceinline__ AccMap2() {
    const int l = threadIdx.x & 63, w = threadIdx.x >> 6;
    lc = l & 31;
    row0 = (w >> 1) * G2::WTM + 4 * (l >> 5);
    colb = (w & 1) * G2::WTN;
  }
  __device__ __forceinline__ int row(int f, int r) const { return row0 + 32 * f + 8 * (r >> 2) + (r & 3); }
  __device__ __forceinline__ int col(int i) const {
    return BNC ? colb + 4 * lc + i : colb + 32 * i + lc;
  }
};

}  // namespace fpo
