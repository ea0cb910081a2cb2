// bf16 MFMA tile core with a 2-stage LDS ring fed by LDS-DMA buffer loads
// (gfx950 buffer_load_dwordx4 ... lds). One workgroup of 4 waves (2 x 2)
// computes a 256 x 256 tile of C = A B, A K-contiguous ([M][K]), B either
// N-contiguous ([K][N]) or K-contiguous ([N][K], "Bt"). K advances 64 per
// stage = four K steps of v_mfma_f32_32x32x16_bf16 (each wave: 4 x 4 blocks of
// 32 x 32, i.e. 128 x 128).
//
// Why these shapes (measured on MI355X with random bf16 operands, where the
// chip runs at its power limit and the clock, not the issue rate, decides):
//  * in a pure MFMA loop over random operands 16x16x32 costs less power per
//    flop (~80% of the bf16 peak at ~1.95 GHz against ~71% at ~1.74 GHz for
//    32x32x16), but a 16x16x32 version of this core (same ring, tiles and
//    copies) turned the higher clock into no speed: its MFMA pipe sat idle
//    more of the time (twice the instructions to issue per flop from the one
//    wave each SIMD holds), so the core keeps the larger instruction;
//  * a 64-deep K stage makes every copy of a K-contiguous row a full 128-byte
//    line: at 32 deep each row gave a half line, twice the L2 requests for the
//    same bytes, and the extra request traffic cost ~25% of the clock.
//
// Pipeline (per K tile j in stage j % 2): the 16 copies of tile j+1 are issued
// from the end of iteration j-1 into the other stage, two between MFMA groups;
// one wait + barrier per tile (after MFMA group 13 of 16) makes tile j+1
// visible and releases stage j % 2; the last two groups then overlap the next
// tile's first operand reads. Out-of-range rows / K chunks are given a buffer
// offset beyond the resource and read as zero. Kernels instantiated with FAST
// (launched only when M and N are multiples of 256 and K of 64) copy with the
// lane's offset fixed in a register and the rest in the scalar offset, so a
// copy costs no vector instructions: the bounds selects of the general form
// were most of the core's non-MFMA vector issue.
//
// LDS layouts (16-byte chunks):
//   K-contiguous tile: [rows][8 chunks], chunk c of row r stored at position
//     c ^ swz8(r); swz8 takes row bits (2, 1, 3) -- fragment reads (32
//     consecutive rows x 2 chunks) are then bank-conflict free under every
//     lane-phase model consistent with ds_read_b128 timings measured on gfx950.
//   N-contiguous tile: [64 K rows][32 chunks] as in memory.
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
  static constexpr int BM = 256, BN = 256, BK = 64, NST = 2;
  static constexpr int WTM = 128, WTN = 128;
  static constexpr int A_CHUNKS = BM * 8;   // 32 KB
  static constexpr int B_CHUNKS = BN * 8;   // 32 KB
  static constexpr int STAGE_CHUNKS = A_CHUNKS + B_CHUNKS;
  static constexpr int LOADS_PER_STAGE = 16;  // DMA instructions per wave per stage
};

struct G2Smem {
  u32x4 s[G2::NST * G2::STAGE_CHUNKS];  // 64 KB per stage
};

__device__ __forceinline__ int swz8(int row) {
  return ((row >> 2) & 1) | (row & 2) | ((row >> 1) & 4);
}

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

// The same copy with a uniform byte offset in soffset: lane l reads
// rsrc + soffset + voff. The buffer range check covers voff only, so this form
// is used only where every lane's address is known to lie inside the operand.
__device__ __forceinline__ void dma16s(u32x4 rsrc, uint32_t lds_addr, uint32_t voff, uint32_t soff) {
  asm volatile(
      "s_mov_b32 m0, %0\n\t"
      "s_nop 0\n\t"
      "buffer_load_dwordx4 %1, %2, %3 offen lds"
      :
      : "s"(lds_addr), "v"(voff), "s"(rsrc), "s"(soff)
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
  uint32_t lds_wave;   // LDS byte address of stage 0 (uniform)
  int w, l;
  // K-contiguous copies: instruction q (0..7) of this wave covers rows
  // 8*(8w+q) .. +7; lane l reads row 8*(8w+q) + (l>>3), global chunk
  // (l&7) ^ swz8(row), which depends on q only through q & 1.
  uint32_t offA[2], offBt[2];  // byte offsets at q = 0 / 1, k = 0
  int kc[2];                   // K index of the lane's chunk for q & 1
  int rowA0;                   // row of the lane at q = 0
  int M_rem, N_rem, K;
  int64_t ldA2, ldB2;          // row strides in bytes
  // N-contiguous copies: instruction q covers K rows 2*(8w+q) + (l>>5),
  // columns 8*(l&31) .. +7.
  uint32_t offBn;
  bool okBn;
  int klast;                   // last K tile (fast form: later copies are clamped to it)

  __device__ __forceinline__ void setup(const u32x4* smem, const Operand& A, const Operand& B,
                                        int M_rem_, int N_rem_, int K_) {
    w = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));  // uniform: LDS addresses go to M0
    l = threadIdx.x & 63;
    ra = make_rsrc(A);
    rb = make_rsrc(B);
    lds_wave = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)smem);
    M_rem = M_rem_;
    N_rem = N_rem_;
    K = K_;
    ldA2 = A.ld * 2;
    ldB2 = B.ld * 2;
    rowA0 = 64 * w + (l >> 3);
#pragma unroll
    for (int p = 0; p < 2; ++p) {
      const int row = rowA0 + 8 * p;
      const int c = (l & 7) ^ swz8(row);
      kc[p] = 8 * c;
      offA[p] = (uint32_t)((int64_t)(l >> 3) * ldA2 + 16 * c);
      offBt[p] = (uint32_t)((int64_t)(l >> 3) * ldB2 + 16 * c);
    }
    offBn = (uint32_t)((int64_t)(l >> 5) * ldB2 + 16 * (l & 31));
    okBn = 8 * (l & 31) < N_rem;
    klast = (K + G2::BK - 1) / G2::BK - 1;
  }

  // Copy j of K tile kt in the fast form, for operands whose tiles are all
  // whole (M and N multiples of the tile, K of BK): the lane's offset is fixed,
  // the rest is uniform (soffset), so a copy needs no vector arithmetic and no
  // bounds selects. Every address lies inside the operand (copies issued past
  // the last K tile are clamped to it by the caller).
  __device__ __forceinline__ void issue_fast(int st, int kt, int j) const {
    const int k0 = kt * G2::BK;
    const uint32_t sbase = lds_wave + (uint32_t)st * (G2::STAGE_CHUNKS * 16);
    const int q = j & 7, inst = 8 * w + q;
    if (j < 8) {
      dma16s(ra, sbase + 1024u * inst, offA[q & 1], (uint32_t)((int64_t)8 * inst * ldA2 + k0 * 2));
    } else if constexpr (BNC) {
      dma16s(rb, sbase + G2::A_CHUNKS * 16 + 1024u * inst, offBn, (uint32_t)((int64_t)(k0 + 2 * inst) * ldB2));
    } else {
      dma16s(rb, sbase + G2::A_CHUNKS * 16 + 1024u * inst, offBt[q & 1],
             (uint32_t)((int64_t)8 * inst * ldB2 + k0 * 2));
    }
  }

  template <bool FAST>
  __device__ __forceinline__ void issue(int st, int kt, int j) const {
    if constexpr (FAST)
      issue_fast(st, kt, j);
    else
      issue_one(st, kt, j);
  }
  // K tile whose copies go out as tile kt (fast form: clamped to the last)
  template <bool FAST>
  __device__ __forceinline__ int copy_tile(int kt) const {
    return FAST ? min(kt, klast) : kt;
  }

  // DMA copy j (0..7: A, 8..15: B) of K tile kt into ring stage st; rows,
  // columns and K chunks out of range read as zero.
  __device__ __forceinline__ void issue_one(int st, int kt, int j) const {
    const int k0 = kt * G2::BK;
    const uint32_t sbase = lds_wave + (uint32_t)st * (G2::STAGE_CHUNKS * 16);
    const int q = j & 7, inst = 8 * w + q;
    if (j < 8) {
      const int row = rowA0 + 8 * q;
      const bool ok = row < M_rem && k0 + kc[q & 1] < K;
      const uint32_t off = offA[q & 1] + (uint32_t)((int64_t)8 * inst * ldA2) + (uint32_t)(k0 * 2);
      dma16(ra, sbase + 1024u * inst, ok ? off : kOOB);
    } else if constexpr (BNC) {
      const int krow = 2 * inst + (l >> 5);
      const bool ok = okBn && k0 + krow < K;
      const uint32_t off = offBn + (uint32_t)((int64_t)(k0 + 2 * inst) * ldB2);
      dma16(rb, sbase + G2::A_CHUNKS * 16 + 1024u * inst, ok ? off : kOOB);
    } else {
      const int row = rowA0 + 8 * q;
      const bool ok = row < N_rem && k0 + kc[q & 1] < K;
      const uint32_t off = offBt[q & 1] + (uint32_t)((int64_t)8 * inst * ldB2) + (uint32_t)(k0 * 2);
      dma16(rb, sbase + G2::A_CHUNKS * 16 + 1024u * inst, ok ? off : kOOB);
    }
  }

  // A fragment (32 rows, K step h) f of a stage.
  __device__ __forceinline__ u32x4 read_a(const u32x4* stage, int f, int h) const {
    const int row = (w >> 1) * G2::WTM + 32 * f + (l & 31);
    return stage[row * 8 + ((2 * h + (l >> 5)) ^ swz8(row))];
  }
  // B of K step h, half `part` (0/1). BNC: raw K rows 16h + 8*(l>>5) + s for
  // s in [4 part, 4 part + 4) (4 columns, 8 bytes each) into raw[s]; Bt: the
  // operands i in {2 part, 2 part + 1} into bq[i].
  __device__ __forceinline__ void read_b(const u32x4* stage, int h, int part, u32x2 (&raw)[8],
                                         u32x4 (&bq)[4]) const {
    const u32x4* sb = stage + G2::A_CHUNKS;
    const int wn = w & 1, lc = l & 31;
    if constexpr (BNC) {
      const u32x2* sb2 = reinterpret_cast<const u32x2*>(sb);
#pragma unroll
      for (int s = 4 * part; s < 4 * part + 4; ++s)
        raw[s] = sb2[(16 * h + 8 * (l >> 5) + s) * 64 + wn * 32 + lc];
    } else {
#pragma unroll
      for (int i = 2 * part; i < 2 * part + 2; ++i) {
        const int row = wn * G2::WTN + 32 * i + lc;
        bq[i] = sb[row * 8 + ((2 * h + (l >> 5)) ^ swz8(row))];
      }
    }
  }
  // B operands i in {2 part, 2 part + 1} of a K step: v_perm packing of K-row
  // pairs (BNC) or as read (Bt).
  __device__ __forceinline__ static void pack_b(const u32x2 (&raw)[8], const u32x4 (&bq)[4],
                                                u32x4 (&b)[4], int part) {
#pragma unroll
    for (int i = 2 * part; i < 2 * part + 2; ++i) {
      if constexpr (BNC) {
        const int q = i >> 1;
        const uint32_t sel = (i & 1) ? 0x07060302u : 0x05040100u;
        b[i] = u32x4{__builtin_amdgcn_perm(raw[1][q], raw[0][q], sel),
                     __builtin_amdgcn_perm(raw[3][q], raw[2][q], sel),
                     __builtin_amdgcn_perm(raw[5][q], raw[4][q], sel),
                     __builtin_amdgcn_perm(raw[7][q], raw[6][q], sel)};
      } else {
        b[i] = bq[i];
      }
    }
  }
};

#define FPO_SB() __builtin_amdgcn_sched_barrier(0)

// One MFMA group (fragment row f of K step with operands b): the four MFMAs
// with up to four items of other work placed one after each (sched_barrier
// keeps the order: with one wave per SIMD the MFMA pipe idles whenever the
// wave stalls on a burst of other issue).
template <class X0, class X1, class X2, class X3>
__device__ __forceinline__ void mfma_group(f32x16 (&acc)[4][4], int f, u32x4 a, const u32x4 (&b)[4],
                                           X0 x0, X1 x1, X2 x2, X3 x3) {
  acc[f][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a),
                                                      __builtin_bit_cast(bf16x8, b[0]), acc[f][0], 0, 0, 0);
  FPO_SB(); x0(); FPO_SB();
  acc[f][1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a),
                                                      __builtin_bit_cast(bf16x8, b[1]), acc[f][1], 0, 0, 0);
  FPO_SB(); x1(); FPO_SB();
  acc[f][2] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a),
                                                      __builtin_bit_cast(bf16x8, b[2]), acc[f][2], 0, 0, 0);
  FPO_SB(); x2(); FPO_SB();
  acc[f][3] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a),
                                                      __builtin_bit_cast(bf16x8, b[3]), acc[f][3], 0, 0, 0);
  FPO_SB(); x3(); FPO_SB();
}

// One K tile j (stage j % 2): 16 MFMA groups g = 4h + f. On entry `bc` holds
// the B operands of K step 0 and a[0], a[1] the A fragments of groups 0, 1.
// Tile j+1's copies 4..15 go out in groups 0..5 (0..3 went out at the end of
// the previous tile); the B operands of step h+1 are read in groups 4h, 4h+1
// and packed in 4h+2, 4h+3; A fragments are read two groups ahead (groups
// 14, 15 four ahead, so that all reads of the stage are complete at the
// barrier). After group 13: wait for tile j+1's copies, barrier. Groups 14, 15
// read tile j+1's first operands and issue tile j+2's copies 0..3 into the
// stage just released.
template <bool BNC, bool FAST>
__device__ __forceinline__ void gemm2_iter(const Pipe2<BNC>& p, G2Smem& sm, f32x16 (&acc)[4][4],
                                           u32x4 (&bc)[4], u32x4 (&a)[2], int j, int kt0) {
  const u32x4* cur = sm.s + (j & 1) * G2::STAGE_CHUNKS;
  const u32x4* nxt = sm.s + ((j + 1) & 1) * G2::STAGE_CHUNKS;
  const int s1 = (j + 1) & 1, t1 = p.template copy_tile<FAST>(kt0 + j + 1);  // tile j+1: copies 4..15 now
  const int s2 = j & 1, t2 = p.template copy_tile<FAST>(kt0 + j + 2);        // tile j+2: copies 0..3 after the barrier
  auto nop = [] {};
  u32x2 raw[8];
  u32x4 bq[4], bn[4];
  u32x4 a2, a3, a4, a5, a6, a7, a8, a9, a10, a11, a12, a13, a14, a15;
  // ---- K step 0
  mfma_group(acc, 0, a[0], bc, [&] { a2 = p.read_a(cur, 2, 0); }, [&] { p.template issue<FAST>(s1, t1, 4); },
             [&] { p.read_b(cur, 1, 0, raw, bq); }, [&] { p.template issue<FAST>(s1, t1, 5); });
  mfma_group(acc, 1, a[1], bc, [&] { a3 = p.read_a(cur, 3, 0); }, [&] { p.template issue<FAST>(s1, t1, 6); },
             [&] { p.read_b(cur, 1, 1, raw, bq); }, [&] { p.template issue<FAST>(s1, t1, 7); });
  mfma_group(acc, 2, a2, bc, [&] { a4 = p.read_a(cur, 0, 1); }, [&] { p.template issue<FAST>(s1, t1, 8); },
             [&] { Pipe2<BNC>::pack_b(raw, bq, bn, 0); }, [&] { p.template issue<FAST>(s1, t1, 9); });
  mfma_group(acc, 3, a3, bc, [&] { a5 = p.read_a(cur, 1, 1); }, [&] { p.template issue<FAST>(s1, t1, 10); },
             [&] { Pipe2<BNC>::pack_b(raw, bq, bn, 1); }, [&] { p.template issue<FAST>(s1, t1, 11); });
  // ---- K step 1
  mfma_group(acc, 0, a4, bn, [&] { a6 = p.read_a(cur, 2, 1); }, [&] { p.template issue<FAST>(s1, t1, 12); },
             [&] { p.read_b(cur, 2, 0, raw, bq); }, [&] { p.template issue<FAST>(s1, t1, 13); });
  mfma_group(acc, 1, a5, bn, [&] { a7 = p.read_a(cur, 3, 1); }, [&] { p.template issue<FAST>(s1, t1, 14); },
             [&] { p.read_b(cur, 2, 1, raw, bq); }, [&] { p.template issue<FAST>(s1, t1, 15); });
  mfma_group(acc, 2, a6, bn, [&] { a8 = p.read_a(cur, 0, 2); }, nop,
             [&] { Pipe2<BNC>::pack_b(raw, bq, bc, 0); }, nop);
  mfma_group(acc, 3, a7, bn, [&] { a9 = p.read_a(cur, 1, 2); }, nop,
             [&] { Pipe2<BNC>::pack_b(raw, bq, bc, 1); }, nop);
  // ---- K step 2 (operands in bc)
  mfma_group(acc, 0, a8, bc, [&] { a10 = p.read_a(cur, 2, 2); }, nop,
             [&] { p.read_b(cur, 3, 0, raw, bq); }, nop);
  mfma_group(acc, 1, a9, bc, [&] { a11 = p.read_a(cur, 3, 2); }, nop,
             [&] { p.read_b(cur, 3, 1, raw, bq); }, nop);
  mfma_group(acc, 2, a10, bc, [&] { a12 = p.read_a(cur, 0, 3); }, [&] { a14 = p.read_a(cur, 2, 3); },
             [&] { Pipe2<BNC>::pack_b(raw, bq, bn, 0); }, nop);
  mfma_group(acc, 3, a11, bc, [&] { a13 = p.read_a(cur, 1, 3); }, [&] { a15 = p.read_a(cur, 3, 3); },
             [&] { Pipe2<BNC>::pack_b(raw, bq, bn, 1); }, nop);
  // ---- K step 3 (operands in bn)
  mfma_group(acc, 0, a12, bn, nop, nop, nop, nop);
  mfma_group(acc, 1, a13, bn, nop, nop, nop, [&] {
    // every read of this stage is complete and tile j+1 has landed
    __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0)
    wait_vmcnt<0>();
    stage_barrier();
  });
  mfma_group(acc, 2, a14, bn, [&] { p.read_b(nxt, 0, 0, raw, bq); }, [&] { a[0] = p.read_a(nxt, 0, 0); },
             [&] { p.read_b(nxt, 0, 1, raw, bq); }, [&] { p.template issue<FAST>(s2, t2, 0); });
  mfma_group(acc, 3, a15, bn, [&] { a[1] = p.read_a(nxt, 1, 0); }, [&] { p.template issue<FAST>(s2, t2, 1); },
             [&] { p.template issue<FAST>(s2, t2, 2); }, [&] { p.template issue<FAST>(s2, t2, 3); });
  Pipe2<BNC>::pack_b(raw, bq, bc, 0);
  Pipe2<BNC>::pack_b(raw, bq, bc, 1);
}
#undef FPO_SB

// C tile accumulated over K tiles [kt0, kt1). A and B point at the band of the
// tile (A: row m0; B: column n0 (N-contiguous) or row n0 (K-contiguous)).
// Copies are issued for every iteration (beyond the last tile they read
// zeros, or the next split's data, into a stage no longer needed), so every
// wait is the same: vmcnt(0) at the barrier of each tile.
template <bool BNC, bool FAST = false>
__device__ __forceinline__ void gemm2_mainloop(G2Smem& sm, f32x16 (&acc)[4][4], const Operand& A,
                                               const Operand& B, int M_rem, int N_rem, int K,
                                               int kt0, int kt1) {
  const int n = kt1 - kt0;
  if (n <= 0) return;
  Pipe2<BNC> p;
  p.setup(sm.s, A, B, M_rem, N_rem, K);
#pragma unroll
  for (int q = 0; q < 16; ++q) p.template issue<FAST>(0, kt0, q);
  wait_vmcnt<0>();
  stage_barrier();
  const int kt1c = p.template copy_tile<FAST>(kt0 + 1);
#pragma unroll
  for (int q = 0; q < 4; ++q) p.template issue<FAST>(1, kt1c, q);
  u32x2 raw[8];
  u32x4 bq[4], bc[4], a[2];
  p.read_b(sm.s, 0, 0, raw, bq);
  p.read_b(sm.s, 0, 1, raw, bq);
  a[0] = p.read_a(sm.s, 0, 0);
  a[1] = p.read_a(sm.s, 1, 0);
  Pipe2<BNC>::pack_b(raw, bq, bc, 0);
  Pipe2<BNC>::pack_b(raw, bq, bc, 1);
  for (int j = 0; j < n; ++j) gemm2_iter<BNC, FAST>(p, sm, acc, bc, a, j, kt0);
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
