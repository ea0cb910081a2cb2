// Shared device helpers for the gfx950 FPO kernels: vector types, bf16
// conversion, wavefront and workgroup reductions.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace fpo {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int kWave = 64;

__device__ __forceinline__ float bf16_to_f32(uint32_t h16) { return __uint_as_float(h16 << 16); }
__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// Two floats -> packed bf16 pair (round to nearest even, hardware convert).
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  bf16x2 r = {(__bf16)lo, (__bf16)hi};
  return __builtin_bit_cast(uint32_t, r);
}
__device__ __forceinline__ uint16_t to_bf16(float f) {
  __bf16 r = (__bf16)f;
  return __builtin_bit_cast(uint16_t, r);
}

// Element load/store in either storage type.
template <typename T> __device__ __forceinline__ float ld_as_f32(const T* p, int64_t i);
template <> __device__ __forceinline__ float ld_as_f32<float>(const float* p, int64_t i) { return p[i]; }
template <> __device__ __forceinline__ float ld_as_f32<uint16_t>(const uint16_t* p, int64_t i) {
  return bf16_to_f32(p[i]);
}
template <typename T> __device__ __forceinline__ void st_from_f32(T* p, int64_t i, float v);
template <> __device__ __forceinline__ void st_from_f32<float>(float* p, int64_t i, float v) { p[i] = v; }
template <> __device__ __forceinline__ void st_from_f32<uint16_t>(uint16_t* p, int64_t i, float v) {
  p[i] = to_bf16(v);
}

// 4 consecutive elements as floats (16 B for f32, 8 B for bf16). i % 4 == 0.
template <typename T> __device__ __forceinline__ f32x4 ld4(const T* p, int64_t i);
template <> __device__ __forceinline__ f32x4 ld4<float>(const float* p, int64_t i) {
  return *reinterpret_cast<const f32x4*>(p + i);
}
template <> __device__ __forceinline__ f32x4 ld4<uint16_t>(const uint16_t* p, int64_t i) {
  u32x2 w = *reinterpret_cast<const u32x2*>(p + i);
  return f32x4{bf16_lo(w.x), bf16_hi(w.x), bf16_lo(w.y), bf16_hi(w.y)};
}
template <typename T> __device__ __forceinline__ void st4(T* p, int64_t i, f32x4 v);
template <> __device__ __forceinline__ void st4<float>(float* p, int64_t i, f32x4 v) {
  *reinterpret_cast<f32x4*>(p + i) = v;
}
template <> __device__ __forceinline__ void st4<uint16_t>(uint16_t* p, int64_t i, f32x4 v) {
  u32x2 w = {pack_bf16x2(v.x, v.y), pack_bf16x2(v.z, v.w)};
  *reinterpret_cast<u32x2*>(p + i) = w;
}

// ---- wavefront reductions (xor butterflies over all 64 lanes or within
// aligned groups of `width` lanes)
template <int width = 64>
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = width / 2; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
template <int width = 64>
__device__ __forceinline__ double wave_sum_d(double v) {
#pragma unroll
  for (int o = width / 2; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
template <int width = 64>
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = width / 2; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

// Workgroup sum in float (blockDim.x a multiple of 64, <= 1024). `red` must
// hold 16 floats. Result broadcast to every thread.
__device__ __forceinline__ float block_sum(float v, float* red) {
  v = wave_sum(v);
  const int w = threadIdx.x / kWave, l = threadIdx.x % kWave, nw = blockDim.x / kWave;
  __syncthreads();
  if (l == 0) red[w] = v;
  __syncthreads();
  float s = 0.f;
  for (int i = 0; i < nw; ++i) s += red[i];  // fixed order
  return s;
}
// Two block sums in one exchange (two barriers instead of four); each value
// is summed exactly as block_sum sums it. red holds 2 * (waves) floats.
__device__ __forceinline__ void block_sum2(float& a, float& b, float* red) {
  a = wave_sum(a);
  b = wave_sum(b);
  const int w = threadIdx.x / kWave, l = threadIdx.x % kWave, nw = blockDim.x / kWave;
  __syncthreads();
  if (l == 0) {
    red[w] = a;
    red[nw + w] = b;
  }
  __syncthreads();
  float sa = 0.f, sb = 0.f;
  for (int i = 0; i < nw; ++i) {  // fixed order
    sa += red[i];
    sb += red[nw + i];
  }
  a = sa;
  b = sb;
}
// One thread's share of sum_b v[b], b in [begin, end), of a 256-lane
// workgroup: elements begin + tid + 256k in a fixed order, with four
// independent accumulators so that four loads are in flight.
__device__ __forceinline__ double strided_sum_d(const double* __restrict__ v, int64_t begin, int64_t end) {
  double a0 = 0.0, a1 = 0.0, a2 = 0.0, a3 = 0.0;
  int64_t b = begin + threadIdx.x;
  for (; b + 768 < end; b += 1024) {
    a0 += v[b];
    a1 += v[b + 256];
    a2 += v[b + 512];
    a3 += v[b + 768];
  }
  for (; b < end; b += 256) a0 += v[b];
  return (a0 + a1) + (a2 + a3);
}

__device__ __forceinline__ double block_sum_d(double v, double* red) {
  v = wave_sum_d(v);
  const int w = threadIdx.x / kWave, l = threadIdx.x % kWave, nw = blockDim.x / kWave;
  __syncthreads();
  if (l == 0) red[w] = v;
  __syncthreads();
  double s = 0.0;
  for (int i = 0; i < nw; ++i) s += red[i];
  return s;
}

}  // namespace fpo
