// Device helpers shared by the kernels of the decode library (gfx950, wave64).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

namespace dbt {

// bfloat16 storage: upper 16 bits of a float32.
__device__ __forceinline__ float bf2f(uint16_t x) { return __uint_as_float(((uint32_t)x) << 16); }

// float32 -> bfloat16, round to nearest even (finite inputs; NaN stays NaN).
__device__ __forceinline__ uint16_t f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

template <typename T> __device__ __forceinline__ float ld(const T *p, size_t i);
template <> __device__ __forceinline__ float ld<float>(const float *p, size_t i) { return p[i]; }
template <> __device__ __forceinline__ float ld<uint16_t>(const uint16_t *p, size_t i) { return bf2f(p[i]); }

template <typename T> __device__ __forceinline__ void st(T *p, size_t i, float v);
template <> __device__ __forceinline__ void st<float>(float *p, size_t i, float v) { p[i] = v; }
template <> __device__ __forceinline__ void st<uint16_t>(uint16_t *p, size_t i, float v) { p[i] = f2bf(v); }

constexpr float kLog2e = 1.4426950408889634f;

// Two floats to packed bf16 with the hardware conversion (round to nearest
// even, the same bits as f2bf for every non-NaN input).
__device__ __forceinline__ uint32_t pack2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, bf16x2{(__bf16)lo, (__bf16)hi});
}

// Maximum over lanes l, l^16, l^32 and l^48 (one column of a 16x16 MFMA
// result held by four 16-lane rows), with the row-swap permutes: no LDS
// round trip.
__device__ __forceinline__ float rows4_max(float x) {
  const auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
  const auto b = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}

// Buffer resource over `bytes` bytes at p (raw, unswizzled, 32-bit data
// format): a raw buffer load at an offset >= bytes returns zeros and reads no
// memory, so a resource of zero bytes turns a wave's loads into no-ops without
// a branch.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buf_rsrc(const void *p, int bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(p), (short)0, bytes, 0x00020000);
}
// 16 bytes at byte offset off, with the non-temporal hint (streamed data,
// read once).
__device__ __forceinline__ u32x4 buf_load_nt(__amdgpu_buffer_rsrc_t r, int off) {
  return __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 2));
}

// Orders a wave's LDS accesses around a hand-over between its own lanes
// (stores by some lanes, loads of that data by others): the hardware runs a
// wave's LDS operations in issue order, so only the compiler has to be kept
// from moving accesses across this point.
__device__ __forceinline__ void wave_lds_fence() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Zero the bf16 lanes of v (positions first .. first+7) at positions >= nvalid.
__device__ __forceinline__ u32x4 mask8(u32x4 v, int first, int nvalid) {
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    if (first + 2 * w >= nvalid) v[w] &= 0xffff0000u;
    if (first + 2 * w + 1 >= nvalid) v[w] &= 0x0000ffffu;
  }
  return v;
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

// Sum of S split-K partial slabs (stride apart) at idx, in split order.
__device__ __forceinline__ float psum(const float *part, long long stride, int S, size_t idx) {
  float s = 0.f;
#pragma unroll 4
  for (int k = 0; k < S; ++k) s += part[k * stride + idx];
  return s;
}

// RoPE of the pair (x0, x1) = (v_i, v_{i+d_h/2}) by the angle with (cos, sin)
// = cs, and the query coupling q2 + a * q1, written with explicit fused
// multiply-adds so that every kernel computing them rounds identically.
__device__ __forceinline__ float2 rope_pair(float x0, float x1, float2 cs) {
  return make_float2(fmaf(x0, cs.x, -(x1 * cs.y)), fmaf(x0, cs.y, x1 * cs.x));
}
__device__ __forceinline__ float couple(float a, float q1, float q2) { return fmaf(a, q1, q2); }

// Sum over a block of up to 1024 threads in a fixed order (deterministic).
// `red` must hold 16 floats; every thread gets the result.
__device__ __forceinline__ float block_sum(float v, float *red) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, nw = (blockDim.x + 63) >> 6;
  v = wave_sum(v);
  __syncthreads();
  if (lane == 0) red[w] = v;
  __syncthreads();
  float t = 0.f;
  for (int i = 0; i < nw; ++i) t += red[i];
  return t;
}
__device__ __forceinline__ float block_max(float v, float *red) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, nw = (blockDim.x + 63) >> 6;
  v = wave_max(v);
  __syncthreads();
  if (lane == 0) red[w] = v;
  __syncthreads();
  float t = -INFINITY;
  for (int i = 0; i < nw; ++i) t = fmaxf(t, red[i]);
  return t;
}

}  // namespace dbt
