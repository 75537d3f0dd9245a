// Device-side helpers: bf16 <-> fp32, vector types, wavefront reductions.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace fs {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef float floatx8 __attribute__((ext_vector_type(8)));
typedef float floatx2 __attribute__((ext_vector_type(2)));
typedef float floatx16 __attribute__((ext_vector_type(16)));

__device__ __forceinline__ float bf2f(uint16_t b) { return __uint_as_float(uint32_t(b) << 16); }

// Round-to-nearest-even fp32 -> bf16 (gfx950 converts in hardware).
__device__ __forceinline__ uint16_t f2bf(float f) {
  __bf16 h = (__bf16)f;
  return __builtin_bit_cast(uint16_t, h);
}

// 8 floats -> 8 packed bf16 (16 bytes).
__device__ __forceinline__ uint4 f8_to_bf8(const float* v) {
  floatx8 f = {v[0], v[1], v[2], v[3], v[4], v[5], v[6], v[7]};
  bf16x8 b = __builtin_convertvector(f, bf16x8);
  return __builtin_bit_cast(uint4, b);
}

__device__ __forceinline__ void bf8_to_f8(uint4 u, float* v) {
  v[0] = __uint_as_float(u.x << 16); v[1] = __uint_as_float(u.x & 0xffff0000u);
  v[2] = __uint_as_float(u.y << 16); v[3] = __uint_as_float(u.y & 0xffff0000u);
  v[4] = __uint_as_float(u.z << 16); v[5] = __uint_as_float(u.z & 0xffff0000u);
  v[6] = __uint_as_float(u.w << 16); v[7] = __uint_as_float(u.w & 0xffff0000u);
}

// Wavefront (64 lanes) reductions with cross-lane shuffles.
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// (value, index) max; ties resolve to the smaller index.
__device__ __forceinline__ void wave_argmax(float& v, int& i) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    float ov = __shfl_xor(v, o, 64);
    int oi = __shfl_xor(i, o, 64);
    if (ov > v || (ov == v && oi < i)) { v = ov; i = oi; }
  }
}

// Workgroups are dispatched round-robin over the 8 XCDs of the chip in
// workgroup-id order.  Remap a linear id so that consecutive logical tiles
// land on the same XCD (sharing its L2): XCD x gets a contiguous range.
__device__ __forceinline__ int xcd_remap(int id, int total) {
  constexpr int NX = 8;
  if (total < NX) return id;
  int q = total / NX, r = total % NX;
  int x = id % NX, pos = id / NX;
  int base = x < r ? x * (q + 1) : r * (q + 1) + (x - r) * q;
  return base + pos;
}

}  // namespace fs
