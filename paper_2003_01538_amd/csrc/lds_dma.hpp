// Building blocks shared by the kernels that feed LDS with direct (LDS-DMA)
// buffer loads: buffer resources, the 128-byte-row XOR swizzle, and waits
// on the vector-memory counter that leave the other counters alone.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace fs {

typedef __attribute__((address_space(3))) void lds_void;
typedef unsigned int v4u __attribute__((ext_vector_type(4)));

constexpr int BK = 64;          // bf16 elements per K-tile row (128 bytes)
constexpr int ROW = 128;        // LDS bytes per tile row
constexpr uint32_t OOB = 0x80000000u;  // a buffer offset past every range: loads read 0, stores drop

// Physical 16-byte chunk of logical chunk c in row `row` is c ^ swz(row).
// An operand read serves 16 lanes (16 rows x 16 bytes) per cycle from 64
// four-byte banks; consecutive rows alternate between the two 128-byte bank
// halves, so the 16 rows need distinct chunks within each parity class.
__device__ __forceinline__ int swz(int row) { return (row & 7) ^ ((row >> 3) & 1); }

__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}

// floor(n / d) for 0 <= n < 2^22 from inv, the correctly rounded 1 / d:
// n + 0.5 is exact, the product carries a relative error below 2^-23, and
// (n + 0.5) / d lies at least 0.5 / d from an integer, so truncating the
// product gives the quotient exactly.
__device__ __forceinline__ int fdiv_small(int n, float inv) { return (int)(((float)n + 0.5f) * inv); }

// s_waitcnt vmcnt(n) leaving the other counters alone (gfx9 encoding)
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

// s_waitcnt lgkmcnt(0), leaving vmcnt and expcnt alone
__device__ __forceinline__ void wait_lgkm0() { __builtin_amdgcn_s_waitcnt(0xF | (0x3 << 14) | (0x7 << 4)); }

// N stores that write nothing (buffer offsets past every range), for steps
// that wait on a fixed vector-memory count.  Each goes to a different offset:
// identical stores to one address would be merged by the compiler, leaving
// fewer in flight than the count assumes and releasing the wait early.
template <int N>
__device__ __forceinline__ void dummy_stores(__amdgpu_buffer_rsrc_t r) {
#pragma unroll
  for (int u = 0; u < N; ++u) __builtin_amdgcn_raw_buffer_store_b128(v4u{0, 0, 0, 0}, r, OOB + 16u * u, 0, 0);
}

// Workgroup barrier without a memory fence (so it does not wait for vector
// memory operations); the compiler may not move memory accesses across it.
__device__ __forceinline__ void wg_barrier() {
  __asm__ __volatile__("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  __asm__ __volatile__("" ::: "memory");
}

}  // namespace fs
