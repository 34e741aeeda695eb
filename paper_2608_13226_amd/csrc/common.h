// Device-side helpers shared by the CoverPrune kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace cp {

constexpr int kWave = 64;

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16;

// Raw bits of a bfloat16 widened exactly to float.
__device__ __forceinline__ float bf16_bits_to_float(uint32_t bits16) {
  return __uint_as_float(bits16 << 16);
}

__device__ __forceinline__ float wave_max(float x) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x = fmaxf(x, __shfl_xor(x, o));
  return x;
}

__device__ __forceinline__ double wave_max(double x) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x = fmax(x, __shfl_xor(x, o));
  return x;
}

__device__ __forceinline__ double wave_sum(double x) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o);
  return x;
}

__device__ __forceinline__ int wave_max(int x) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x = max(x, __shfl_xor(x, o));
  return x;
}

__device__ __forceinline__ int wave_min(int x) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x = min(x, __shfl_xor(x, o));
  return x;
}

// For x >= 0 the IEEE bit pattern orders like the value, so an unsigned
// integer atomicMax on the bits is an exact, order-independent float max.
__device__ __forceinline__ void atomic_max_nonneg(unsigned int* bits, float x) {
  atomicMax(bits, __float_as_uint(x));
}
__device__ __forceinline__ void atomic_max_nonneg(unsigned long long* bits, double x) {
  atomicMax(bits, (unsigned long long)__double_as_longlong(x));
}

// Total order on float bit patterns (negative values included) for min/max
// through unsigned integer atomics.
__device__ __forceinline__ unsigned int float_order_key(float x) {
  unsigned int u = __float_as_uint(x);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ float float_from_order_key(unsigned int k) {
  unsigned int u = (k & 0x80000000u) ? (k & 0x7fffffffu) : ~k;
  return __uint_as_float(u);
}

// Device-scope relaxed atomic loads and stores.  Data that one block writes
// and another block reads inside the same launch goes through these: they are
// coherent across the chip's per-XCD L2 caches without device-scope fences
// (each of which writes back a whole L2).  A block's stores are complete at
// the workgroup barrier that precedes its arrival at a counter.
__device__ __forceinline__ void put(unsigned int* p, unsigned int x) {
  __hip_atomic_store(p, x, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ unsigned int get(const unsigned int* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void put(int* p, int x) {
  __hip_atomic_store(p, x, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ int get(const int* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void put(unsigned long long* p, unsigned long long x) {
  __hip_atomic_store(p, x, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ unsigned long long get(const unsigned long long* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void put(double* p, double x) {
  put(reinterpret_cast<unsigned long long*>(p), (unsigned long long)__double_as_longlong(x));
}
__device__ __forceinline__ double get(const double* p) {
  return __longlong_as_double((long long)get(reinterpret_cast<const unsigned long long*>(p)));
}

// Grid barrier for a cooperative launch: every block counts itself in and
// waits until all gridDim.x blocks have arrived `round` times.  `counter`
// must be zero at launch.  Only data written with put() before the barrier
// may be read with get() after it.
__device__ __forceinline__ void grid_barrier(unsigned int* counter, unsigned int round) {
  __syncthreads();
  if (threadIdx.x == 0) {
    __hip_atomic_fetch_add(counter, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const unsigned int target = round * gridDim.x;
    while (get(counter) < target) __builtin_amdgcn_s_sleep(1);
  }
  __syncthreads();
}

// (gain, index) pair ordering used by every argmax: larger gain first, then
// smaller index.
__device__ __forceinline__ bool better(double g, int i, double bg, int bi) {
  return g > bg || (g == bg && i < bi);
}

__device__ __forceinline__ void wave_argmax(double& g, int& i) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    double og = __shfl_xor(g, o);
    int oi = __shfl_xor(i, o);
    if (better(og, oi, g, i)) { g = og; i = oi; }
  }
}

}  // namespace cp
