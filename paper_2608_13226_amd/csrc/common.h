// Device-side helpers shared by the CoverPrune kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <cstdlib>

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

// A 64-bit value moved between lanes by a DPP pattern (both halves).  Every
// lane of the wave must be active.
template <int CTRL>
__device__ __forceinline__ unsigned long long dpp_u64(unsigned long long x) {
  const unsigned a = __builtin_amdgcn_mov_dpp(unsigned(x), CTRL, 0xf, 0xf, false);
  const unsigned b = __builtin_amdgcn_mov_dpp(unsigned(x >> 32), CTRL, 0xf, 0xf, false);
  return ((unsigned long long)b << 32) | a;
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

// Bounded waits.  Every poll loop in the library reads the launch's abort
// flag after each 64th failed poll (a device-scope load costs a round trip
// through memory, so not after every one) and after every failed poll once
// `limit` polls have failed; past the limit the wait raises the flag itself.
// A wait that gives up makes its block leave the launch, every other block
// gives up at its next unmet wait, and a kernel after the launch marks the
// outputs (selected = -1).  kSpinLimit polls with a short sleep take about a
// second, far beyond any legitimate wait.
constexpr unsigned int kSpinLimit = 1u << 22;

__device__ __forceinline__ bool give_up(unsigned int spins, unsigned int limit, unsigned int* abort) {
  if ((spins & 63u) != 63u && spins < limit) return false;
  if (get(abort)) return true;
  if (spins >= limit) {
    put(abort, 1u);
    return true;
  }
  return false;
}

// Host side: the poll limit of the bounded waits and the abort flag's value
// at launch.  COVERPRUNE_TEST_ABORT=1 in the environment starts every launch
// with the flag raised and a zero limit, so that each wait gives up at its
// first failed poll: the failure path runs, and every kernel still exits
// normally (tests of that path; never set otherwise).
struct WaitPolicy {
  unsigned int limit;
  unsigned int preset;
};
inline WaitPolicy wait_policy() {
  const char* s = std::getenv("COVERPRUNE_TEST_ABORT");
  if (s && s[0] == '1' && s[1] == 0) return {0u, 1u};
  return {kSpinLimit, 0u};
}

// After a launch whose waits are bounded: every selected[] entry becomes -1
// when the launch gave up.  A kernel of its own, so that it runs after every
// block of the launch has finished and no block's late store of a pick can
// land after the mark.
namespace {
__global__ void mark_aborted_kernel(const unsigned int* abort, int32_t* selected, int k) {
  if (!*abort) return;
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < k; i += gridDim.x * blockDim.x) selected[i] = -1;
}
hipError_t launch_mark_aborted(const unsigned int* abort, int32_t* selected, int k, hipStream_t stream) {
  mark_aborted_kernel<<<(k + 255) / 256 < 64 ? (k + 255) / 256 : 64, 256, 0, stream>>>(abort, selected, k);
  return hipGetLastError();
}
}  // namespace

// Grid barrier for a cooperative launch: every block counts itself in and
// waits until all gridDim.x blocks have arrived `round` times.  `counter`
// must be zero at launch.  Only data written with put() (or device-scope
// atomics) before the barrier may be read with get() after it: every wave
// first waits until its own such writes are acknowledged, then the block's
// waves meet, and only then does the block count itself in.  Returns false,
// in every thread of the block, when the wait gave up (see give_up): the
// block must then leave.
__device__ __forceinline__ bool grid_barrier(unsigned int* counter, unsigned int round, unsigned int* abort,
                                             unsigned int limit, int* sflag) {
  __builtin_amdgcn_s_waitcnt(0x0F70);   // vmcnt(0): this wave's stores and atomics are done
  __syncthreads();
  if (threadIdx.x == 0) {
    __hip_atomic_fetch_add(counter, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const unsigned int target = round * gridDim.x;
    int ok = 1;
    for (unsigned int spins = 0; get(counter) < target; ++spins) {
      if (give_up(spins, limit, abort)) {
        ok = 0;
        break;
      }
      __builtin_amdgcn_s_sleep(1);
    }
    *sflag = ok;
  }
  __syncthreads();
  const bool ok = *sflag != 0;
  __syncthreads();
  return ok;
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
