// 3D nearest-neighbour tables for the local greedy (Sec. 3.5, Eq. 13).
//
// M_g(t) = the g tokens nearest to t, ordered by (distance, index), t itself
// included.  Distances compare as float64 squared distances formed from the
// float32 positions as (dx^2 + dy^2) + dz^2 without fused multiply-adds, so
// the order is reproducible bit for bit.  A nonnegative double's bit pattern
// orders like its value, so each distance is a 64-bit integer key.
//
// One block per query token (exact, brute force over all n tokens, n <=
// kKnnMaxN): the n keys go to LDS; an 8-bit radix select over the key's eight
// bytes finds the g-th smallest key T and how many keys equal to T belong to
// the answer; the tokens with key < T, and the first of those with key == T in
// index order, are collected and each is placed by counting the collected
// (key, index) pairs that precede it.
#include <hip/hip_runtime.h>

#include "common.h"
#include "launch.h"

namespace cp {
namespace {

constexpr int kKnnMaxN = 16384;   // n float64 keys fill 128 KiB of LDS
constexpr int kKnnMaxG = 1024;
constexpr int kKnnBlock = 256;
constexpr int kKnnWaves = kKnnBlock / 64;

__device__ __forceinline__ unsigned long long sq_dist_key(float ax, float ay, float az, float bx, float by, float bz) {
#pragma clang fp contract(off)
  const double dx = double(ax) - double(bx), dy = double(ay) - double(by), dz = double(az) - double(bz);
  return (unsigned long long)__double_as_longlong((dx * dx + dy * dy) + dz * dz);
}

// Exclusive prefix sum over the block (thread order) with the block total.
__device__ int block_exclusive_scan(int x, int* swt, int& total) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  int incl = x;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(incl, o);
    if (lane >= o) incl += y;
  }
  if (lane == 63) swt[w] = incl;
  __syncthreads();
  int before = 0;
  total = 0;
#pragma unroll
  for (int q = 0; q < kKnnWaves; ++q) {
    if (q < w) before += swt[q];
    total += swt[q];
  }
  __syncthreads();
  return before + incl - x;
}

__global__ __launch_bounds__(kKnnBlock) void knn_kernel(const float* __restrict__ pos, int n, int g,
                                                        int32_t* __restrict__ out) {
  extern __shared__ unsigned long long keys[];          // [n], then the collected pairs
  unsigned long long* ckey = keys + n;                  // [g]
  int* cidx = reinterpret_cast<int*>(ckey + g);         // [g]
  __shared__ unsigned int hist[256];
  __shared__ int swt[kKnnWaves];
  __shared__ unsigned long long s_prefix;
  __shared__ int s_rank;
  const int tid = threadIdx.x;
  const int c = blockIdx.x;
  const float qx = pos[3 * c], qy = pos[3 * c + 1], qz = pos[3 * c + 2];
  for (int j = tid; j < n; j += kKnnBlock)
    keys[j] = sq_dist_key(qx, qy, qz, pos[3 * j], pos[3 * j + 1], pos[3 * j + 2]);
  if (tid == 0) {
    s_prefix = 0ull;
    s_rank = g - 1;                                     // 0-based rank of the g-th smallest
  }
  __syncthreads();

  // Radix select, most significant byte first, over the keys that share the
  // bytes chosen so far.
  unsigned long long mask = 0ull;
  for (int shift = 56; shift >= 0; shift -= 8) {
    hist[tid] = 0u;
    __syncthreads();
    const unsigned long long prefix = s_prefix;
    for (int j = tid; j < n; j += kKnnBlock) {
      const unsigned long long k = keys[j];
      if ((k & mask) == prefix) atomicAdd(&hist[(k >> shift) & 255u], 1u);
    }
    __syncthreads();
    if (tid == 0) {
      int r = s_rank;
      int bucket = 0;
      while (bucket < 255 && r >= int(hist[bucket])) {
        r -= int(hist[bucket]);
        ++bucket;
      }
      s_rank = r;
      s_prefix = prefix | ((unsigned long long)bucket << shift);
    }
    mask |= 255ull << shift;
    __syncthreads();
  }
  const unsigned long long T = s_prefix;
  const int take_eq = s_rank + 1;                       // keys equal to T that belong to the answer

  // Collect in index order: thread tid scans the contiguous range of indices
  // [tid * span, (tid + 1) * span).
  const int span = (n + kKnnBlock - 1) / kKnnBlock;
  const int j0 = min(n, tid * span), j1 = min(n, j0 + span);
  int n_less = 0, n_eq = 0;
  for (int j = j0; j < j1; ++j) {
    const unsigned long long k = keys[j];
    n_less += k < T;
    n_eq += k == T;
  }
  int less_total, eq_total;
  const int less_before = block_exclusive_scan(n_less, swt, less_total);
  const int eq_before = block_exclusive_scan(n_eq, swt, eq_total);
  (void)eq_total;
  int o_less = less_before, o_eq = eq_before;
  for (int j = j0; j < j1; ++j) {
    const unsigned long long k = keys[j];
    if (k < T) {
      ckey[o_less] = k;
      cidx[o_less] = j;
      ++o_less;
    } else if (k == T) {
      if (o_eq < take_eq) {
        ckey[less_total + o_eq] = k;
        cidx[less_total + o_eq] = j;
      }
      ++o_eq;
    }
  }
  __syncthreads();

  // Place each collected pair by counting the pairs that precede it.
  for (int a = tid; a < g; a += kKnnBlock) {
    const unsigned long long ka = ckey[a];
    const int ia = cidx[a];
    int rank = 0;
    for (int b = 0; b < g; ++b) {
      const unsigned long long kb = ckey[b];
      rank += kb < ka || (kb == ka && cidx[b] < ia);
    }
    out[size_t(c) * g + rank] = ia;
  }
}

}  // namespace

static size_t knn_lds_bytes(int n, int g) { return size_t(n) * 8 + size_t(g) * 12; }

hipError_t launch_knn(const float* pos, int n, int g, int32_t* out, hipStream_t stream) {
  if (n < 1 || n > kKnnMaxN || g < 1 || g > n || g > kKnnMaxG) return hipErrorInvalidValue;
  const size_t lds = knn_lds_bytes(n, g);
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(knn_kernel),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, int(lds));
  if (e != hipSuccess) return e;
  knn_kernel<<<n, kKnnBlock, lds, stream>>>(pos, n, g, out);
  return hipGetLastError();
}

}  // namespace cp
