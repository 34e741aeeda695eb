// 3D nearest-neighbour tables for the local greedy (Sec. 3.5, Eq. 13).
//
// M_g(t) = the g tokens nearest to t, ordered by (distance, index), t itself
// included.  Distances compare as float64 squared distances formed from the
// float32 positions as (dx^2 + dy^2) + dz^2 without fused multiply-adds, so
// the order is reproducible bit for bit.  A nonnegative double's bit pattern
// orders like its value, so each distance is a 64-bit integer key.
//
// Exact brute force over all n tokens, in two kernels.
//  - knn_bound_kernel (g <= kBoundMaxG), kQ query tokens per block: every
//    thread keeps the smallest key it sees for each query; the g-th smallest
//    of those per-thread minima is an upper bound U on the g-th smallest key
//    (g distinct tokens lie at or below it).  A second pass collects the keys
//    <= U, which hold every member of M_g together with all keys tied with
//    the g-th, and ranks them by (key, index).  A row whose collection
//    overflows kCap is marked with -1 in its first entry.
//  - knn_radix_kernel, one row at a time per block with all n keys in LDS
//    (n <= kKnnLdsN; for larger n each pass recomputes the keys from the
//    positions, which stay in L2): an 8-bit radix select over the key's eight
//    bytes finds the g-th smallest key T and how many keys equal to T belong
//    to the answer; the tokens below T, and the first tokens equal to T in
//    index order, are collected and ranked.  It serves g > kBoundMaxG and the
//    rows the first kernel marked.
#include <hip/hip_runtime.h>

#include <algorithm>

#include "common.h"
#include "launch.h"

namespace cp {
namespace {

constexpr int kKnnMaxN = 32768;
constexpr int kKnnLdsN = 16384;   // up to here the radix select keeps n float64 keys (128 KiB) in LDS
constexpr int kKnnMaxG = 1024;
constexpr int kKnnBlock = 256;
constexpr int kKnnWaves = kKnnBlock / 64;
constexpr int kBoundMaxG = 128;         // <= kKnnBlock: the bound needs g per-thread minima; beyond
                                        // 128 it is loose enough that rows overflow kCap
constexpr int kQ = 8;                   // query tokens per block of the bounding kernel
constexpr int kCap = 256;               // collected keys per query
constexpr unsigned long long kNoKey = ~0ull;

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

__global__ __launch_bounds__(kKnnBlock) void knn_bound_kernel(const float* __restrict__ pos, int n, int g,
                                                              int32_t* __restrict__ out) {
  __shared__ unsigned long long smin[kQ][kKnnBlock];
  __shared__ unsigned long long ck[kQ][kCap];
  __shared__ int ci[kQ][kCap];
  __shared__ unsigned long long sU[kQ];
  __shared__ int scount[kQ];
  const int tid = threadIdx.x;
  const int q0 = blockIdx.x * kQ;
  const int nq = min(kQ, n - q0);
  float qx[kQ], qy[kQ], qz[kQ];
#pragma unroll
  for (int q = 0; q < kQ; ++q) {
    const int c = q0 + min(q, nq - 1);
    qx[q] = pos[3 * c];
    qy[q] = pos[3 * c + 1];
    qz[q] = pos[3 * c + 2];
  }

  // Pass 1: every thread's smallest key for each query.
  unsigned long long m[kQ];
#pragma unroll
  for (int q = 0; q < kQ; ++q) m[q] = kNoKey;
  for (int j = tid; j < n; j += kKnnBlock) {
    const float px = pos[3 * j], py = pos[3 * j + 1], pz = pos[3 * j + 2];
#pragma unroll
    for (int q = 0; q < kQ; ++q) {
      const unsigned long long k = sq_dist_key(qx[q], qy[q], qz[q], px, py, pz);
      m[q] = k < m[q] ? k : m[q];
    }
  }
#pragma unroll
  for (int q = 0; q < kQ; ++q) smin[q][tid] = m[q];
  if (tid < kQ) scount[tid] = 0;
  __syncthreads();

  // U_q = the g-th smallest per-thread minimum, by (value, thread).  Threads
  // that saw no token hold kNoKey; at least min(n, kKnnBlock) >= g did.
#pragma unroll
  for (int q = 0; q < kQ; ++q) {
    int rank = 0;
    for (int b = 0; b < kKnnBlock; ++b) {
      const unsigned long long x = smin[q][b];
      rank += x < m[q] || (x == m[q] && b < tid);
    }
    if (rank == g - 1) sU[q] = m[q];
  }
  __syncthreads();

  // Pass 2: every key <= U_q.
  unsigned long long U[kQ];
#pragma unroll
  for (int q = 0; q < kQ; ++q) U[q] = sU[q];
  for (int j = tid; j < n; j += kKnnBlock) {
    const float px = pos[3 * j], py = pos[3 * j + 1], pz = pos[3 * j + 2];
#pragma unroll
    for (int q = 0; q < kQ; ++q) {
      const unsigned long long k = sq_dist_key(qx[q], qy[q], qz[q], px, py, pz);
      if (k <= U[q]) {
        const int slot = atomicAdd(&scount[q], 1);
        if (slot < kCap) {
          ck[q][slot] = k;
          ci[q][slot] = j;
        }
      }
    }
  }
  __syncthreads();

  // Rank the collected keys; the first g by (key, index) form the row.
  for (int q = 0; q < nq; ++q) {
    const int mq = scount[q];
    int32_t* row = out + size_t(q0 + q) * g;
    if (mq > kCap) {
      if (tid == 0) row[0] = -1;
      continue;
    }
    for (int a = tid; a < mq; a += kKnnBlock) {
      const unsigned long long ka = ck[q][a];
      const int ia = ci[q][a];
      int rank = 0;
      for (int b = 0; b < mq; ++b) {
        const unsigned long long kb = ck[q][b];
        rank += kb < ka || (kb == ka && ci[q][b] < ia);
      }
      if (rank < g) row[rank] = ia;
    }
  }
}

// Row c by radix select; keys is the block's dynamic LDS: n keys (kLds
// only), then g collected keys and g indices.  Without kLds every read of a
// key recomputes it from the positions (the same float64 value).
template <bool kLds>
__device__ void knn_radix_row(const float* __restrict__ pos, int n, int g, int c, unsigned long long* keys,
                              int32_t* __restrict__ out) {
  unsigned long long* ckey = kLds ? keys + n : keys;
  int* cidx = reinterpret_cast<int*>(ckey + g);
  __shared__ unsigned int hist[256];
  __shared__ int swt[kKnnWaves];
  __shared__ unsigned long long s_prefix;
  __shared__ int s_rank;
  const int tid = threadIdx.x;
  const float qx = pos[3 * c], qy = pos[3 * c + 1], qz = pos[3 * c + 2];
  auto key = [&](int j) -> unsigned long long {
    return kLds ? keys[j] : sq_dist_key(qx, qy, qz, pos[3 * j], pos[3 * j + 1], pos[3 * j + 2]);
  };
  if (kLds)
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
      const unsigned long long k = key(j);
      if ((k & mask) == prefix) atomicAdd(&hist[(k >> shift) & 255u], 1u);
    }
    __syncthreads();
    // The bucket holding rank r: its exclusive prefix count is <= r and its
    // inclusive count exceeds r.
    const int r = s_rank;
    const int h = int(hist[tid]);
    int total;
    const int before = block_exclusive_scan(h, swt, total);
    if (before <= r && r < before + h) {
      s_rank = r - before;
      s_prefix = prefix | ((unsigned long long)tid << shift);
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
    const unsigned long long k = key(j);
    n_less += k < T;
    n_eq += k == T;
  }
  int less_total, eq_total;
  const int less_before = block_exclusive_scan(n_less, swt, less_total);
  const int eq_before = block_exclusive_scan(n_eq, swt, eq_total);
  (void)eq_total;
  int o_less = less_before, o_eq = eq_before;
  for (int j = j0; j < j1; ++j) {
    const unsigned long long k = key(j);
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
  __syncthreads();
}

// Rows handled by the radix select: every row (marked_only == 0) or the rows
// whose first entry the bounding kernel set to -1.  Block b takes rows
// b, b + gridDim.x, ...; it checks kKnnBlock of them at a time and selects the
// ones it must redo one after another.
template <bool kLds>
__global__ __launch_bounds__(kKnnBlock) void knn_radix_kernel(const float* __restrict__ pos, int n, int g,
                                                              int marked_only, int32_t* __restrict__ out) {
  extern __shared__ unsigned long long keys[];
  __shared__ int rows[kKnnBlock];
  __shared__ int nrows;
  const int tid = threadIdx.x;
  const int stride = gridDim.x;
  for (int base = blockIdx.x; base < n; base += stride * kKnnBlock) {
    if (tid == 0) nrows = 0;
    __syncthreads();
    const int c = base + stride * tid;
    if (c < n && (!marked_only || out[size_t(c) * g] == -1)) rows[atomicAdd(&nrows, 1)] = c;
    __syncthreads();
    const int cnt = nrows;
    for (int r = 0; r < cnt; ++r) knn_radix_row<kLds>(pos, n, g, rows[r], keys, out);
    __syncthreads();
  }
}

}  // namespace

static size_t knn_lds_bytes(int n, int g) { return (n <= kKnnLdsN ? size_t(n) * 8 : 0) + size_t(g) * 12; }

hipError_t launch_knn(const float* pos, int n, int g, int32_t* out, hipStream_t stream) {
  if (n < 1 || n > kKnnMaxN || g < 1 || g > n || g > kKnnMaxG) return hipErrorInvalidValue;
  hipError_t e;
  const bool bound = g <= kBoundMaxG;
  if (bound) {
    knn_bound_kernel<<<(n + kQ - 1) / kQ, kKnnBlock, 0, stream>>>(pos, n, g, out);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  const size_t lds = knn_lds_bytes(n, g);
  const bool in_lds = n <= kKnnLdsN;
  const void* radix = in_lds ? reinterpret_cast<const void*>(knn_radix_kernel<true>)
                             : reinterpret_cast<const void*>(knn_radix_kernel<false>);
  if ((e = hipFuncSetAttribute(radix, hipFuncAttributeMaxDynamicSharedMemorySize, int(lds))) != hipSuccess)
    return e;
  int dev = 0, cus = 0;
  if ((e = hipGetDevice(&dev)) != hipSuccess) return e;
  if ((e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev)) != hipSuccess) return e;
  const int grid = std::max(1, std::min(n, bound ? cus : 4 * cus));
  if (in_lds)
    knn_radix_kernel<true><<<grid, kKnnBlock, lds, stream>>>(pos, n, g, bound ? 1 : 0, out);
  else
    knn_radix_kernel<false><<<grid, kKnnBlock, lds, stream>>>(pos, n, g, bound ? 1 : 0, out);
  return hipGetLastError();
}

}  // namespace cp
