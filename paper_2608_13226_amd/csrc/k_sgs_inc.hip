// Greedy coverage selection, incremental form (Sec. 3.5, Eq. 14-16).
//
// Same greedy as the dense sweep: step l picks
//   t_l = argmax_{c not chosen} gain(c),  gain(c) = sum_j v_j max(0, b_j - C_tm[j][c])
// and then b_j <- min(b_j, C_tm[j][t_l]).  Only the targets whose best cost
// drops at step l (the set J_l: C_tm[j][t_l] < b_j) change any gain, by
//   v_j (max(0, b'_j - C_tm[j][c]) - max(0, b_j - C_tm[j][c])),
// so the gains are computed once in full (b = c0) and then kept up to date
// from the rows of J_l alone: about sum_l |J_l| rows of C_tm are read instead
// of K full matrices.  Every term v_j max(0, b_j - C) is formed as in the
// dense sweep (the difference in float32, the product exactly in float64) and
// then rounded down onto a fixed-point grid of 2^-S, S chosen per launch so
// that c0 sum(v) stays below 2^101; gains are sums of these integers in 128
// bits.  Integer sums do not depend on their order, so the running gains are
// bit-identical to gains summed afresh from the current b (a gain that has
// dropped to zero is exactly zero), the result does not depend on the grid,
// and equal gains go to the smaller index.
//
// One cooperative launch, one block per compute unit.  Block b owns the rows
// and the columns [b W, (b + 1) W): the best costs b_j and capacities of its
// rows and the running gains of its columns stay in LDS for the whole launch.
// Per step:
//   1. every block reads the step's winner, and tests its own rows against
//      the winner's column; the rows that improve are written, compacted, to
//      the block's slice of the change list (row, v, old b, new b);
//   2. grid barrier;
//   3. every block walks the whole change list (all slices, in block order)
//      and applies the changes to its columns' gains, reading each changed
//      row's segment over its columns (one coalesced 256-byte read per row and
//      64 columns); block 0 also folds the drop of the objective;
//   4. every block takes the exact argmax of its unchosen columns and folds it
//      into the next step's packed (gain, index) maximum; grid barrier.
// Cross-block data (change lists, counts, the packed maxima, the barrier
// counter) goes through device-scope atomic operations, coherent across the
// chip's L2 caches without fences.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <climits>

#include "common.h"
#include "launch.h"

namespace cp {
namespace {

constexpr int kBlock = 256;
constexpr int kWaves = kBlock / 64;
constexpr int kMaxBlocks = 256;    // at most one block per compute unit
constexpr int kBatch = 32;         // change-list entries a wave has in flight
constexpr int kInitRows = 16;      // rows a wave has in flight in the full pass
constexpr int kIndexBits = 20;     // packed key: [44-bit gain | 20-bit inverted index]
constexpr unsigned long long kIndexMask = (1ull << kIndexBits) - 1ull;

// Fixed-point value of a nonnegative term: floor(t 2^S) in 128 bits (t 2^S <
// 2^102, so the high part stays below 2^38).
__device__ __forceinline__ __int128 fx(double t, int S) {
  const double y = __builtin_ldexp(fmax(t, 0.0), S);
  const double hi = __builtin_floor(y * 0x1p-64);
  const double lo = __builtin_fma(-hi, 0x1p64, y);
  return ((__int128)(unsigned long long)hi << 64) + (__int128)(unsigned long long)lo;
}

__device__ __forceinline__ double fx_to_double(__int128 g, int S) {
  const double x = (double)(long long)(g >> 64) * 0x1p64 + (double)(unsigned long long)g;
  return __builtin_ldexp(x, -S);
}

struct IncDev {
  const float* C;
  const float* v;
  int n, k;
  float c0;
  int32_t* selected;
  double* step_gain;
  double* step_obj;
  int32_t* assign;
  unsigned long long* list;   // [blocks][W][2]: (row | v << 32), (old b | new b << 32)
  unsigned int* count;        // [blocks] entries in each slice
  unsigned long long* key;    // [k] packed step maxima
  unsigned int* bar;          // grid barrier counter
  int W;                      // rows and columns per block
};

struct Layout {
  size_t list, count, key, ctrl, total;
};

size_t a256(size_t x) { return (x + 255) / 256 * 256; }

int blocks_for(int64_t n, int cus) {
  return int(std::max<int64_t>(1, std::min<int64_t>(std::min(cus, kMaxBlocks), (n + 63) / 64)));
}

// Sized for the largest grid (kMaxBlocks blocks of W = ceil(n / blocks) rows).
Layout layout(int64_t n, int64_t k) {
  Layout L;
  size_t o = 0;
  L.list = o;  o += a256(size_t(n + kMaxBlocks) * 16);
  L.count = o; o += a256(size_t(kMaxBlocks) * 4);
  L.key = o;   o += a256(size_t(k) * 8);
  L.ctrl = o;  o += 256;
  L.total = o;
  return L;
}

__device__ __forceinline__ unsigned long long pack_key(double g, int idx) {
  const unsigned long long gb = (unsigned long long)__double_as_longlong(g) >> kIndexBits;
  return (gb << kIndexBits) | (kIndexMask - (unsigned long long)idx);
}

__global__ void sgs_inc_init_kernel(IncDev a, int blocks) {
  const int gt = blockIdx.x * blockDim.x + threadIdx.x, nt = gridDim.x * blockDim.x;
  for (int s = gt; s < a.k; s += nt) a.key[s] = 0ull;
  for (int s = gt; s < blocks; s += nt) a.count[s] = 0u;
  for (int j = gt; j < a.n; j += nt)
    if (a.assign) a.assign[j] = -1;
  if (gt == 0) *a.bar = 0u;
}

// Fixed-order block sum, result in every thread.
__device__ double block_sum_all(double x, double* sd) {
  x = wave_sum(x);
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  __syncthreads();
  if (lane == 0) sd[w] = x;
  __syncthreads();
  double s = 0.0;
#pragma unroll
  for (int q = 0; q < kWaves; ++q) s += sd[q];
  __syncthreads();
  return s;
}

// Inclusive prefix sum over the block (thread order), result in every thread.
__device__ int block_inclusive_scan(int x, int* swt) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(x, o);
    if (lane >= o) x += y;
  }
  if (lane == 63) swt[w] = x;
  __syncthreads();
#pragma unroll
  for (int q = 0; q < kWaves; ++q)
    if (q < w) x += swt[q];
  __syncthreads();
  return x;
}

// Exact argmax (ties to the smaller index) of the block's unchosen columns,
// folded into *key; the cross-block key compares the gains as doubles
// truncated to 44 bits.
__device__ void publish_argmax(const unsigned long long* sGlo, const long long* sGhi, const unsigned char* ssel,
                               int lo, int cnt, int S, unsigned long long* key, __int128* sg, int* si) {
  __int128 g = -1;
  int gi = INT_MAX;
  for (int i = threadIdx.x; i < cnt; i += kBlock)
    if (!ssel[i]) {
      const __int128 x = ((__int128)sGhi[i] << 64) | (__int128)sGlo[i];
      if (x > g || (x == g && lo + i < gi)) {
        g = x;
        gi = lo + i;
      }
    }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const unsigned long long olo = __shfl_xor((unsigned long long)g, o);
    const long long ohi = __shfl_xor((long long)(g >> 64), o);
    const int oi = __shfl_xor(gi, o);
    const __int128 og = ((__int128)ohi << 64) | (__int128)olo;
    if (og > g || (og == g && oi < gi)) {
      g = og;
      gi = oi;
    }
  }
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  if (lane == 0) {
    sg[w] = g;
    si[w] = gi;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int q = 1; q < kWaves; ++q)
      if (sg[q] > g || (sg[q] == g && si[q] < gi)) {
        g = sg[q];
        gi = si[q];
      }
    if (gi != INT_MAX)
      __hip_atomic_fetch_max(key, pack_key(fx_to_double(g, S), gi), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  __syncthreads();
}

__global__ __launch_bounds__(kBlock) void sgs_inc_kernel(IncDev a) {
  extern __shared__ unsigned long long smem[];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int nb = gridDim.x, blk = blockIdx.x;
  const int lo = blk * a.W;
  const int cnt = max(0, min(a.n, lo + a.W) - lo);
  unsigned long long* sGlo = smem;                                 // [W] running gains, low words
  long long* sGhi = reinterpret_cast<long long*>(sGlo + a.W);      // [W] high words
  float* sb = reinterpret_cast<float*>(sGhi + a.W);                // [W] best costs of own rows
  float* sv = sb + a.W;                                            // [W] capacities of own rows
  int* spre = reinterpret_cast<int*>(sv + a.W);                    // [nb + 1] list offsets
  unsigned char* ssel = reinterpret_cast<unsigned char*>(spre + nb + 1);   // [W] chosen columns
  __shared__ __int128 red[kBlock];
  __shared__ __int128 sg[kWaves];
  __shared__ double sd[kWaves];
  __shared__ int si[kWaves];
  __shared__ int swt[kWaves];
  __shared__ int s_t;

  for (int i = tid; i < cnt; i += kBlock) {
    sb[i] = a.c0;
    sv[i] = a.v[lo + i];
    ssel[i] = 0;
  }

  // Fixed-point scale, the same in every block (same sum, same order): every
  // partial gain is at most c0 sum(v) < 2^(101 - S).
  double vsum;
  {
    double x = 0.0;
    for (int j = tid; j < a.n; j += kBlock) x += double(a.v[j]);
    vsum = block_sum_all(x, sd);
  }
  const double M = double(a.c0) * vsum;
  int S = 0;
  if (M > 0.0) {
    int e = 0;
    (void)__builtin_frexp(M, &e);   // M < 2^e
    S = 101 - e;
  }

  // Step-0 gains of the own columns: every row at b = c0.  Wave w takes the
  // 16-row chunks w, w + 4, ...; the waves' sums are added in wave order.
  for (int cc = 0; cc < cnt; cc += 64) {
    const bool colok = cc + lane < cnt;
    const int col = lo + cc + lane;
    __int128 g = 0;
    for (int j0 = w * kInitRows; j0 < a.n; j0 += kWaves * kInitRows) {
      float x[kInitRows];
#pragma unroll
      for (int u = 0; u < kInitRows; ++u) {
        const int j = j0 + u;
        x[u] = (colok && j < a.n) ? __builtin_nontemporal_load(a.C + size_t(j) * a.n + col) : a.c0;
      }
#pragma unroll
      for (int u = 0; u < kInitRows; ++u) {
        const int j = j0 + u;
        const float vj = j < a.n ? a.v[j] : 0.f;
        g += fx(double(vj) * double(fmaxf(a.c0 - x[u], 0.f)), S);
      }
    }
    red[tid] = g;
    __syncthreads();
    if (tid < 64 && cc + tid < cnt) {
      __int128 s = 0;
#pragma unroll
      for (int q = 0; q < kWaves; ++q) s += red[q * 64 + tid];
      sGlo[cc + tid] = (unsigned long long)s;
      sGhi[cc + tid] = (long long)(s >> 64);
    }
    __syncthreads();
  }

  // Block 0 keeps the objective L = sum_j v_j b_j, starting from c0 sum v.
  double L = double(a.c0) * vsum;

  publish_argmax(sGlo, sGhi, ssel, lo, cnt, S, a.key, sg, si);
  unsigned int round = 0;
  grid_barrier(a.bar, ++round);

  for (int step = 0; step < a.k; ++step) {
    if (tid == 0) {
      const unsigned long long kk = __hip_atomic_load(a.key + step, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      // Some block always publishes while unchosen columns remain; the clamp
      // only keeps a broken key from addressing past the matrix.
      s_t = min(int(kIndexMask - (kk & kIndexMask)), a.n - 1);
    }
    __syncthreads();
    const int t = s_t;
    if (t >= lo && t < lo + cnt && tid == 0) {
      ssel[t - lo] = 1;
      a.selected[step] = t;
      if (a.step_gain) a.step_gain[step] = fx_to_double(((__int128)sGhi[t - lo] << 64) | (__int128)sGlo[t - lo], S);
    }

    // 1. Own rows that the pick improves, compacted into the block's slice.
    int base = 0;
    unsigned long long* mine = a.list + size_t(blk) * a.W * 2;
    for (int i0 = 0; i0 < cnt; i0 += kBlock) {
      const int i = i0 + tid;
      float cv = 0.f, bo = 0.f;
      bool hit = false;
      if (i < cnt) {
        cv = a.C[size_t(lo + i) * a.n + t];
        bo = sb[i];
        hit = cv < bo;
      }
      const unsigned long long m = __ballot(hit);
      const int rank = __popcll(m & ((1ull << lane) - 1ull));
      if (lane == 0) swt[w] = __popcll(m);
      __syncthreads();
      int off = base, tot = 0;
#pragma unroll
      for (int q = 0; q < kWaves; ++q) {
        if (q < w) off += swt[q];
        tot += swt[q];
      }
      if (hit) {
        const int slot = off + rank;
        put(mine + size_t(slot) * 2,
            (unsigned long long)(unsigned int)(lo + i) | ((unsigned long long)__float_as_uint(sv[i]) << 32));
        put(mine + size_t(slot) * 2 + 1,
            (unsigned long long)__float_as_uint(bo) | ((unsigned long long)__float_as_uint(cv) << 32));
        sb[i] = cv;
        if (a.assign) a.assign[lo + i] = t;
      }
      base += tot;
      __syncthreads();
    }
    if (tid == 0) put(a.count + blk, unsigned(base));
    grid_barrier(a.bar, ++round);

    // The last step's changes only feed the objective, kept by block 0.
    if (step + 1 == a.k && blk != 0) break;

    // 2. Offsets of every block's slice in the flattened change list.
    {
      const int c = tid < nb ? int(get(a.count + tid)) : 0;
      const int incl = block_inclusive_scan(c, swt);
      if (tid < nb) spre[tid + 1] = incl;
      if (tid == 0) spre[0] = 0;
      __syncthreads();
    }
    const int total = spre[nb];

    // 3. Apply the changes to the own columns' gains.  Lanes < kBatch locate
    // and fetch one entry each; the entries are then broadcast and every lane
    // reads its column of the entry's row.
    double dobj = 0.0;
    for (int cc = 0; cc < cnt; cc += 64) {
      const bool colok = cc + lane < cnt;
      const int col = lo + cc + lane;
      __int128 g = 0;
      for (int e0 = w * kBatch; e0 < total; e0 += kWaves * kBatch) {
        const int e = e0 + lane;
        unsigned long long h0 = 0ull, h1 = 0ull;
        if (lane < kBatch && e < total) {
          int s0 = 0, s1 = nb;   // spre[s0] <= e < spre[s1]
          while (s1 - s0 > 1) {
            const int mid = (s0 + s1) >> 1;
            if (spre[mid] <= e) s0 = mid;
            else s1 = mid;
          }
          const unsigned long long* src = a.list + (size_t(s0) * a.W + size_t(e - spre[s0])) * 2;
          h0 = get(src);
          h1 = get(src + 1);
        }
        const int m = min(kBatch, total - e0);
        float x[kBatch];
#pragma unroll
        for (int u = 0; u < kBatch; ++u) {
          const int j = int(__shfl(unsigned(h0 & 0xffffffffull), u));
          x[u] = (u < m && colok) ? a.C[size_t(j) * a.n + col] : 0.f;
        }
#pragma unroll
        for (int u = 0; u < kBatch; ++u) {
          if (u < m) {
            const double vj = double(__uint_as_float(__shfl(unsigned(h0 >> 32), u)));
            const float bo = __uint_as_float(__shfl(unsigned(h1 & 0xffffffffull), u));
            const float bn = __uint_as_float(__shfl(unsigned(h1 >> 32), u));
            g += fx(vj * double(fmaxf(bn - x[u], 0.f)), S) - fx(vj * double(fmaxf(bo - x[u], 0.f)), S);
          }
        }
        if (blk == 0 && cc == 0 && lane < kBatch && e < total) {
          const float vj = __uint_as_float(unsigned(h0 >> 32));
          const float bo = __uint_as_float(unsigned(h1 & 0xffffffffull));
          const float bn = __uint_as_float(unsigned(h1 >> 32));
          dobj = fma(double(vj), double(bo) - double(bn), dobj);
        }
      }
      red[tid] = g;
      __syncthreads();
      if (tid < 64 && cc + tid < cnt) {
        __int128 s = ((__int128)sGhi[cc + tid] << 64) | (__int128)sGlo[cc + tid];
#pragma unroll
        for (int q = 0; q < kWaves; ++q) s += red[q * 64 + tid];
        sGlo[cc + tid] = (unsigned long long)s;
        sGhi[cc + tid] = (long long)(s >> 64);
      }
      __syncthreads();
    }
    if (blk == 0) {
      L -= block_sum_all(dobj, sd);
      if (tid == 0 && a.step_obj) a.step_obj[step] = L;
    }

    // 4. Next step's winner.
    if (step + 1 < a.k) {
      publish_argmax(sGlo, sGhi, ssel, lo, cnt, S, a.key + step + 1, sg, si);
      grid_barrier(a.bar, ++round);
    }
  }
}

}  // namespace

size_t sgs_inc_workspace_bytes(int64_t n, int64_t k) { return layout(n, k).total; }

hipError_t launch_sgs_incremental(const SgsParams& p, hipStream_t stream) {
  int dev = 0, cus = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if ((e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev)) != hipSuccess) return e;
  const int nb = blocks_for(p.n, cus);
  const int W = (p.n + nb - 1) / nb;
  const size_t lds = size_t(W) * (16 + 4 + 4 + 1) + size_t(nb + 1) * 4 + 16;
  int per_cu = 0;
  if ((e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, reinterpret_cast<const void*>(sgs_inc_kernel),
                                                        kBlock, lds)) != hipSuccess)
    return e;
  if (per_cu < 1) return hipErrorCooperativeLaunchTooLarge;

  const Layout L = layout(p.n, p.k);
  char* w = static_cast<char*>(p.workspace);
  IncDev a;
  a.C = p.cost;
  a.v = p.capacity;
  a.n = p.n;
  a.k = p.k;
  a.c0 = p.c0;
  a.selected = p.selected;
  a.step_gain = p.step_gain;
  a.step_obj = p.step_objective;
  a.assign = p.assign;
  a.list = reinterpret_cast<unsigned long long*>(w + L.list);
  a.count = reinterpret_cast<unsigned int*>(w + L.count);
  a.key = reinterpret_cast<unsigned long long*>(w + L.key);
  a.bar = reinterpret_cast<unsigned int*>(w + L.ctrl);
  a.W = W;

  sgs_inc_init_kernel<<<std::min(1024, (std::max(p.n, p.k) + 255) / 256), 256, 0, stream>>>(a, nb);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  void* args[] = {&a};
  return hipLaunchCooperativeKernel(reinterpret_cast<const void*>(sgs_inc_kernel), dim3(nb), dim3(kBlock), args,
                                    lds, stream);
}

}  // namespace cp
