// CoverPrune-Lite (Sec. 4, Eq. 17-20) on one GPU.
//
//   front (seven ordinary launches; each hands its results to the next
//          through the workspace, so no block waits for another)
//     bbox     per-block partials of the per-axis minimum (the Morton origin)
//              and maximum (which bounds the key bits in use)
//     keys     q = floor((x - min) * 256 / h) in float64, clamped to 21 bits;
//              key = 3-way bit interleave; voxel = q >> 8.  The top 12 key
//              bits in use pick a bucket: counts and capacity sums per bucket
//              by atomics, and every token's place in its bucket
//     place    bucket starts; each block owns the whole buckets that start in
//              its range of positions (its span); every token goes straight
//              to its bucket
//     sort     each block sorts its span by (key, token): in registers (a
//              bitonic network on key and token packed into 64 bits) when it
//              fits, else by a stable LSD radix sort inside the block; then
//              the permutation, the voxels by position and, with V =
//              floor(v * 2^40) in exact integers and the mass before each
//              position, t(p) = min(K-1, K * mass / W) and the offset t(p) - p
//     groups   a prefix minimum of t(p) - p and the K - N + p floor give the
//              group of every position (the walk of Eq. 17 in scan form),
//              and the group starts
//     tiles    16-row tiles per group, their prefix, the group of every
//              tile and the list of big groups' tiles (work units below)
//   pairs    per 16-row tile of a group, the tile's rows against the whole
//            group on the matrix cores (16 x 16 tiles over D), d_f,
//            A(p) = sum_j v_j d_f over adjacent pairs, and the global M_f,
//            M_x, M_tau over those pairs: one wave per tile for groups of at
//            most two tiles, one block per tile (waves splitting the column
//            tiles) for larger groups
//   B(p)     sum_j v_j (lam_x phi(d_x / M_x) + lam_tau d_tau / M_tau), or
//            v_j c0 for a non-adjacent pair: every term of the group cost that
//            does not involve features (a wave per position, after the pairs)
//   select   cost(p) = (lam_f / M_f) A(p) + B(p); per-group argmin (Eq. 18)
//   total    fixed-order sum of the K prototype costs (Eq. 20 objective)
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cfloat>
#include <climits>

#include "common.h"
#include "launch.h"

namespace cp {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;
constexpr int kFrontBlocks = 64;
constexpr int kBins = 256;             // 8-bit digits of the radix sort of long spans
constexpr int kAxisBits = 21;
constexpr int kSubBits = 8;
constexpr int kTileRows = 16;
// Bucket pass of the sort: the top kBucketBits key bits in use pick one of
// kBuckets buckets; every block then sorts its span of whole buckets in LDS
// when no span holds more than kSortCap elements.
constexpr int kBucketBits = 12;
constexpr int kBuckets = 1 << kBucketBits;
constexpr int kPerThread = kBuckets / kThreads;
constexpr int kSortCap = 4096;
static_assert(kSortCap >= kBuckets && kBuckets % kThreads == 0, "bucket tables share LDS with the sort");

struct LiteDev {
  const void* feats;
  int n, d, k;
  const float* pos;
  const int32_t* frame;
  const float* v;
  float lam_f, lam_x, lam_t, kappa;
  double inv_log1p_kappa, grid_scale;
  int32_t* selected;
  int32_t* group;
  double* objective;
  double* token_cost;           // [n] or nullptr: each token's cost to its group (Eq. 18)
  // workspace
  unsigned long long* key[2];
  int* tok[2];
  unsigned long long* vox_pos;  // [n] packed voxel of each sorted position
  unsigned int* bbox_part;      // [G][6]: order keys of each front block's per-axis minima, then maxima
  unsigned int* within;         // [n] a token's place in its bucket
  int* span;                    // [G + 1]: the front blocks' spans of sorted positions
  unsigned long long* span_run; // [G]: capacity units before each span
  double* geom;                 // [4]: the Morton origin (3 axes) and the key bits in use
  unsigned int* bcnt;           // [kBuckets] elements per bucket
  unsigned long long* bval;     // [kBuckets] capacity units per bucket
  unsigned long long* bsum;     // [G]
  int* bmin;                    // [G]
  int* gid;                     // [n] group of each sorted position
  int* gstart;                  // [k + 1]
  int* rt_start;                // [k + 1] first 16-row tile of each group
  int* unit_group;              // [n / 16 + k] group of every 16-row tile
  int* big_unit;                // [n / 16 + k] tiles of groups of more than kSplitTiles tiles, in order
  unsigned long long* bsum2;    // [G]
  double* A;                    // [n]
  double* B;                    // [n]
  double* gcost;                // [k]
  unsigned int* ctrl;           // see kCtrl* offsets
  unsigned int* pmax;           // [kMaxSlots][kSlotWords]: maxima over evaluated pairs, see kSlot*
};

// ctrl words
constexpr int kCtrlW = 4;          // u64 (words 4, 5): all capacity units
constexpr int kCtrlTiles = 12;     // total number of 16-row tiles
constexpr int kCtrlBig = 13;       // tiles of groups of more than kSplitTiles tiles

// The maxima over evaluated pairs (M_f, M_x, M_tau) are raised by every pair
// block; block b raises those of slot b % kMaxSlots, each slot on a cache
// line of its own (one line for all of them serialized a thousand blocks),
// and the kernels that use them take the maximum over the slots.
constexpr int kMaxSlots = 32;
constexpr int kSlotWords = 32;      // 128 bytes
constexpr int kSlotMf = 0;          // float bits of max d_f
constexpr int kSlotMt = 1;          // max |d tau|
constexpr int kSlotMx2 = 2;         // u64 bits of max squared distance (words 2, 3)

struct Layout {
  size_t key0, key1, tok0, tok1, vox_pos, bbox_part, within, span, span_run, geom, bcnt, bval, bsum, bsum2, bmin,
      gid, gstart, rt_start, unit_group, big_unit, A, B, gcost, ctrl, pmax, total;
};

// Groups of more than this many 16-row tiles are split over a block's waves.
constexpr int kSplitTiles = 2;

size_t a256(size_t x) { return (x + 255) / 256 * 256; }

Layout layout(int64_t n, int64_t k) {
  Layout L;
  size_t o = 0;
  L.key0 = o;     o += a256(size_t(n) * 8);
  L.key1 = o;     o += a256(size_t(n) * 8);
  L.tok0 = o;     o += a256(size_t(n) * 4);
  L.tok1 = o;     o += a256(size_t(n) * 4);
  L.vox_pos = o;  o += a256(size_t(n) * 8);
  L.bbox_part = o; o += a256(size_t(kFrontBlocks) * 6 * 4);
  L.within = o;   o += a256(size_t(n) * 4);
  L.span = o;     o += a256(size_t(kFrontBlocks + 1) * 4);
  L.span_run = o; o += a256(size_t(kFrontBlocks) * 8);
  L.geom = o;     o += a256(4 * 8);
  L.bcnt = o;     o += a256(size_t(kBuckets) * 4);
  L.bval = o;     o += a256(size_t(kBuckets) * 8);
  L.bsum = o;     o += a256(size_t(kFrontBlocks) * 8);
  L.bsum2 = o;    o += a256(size_t(kFrontBlocks) * 8);
  L.bmin = o;     o += a256(size_t(kFrontBlocks) * 4);
  L.gid = o;      o += a256(size_t(n) * 4);
  L.gstart = o;   o += a256(size_t(k + 1) * 4);
  L.rt_start = o; o += a256(size_t(k + 1) * 4);
  L.unit_group = o; o += a256(size_t(n / kTileRows + k) * 4);
  L.big_unit = o; o += a256(size_t(n / kTileRows + k) * 4);
  L.A = o;        o += a256(size_t(n) * 8);
  L.B = o;        o += a256(size_t(n) * 8);
  L.gcost = o;    o += a256(size_t(k) * 8);
  L.ctrl = o;     o += 256;
  L.pmax = o;     o += a256(size_t(kMaxSlots) * kSlotWords * 4);
  L.total = o;
  return L;
}

__device__ __forceinline__ unsigned long long spread3(unsigned int x) {
  unsigned long long r = 0;
  for (int i = 0; i < kAxisBits; ++i) r |= (unsigned long long)((x >> i) & 1u) << (3 * i);
  return r;
}

// Voxel coordinates (q >> 8, at most 13 bits each) packed 21 bits apart.
__device__ __forceinline__ unsigned long long pack_vox(unsigned int x, unsigned int y, unsigned int z) {
  return (unsigned long long)x | ((unsigned long long)y << 21) | ((unsigned long long)z << 42);
}

__device__ __forceinline__ bool adjacent(unsigned long long a, unsigned long long b) {
  const int ax = int(a & 0x1fffff), ay = int((a >> 21) & 0x1fffff), az = int(a >> 42);
  const int bx = int(b & 0x1fffff), by = int((b >> 21) & 0x1fffff), bz = int(b >> 42);
  return abs(ax - bx) <= 1 && abs(ay - by) <= 1 && abs(az - bz) <= 1;
}

__device__ __forceinline__ double sq_dist(double ax, double ay, double az, double bx, double by,
                                          double bz) {
#pragma clang fp contract(off)
  const double dx = ax - bx, dy = ay - by, dz = az - bz;
  return (dx * dx + dy * dy) + dz * dz;
}

// floor(K * before / W), capped at K - 1, in exact 128-bit integer arithmetic.
// The float64 estimate before * kw (kw = K / W) carries a relative error of a
// few units in the last place on a value below K < 2^31, so it is off by less
// than 1e-5 and its floor by at most one: one exact correction each way
// gives the result.
__device__ __forceinline__ bool ge128(unsigned long long ah, unsigned long long al,
                                      unsigned long long bh, unsigned long long bl) {
  return ah > bh || (ah == bh && al >= bl);
}
__device__ __forceinline__ long long thresholds_crossed(unsigned long long K, unsigned long long before,
                                                       unsigned long long W, double kw) {
  const unsigned long long ph = __umul64hi(K, before), pl = K * before;
  double est = floor(double(before) * kw);
  est = fmin(fmax(est, 0.0), double(K - 1));
  unsigned long long tq = (unsigned long long)(unsigned int)est;
  if (tq > 0 && !ge128(ph, pl, __umul64hi(tq, W), tq * W)) --tq;
  if (tq + 1 < K && ge128(ph, pl, __umul64hi(tq + 1, W), (tq + 1) * W)) ++tq;
  return (long long)tq;
}

__device__ __forceinline__ unsigned long long capacity_units(float v) {
  return (unsigned long long)floor(double(v) * 1099511627776.0);   // v * 2^40
}

// Block scans over 256 threads.
__device__ unsigned long long block_excl_sum_u64(unsigned long long x, unsigned long long* sh,
                                                 unsigned long long& total) {
  const int t = threadIdx.x;
  sh[t] = x;
  __syncthreads();
  for (int o = 1; o < kThreads; o <<= 1) {
    const unsigned long long y = t >= o ? sh[t - o] : 0ull;
    __syncthreads();
    sh[t] += y;
    __syncthreads();
  }
  total = sh[kThreads - 1];
  const unsigned long long incl = sh[t];
  __syncthreads();
  return incl - x;
}

__device__ int block_incl_min(int x, int* sh) {
  const int t = threadIdx.x;
  sh[t] = x;
  __syncthreads();
  for (int o = 1; o < kThreads; o <<= 1) {
    const int y = t >= o ? sh[t - o] : INT_MAX;
    __syncthreads();
    sh[t] = min(sh[t], y);
    __syncthreads();
  }
  const int r = sh[t];
  __syncthreads();
  return r;
}

__device__ __forceinline__ int clamp_range(int x, int n) { return min(max(x, 0), n); }

// Sum of vals[0..G) and of vals[0..blk), read in parallel (one thread per
// block, G <= 256) and reduced in LDS.  Result valid in every thread.
__device__ void block_prefix_u64(const unsigned long long* vals, int G, int blk, unsigned long long* sh,
                                 unsigned long long& before, unsigned long long& total) {
  const int t = threadIdx.x;
  sh[t] = t < G ? get(vals + t) : 0ull;
  __syncthreads();
  if (t == 0) {
    unsigned long long b = 0ull, s = 0ull;
    for (int x = 0; x < G; ++x) {
      if (x < blk) b += sh[x];
      s += sh[x];
    }
    sh[kThreads] = b;
    sh[kThreads + 1] = s;
  }
  __syncthreads();
  before = sh[kThreads];
  total = sh[kThreads + 1];
  __syncthreads();
}

// Grid coordinate of one position component (Morton cell of 1 / 256 voxel).
__device__ __forceinline__ unsigned int grid_coord(float x, double org, double scale) {
  double g = floor((double(x) - org) * scale);
  g = fmin(fmax(g, 0.0), double((1 << kAxisBits) - 1));
  return (unsigned int)g;
}

__device__ __forceinline__ unsigned long long morton3(unsigned int x, unsigned int y, unsigned int z) {
  return spread3(x) | (spread3(y) << 1) | (spread3(z) << 2);
}

// Bucket of a key.  The bit-length bound makes the clamp a no-op for finite
// positions; a key above the bound (non-finite input) still lands in a
// bucket of the tables, so no slot leaves the key array.
__device__ __forceinline__ int bucket_of(unsigned long long key, int bshift) {
  return int(min(key >> bshift, (unsigned long long)(kBuckets - 1)));
}

// Sum over the block's threads, valid in every thread.
__device__ unsigned long long block_sum_u64(unsigned long long x, unsigned long long* sh) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o);
  if ((threadIdx.x & 63) == 0) sh[threadIdx.x >> 6] = x;
  __syncthreads();
  unsigned long long r = 0ull;
  for (int q = 0; q < kWaves; ++q) r += sh[q];
  __syncthreads();
  return r;
}

// Compare-exchange of x[r] and x[r ^ J] inside one thread, for the
// bitonic stage of block size k (element index t R + r).
template <int R, int J>
__device__ __forceinline__ void cx_in_thread(unsigned long long (&x)[R], int t, int k) {
#pragma unroll
  for (int r = 0; r < R; ++r)
    if ((r ^ J) > r) {
      const unsigned long long lo = x[r], hi = x[r ^ J];
      const bool up = ((t * R + r) & k) == 0;
      const bool sw = (lo > hi) == up;
      x[r] = sw ? hi : lo;
      x[r ^ J] = sw ? lo : hi;
    }
}

// The value of lane (lane ^ M) of the wave, M in {1, 2, 4, 8, 16, 32}; every
// lane must be active.  Quad permutations give 1 and 2; a lane mirror within
// 8 (or 16) after a quad reversal (or an 8-mirror) gives 4 (or 8); a swizzle
// within 32 lanes gives 16, a permute 32.
template <int M>
__device__ __forceinline__ unsigned long long lane_xor_u64(unsigned long long x) {
  if constexpr (M == 1) return dpp_u64<0xB1>(x);                   // quad [1, 0, 3, 2]
  else if constexpr (M == 2) return dpp_u64<0x4E>(x);              // quad [2, 3, 0, 1]
  else if constexpr (M == 4) return dpp_u64<0x141>(dpp_u64<0x1B>(x));   // half-row mirror of quad [3, 2, 1, 0]
  else if constexpr (M == 8) return dpp_u64<0x140>(dpp_u64<0x141>(x));  // row mirror of half-row mirror
  else if constexpr (M == 16) {
    constexpr int kXor16 = 0x1f | (0x10 << 10);   // bit-mask swizzle: and 31, xor 16
    const unsigned lo = unsigned(__builtin_amdgcn_ds_swizzle(int(unsigned(x)), kXor16));
    const unsigned hi = unsigned(__builtin_amdgcn_ds_swizzle(int(unsigned(x >> 32)), kXor16));
    return ((unsigned long long)hi << 32) | lo;
  } else {
    static_assert(M == 32, "lane distance");
    return __shfl_xor(x, 32);
  }
}

// One bitonic stage whose partner of element t R + r is (t ^ M) R + r, a lane
// M away in the same wave.
template <int R, int M>
__device__ __forceinline__ void cx_lanes(unsigned long long (&x)[R], bool keep_min) {
  unsigned long long y[R];
#pragma unroll
  for (int r = 0; r < R; ++r) y[r] = lane_xor_u64<M>(x[r]);
#pragma unroll
  for (int r = 0; r < R; ++r) x[r] = keep_min ? min(x[r], y[r]) : max(x[r], y[r]);
}

// Ascending bitonic sort of the block's kThreads * R values, thread t
// holding elements t R .. t R + R - 1 in x.  Stages whose partner is in the
// same thread run in registers, those whose partner is in the same wave by
// lane exchanges; for the rest (partner in another wave) every thread stores
// its R values to LDS and reads its partner's, alternating between two
// buffers (lds0, lds1: kThreads * R values each) so that one barrier per
// stage suffices.  Value r of thread t sits at r kThreads + t, so that a
// wave's 8-byte accesses fall on consecutive banks.  On return thread t holds
// the sorted elements t R .. t R + R - 1.
template <int R>
__device__ void bitonic_regs(unsigned long long (&x)[R], unsigned long long* lds0, unsigned long long* lds1) {
  const int t = threadIdx.x;
  constexpr int P = kThreads * R;
  int flip = 0;
  for (int k = 2; k <= P; k <<= 1)
    for (int j = k >> 1; j > 0; j >>= 1) {
      if (j < R) {
        if constexpr (R > 1) if (j == 1) cx_in_thread<R, 1>(x, t, k);
        if constexpr (R > 2) if (j == 2) cx_in_thread<R, 2>(x, t, k);
        if constexpr (R > 4) if (j == 4) cx_in_thread<R, 4>(x, t, k);
        if constexpr (R > 8) if (j == 8) cx_in_thread<R, 8>(x, t, k);
        continue;
      }
      const int tj = j / R;                          // partner thread t ^ tj
      const bool keep_min = ((t & tj) == 0) == (((t * R) & k) == 0);
      switch (tj) {
        case 1: cx_lanes<R, 1>(x, keep_min); continue;
        case 2: cx_lanes<R, 2>(x, keep_min); continue;
        case 4: cx_lanes<R, 4>(x, keep_min); continue;
        case 8: cx_lanes<R, 8>(x, keep_min); continue;
        case 16: cx_lanes<R, 16>(x, keep_min); continue;
        case 32: cx_lanes<R, 32>(x, keep_min); continue;
        default: break;
      }
      unsigned long long* buf = flip ? lds1 : lds0;
      flip ^= 1;
#pragma unroll
      for (int r = 0; r < R; ++r) buf[r * kThreads + t] = x[r];
      __syncthreads();
      unsigned long long y[R];
#pragma unroll
      for (int r = 0; r < R; ++r) y[r] = buf[r * kThreads + (t ^ tj)];
#pragma unroll
      for (int r = 0; r < R; ++r) x[r] = keep_min ? min(x[r], y[r]) : max(x[r], y[r]);
    }
}

// The same network with every stage's sizes known at compile time (no loop
// or branch between stages), for R <= 8; the loop above serves R = 16.
template <int R, int K, int J>
__device__ __forceinline__ void bitonic_stage(unsigned long long (&x)[R], unsigned long long* lds0,
                                              unsigned long long* lds1, int& flip) {
  const int t = threadIdx.x;
  if constexpr (J < R) {
    cx_in_thread<R, J>(x, t, K);
  } else {
    constexpr int TJ = J / R;
    const bool keep_min = ((t & TJ) == 0) == (((t * R) & K) == 0);
    if constexpr (TJ < 64) {
      cx_lanes<R, TJ>(x, keep_min);
    } else {
      unsigned long long* buf = flip ? lds1 : lds0;
      flip ^= 1;
#pragma unroll
      for (int r = 0; r < R; ++r) buf[r * kThreads + t] = x[r];
      __syncthreads();
      unsigned long long y[R];
#pragma unroll
      for (int r = 0; r < R; ++r) y[r] = buf[r * kThreads + (t ^ TJ)];
#pragma unroll
      for (int r = 0; r < R; ++r) x[r] = keep_min ? min(x[r], y[r]) : max(x[r], y[r]);
    }
  }
  if constexpr (J > 1) bitonic_stage<R, K, J / 2>(x, lds0, lds1, flip);
}

template <int R, int K>
__device__ __forceinline__ void bitonic_merges(unsigned long long (&x)[R], unsigned long long* lds0,
                                               unsigned long long* lds1, int& flip) {
  bitonic_stage<R, K, K / 2>(x, lds0, lds1, flip);
  if constexpr (K < kThreads * R) bitonic_merges<R, 2 * K>(x, lds0, lds1, flip);
}

template <int R>
__device__ void bitonic_unrolled(unsigned long long (&x)[R], unsigned long long* lds0, unsigned long long* lds1) {
  int flip = 0;
  bitonic_merges<R, 2>(x, lds0, lds1, flip);
}

// After the span sort (s_sorted: the span's packed (key, token) values in
// order, m >= 1 of them): thread t's positions i in [i0, i1) of the span, at
// most R of them.  Writes the permutation and the voxels by position, scans
// the capacity units over the span (run: units before it, W: all units) and
// writes tp - p of each position to gid (Eq. 17 in scan form).  Work on
// absent positions reads position m - 1 and is dropped, so that the R
// positions' loads and arithmetic overlap.  Returns the thread's minimum
// tp - p (INT_MAX without positions).
template <int R>
__device__ int span_offsets(const LiteDev& a, int r0, int m, int i0, int i1, unsigned long long tmask,
                            const double (&org)[3], unsigned long long run, unsigned long long W,
                            const unsigned long long* s_sorted, unsigned long long* s_u64) {
  int tk[R];
  unsigned long long vx[R], V[R];
#pragma unroll
  for (int u = 0; u < R; ++u) {
    tk[u] = int(s_sorted[min(i0 + u, m - 1)] & tmask);
    vx[u] = pack_vox(grid_coord(a.pos[3 * tk[u]], org[0], a.grid_scale) >> kSubBits,
                     grid_coord(a.pos[3 * tk[u] + 1], org[1], a.grid_scale) >> kSubBits,
                     grid_coord(a.pos[3 * tk[u] + 2], org[2], a.grid_scale) >> kSubBits);
    V[u] = capacity_units(a.v[tk[u]]);
  }
  unsigned long long loc = 0ull;
#pragma unroll
  for (int u = 0; u < R; ++u)
    if (i0 + u < i1) {
      loc += V[u];
      a.tok[1][r0 + i0 + u] = tk[u];
      a.vox_pos[r0 + i0 + u] = vx[u];
    }
  unsigned long long span_tot;
  unsigned long long before = run + block_excl_sum_u64(loc, s_u64, span_tot);
  const double kw = W ? double(a.k) / double(W) : 0.0;
  long long tp[R];
#pragma unroll
  for (int u = 0; u < R; ++u) {
    const int pos = r0 + i0 + u;
    tp[u] = pos == 0 ? 0 : (W == 0ull ? a.k - 1 : thresholds_crossed((unsigned long long)a.k, before, W, kw));
    before += V[u];
  }
  int bmin = INT_MAX;
#pragma unroll
  for (int u = 0; u < R; ++u)
    if (i0 + u < i1) {
      const int mm = int(tp[u] - (r0 + i0 + u));
      a.gid[r0 + i0 + u] = mm;
      bmin = min(bmin, mm);
    }
  return bmin;
}

// Packs keys[0, m) and toks[0, m) as key * 2^tokbits + token (m <= kThreads
// * R; the rest padded with the largest value), sorts them and leaves the
// sorted values in dst[0, kThreads * R) (tmp: LDS of the same size,
// clobbered).
template <int R>
__device__ void span_sort(const unsigned long long* keys, const int* toks, int tokbits, int m,
                          unsigned long long* dst, unsigned long long* tmp) {
  const int t = threadIdx.x;
  unsigned long long x[R];
  // Every load is issued before any is used: indices past m read element
  // m - 1 and are then replaced by the padding.
  if (m > 0) {
#pragma unroll
    for (int r = 0; r < R; ++r) {
      const int i = min(t * R + r, m - 1);
      x[r] = (keys[i] << tokbits) | (unsigned long long)(unsigned int)toks[i];
    }
#pragma unroll
    for (int r = 0; r < R; ++r)
      if (t * R + r >= m) x[r] = ~0ull;
  } else {
#pragma unroll
    for (int r = 0; r < R; ++r) x[r] = ~0ull;
  }
  if constexpr (R <= 8) bitonic_unrolled<R>(x, dst, tmp);
  else bitonic_regs<R>(x, dst, tmp);
  __syncthreads();
#pragma unroll
  for (int r = 0; r < R; ++r) dst[t * R + r] = x[r];
  __syncthreads();
}

// ---------------------------------------------------------------------------
// The front: seven ordinary launches of G blocks.  Each hands its results to
// the next through the workspace (the launch boundary orders them), so no
// block ever waits for another.  Block b owns positions [b tile, (b + 1)
// tile) up to the placement and its span of whole buckets from the sort on.
struct FrontRange {
  int tile, p0, p1;
};
__device__ __forceinline__ FrontRange front_range(int n) {
  const int tile = (n + int(gridDim.x) - 1) / int(gridDim.x);
  const int p0 = min(n, int(blockIdx.x) * tile);
  return {tile, p0, min(n, p0 + tile)};
}

// The key geometry of the scene from the bbox: the Morton origin and the
// bit length of every key (the Morton code of the grid coordinates of the
// bbox maximum bounds it).
__device__ __forceinline__ int tok_bits(int n) { return n > 1 ? 32 - __clz(n - 1) : 0; }
__device__ __forceinline__ int bucket_shift(int kbits) { return kbits - min(kBucketBits, kbits); }

// 1. Per-block bbox partials (order keys of the per-axis minima and maxima).
// The call's tile counts, the pair maxima's slots and the bucket tables start
// at zero here.
__global__ __launch_bounds__(kThreads) void lite_bbox_kernel(LiteDev a) {
  const int t = threadIdx.x, lane = t & 63, w = t >> 6, blk = blockIdx.x;
  if (blk == 0) {
    if (t == 0) {
      a.ctrl[kCtrlTiles] = 0u;
      a.ctrl[kCtrlBig] = 0u;
    }
    for (int q = t; q < kMaxSlots * 4; q += kThreads) a.pmax[(q / 4) * kSlotWords + q % 4] = 0u;
  }
  for (int q = blk * kThreads + t; q < kBuckets; q += int(gridDim.x) * kThreads) {
    a.bcnt[q] = 0u;
    a.bval[q] = 0ull;
  }
  const FrontRange r = front_range(a.n);
  __shared__ unsigned int s_u32[6][kWaves];
  unsigned int m[6] = {0xffffffffu, 0xffffffffu, 0xffffffffu, 0u, 0u, 0u};
  for (int i = r.p0 + t; i < r.p1; i += kThreads)
    for (int ax = 0; ax < 3; ++ax) {
      const unsigned int o = float_order_key(a.pos[3 * i + ax]);
      m[ax] = min(m[ax], o);
      m[3 + ax] = max(m[3 + ax], o);
    }
  for (int e = 0; e < 6; ++e) {
    unsigned int x = m[e];
    for (int o = 32; o > 0; o >>= 1) {
      const unsigned int y = (unsigned int)__shfl_xor((int)x, o);
      x = e < 3 ? min(x, y) : max(x, y);
    }
    if (lane == 0) s_u32[e][w] = x;
  }
  __syncthreads();
  if (t < 6) {
    unsigned int x = s_u32[t][0];
    for (int q = 1; q < kWaves; ++q) x = t < 3 ? min(x, s_u32[t][q]) : max(x, s_u32[t][q]);
    a.bbox_part[blk * 6 + t] = x;
  }
}

// 2. Morton keys, bucket counts and capacity sums.  Each block counts its
// keys per bucket in LDS (a key's rank among the block's keys of its
// bucket), adds its counts and capacity units to the bucket tables with one
// returning atomic per non-empty bucket (the return is the block's base in
// that bucket, blocks landing in any order) and stores every token's place
// in its bucket, base plus rank.
__global__ __launch_bounds__(kThreads) void lite_keys_kernel(LiteDev a) {
  const int t = threadIdx.x, lane = t & 63, blk = blockIdx.x, G = gridDim.x;
  const FrontRange r = front_range(a.n);
  __shared__ unsigned int s_bb[6];
  __shared__ unsigned int s_cnt[kBuckets];
  __shared__ unsigned long long s_vb[kBuckets];
  if (t < 64) {
    // lane b reads block b's partials (blocks past G repeat the last one)
#pragma unroll
    for (int e = 0; e < 6; ++e) {
      unsigned int x = a.bbox_part[min(lane, G - 1) * 6 + e];
      for (int o = 32; o > 0; o >>= 1) {
        const unsigned int y = (unsigned int)__shfl_xor((int)x, o);
        x = e < 3 ? min(x, y) : max(x, y);
      }
      if (lane == 0) s_bb[e] = x;
    }
  }
  for (int q = t; q < kBuckets; q += kThreads) {
    s_cnt[q] = 0u;
    s_vb[q] = 0ull;
  }
  __syncthreads();
  double org[3];
  unsigned int qmax[3];
  for (int ax = 0; ax < 3; ++ax) {
    org[ax] = double(float_from_order_key(s_bb[ax]));
    qmax[ax] = grid_coord(float_from_order_key(s_bb[3 + ax]), org[ax], a.grid_scale);
  }
  const unsigned long long kbound = morton3(qmax[0], qmax[1], qmax[2]);
  const int kbits = kbound ? 64 - __clzll((long long)kbound) : 0;
  const int bshift = bucket_shift(kbits);
  if (blk == 0 && t == 0) {
    a.geom[0] = org[0];
    a.geom[1] = org[1];
    a.geom[2] = org[2];
    a.geom[3] = double(kbits);
  }
  for (int i = r.p0 + t; i < r.p1; i += kThreads) {
    const unsigned long long key = morton3(grid_coord(a.pos[3 * i], org[0], a.grid_scale),
                                           grid_coord(a.pos[3 * i + 1], org[1], a.grid_scale),
                                           grid_coord(a.pos[3 * i + 2], org[2], a.grid_scale));
    a.key[0][i] = key;
    const int bk = bucket_of(key, bshift);
    a.within[i] = atomicAdd(&s_cnt[bk], 1u);
    atomicAdd(&s_vb[bk], capacity_units(a.v[i]));
  }
  __syncthreads();
  for (int q = t; q < kBuckets; q += kThreads) {
    const unsigned int c = s_cnt[q];
    if (c) {
      s_cnt[q] = __hip_atomic_fetch_add(a.bcnt + q, c, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_fetch_add(a.bval + q, s_vb[q], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
  __syncthreads();
  // Each thread revisits its own tokens (its own stores, read back).
  for (int i = r.p0 + t; i < r.p1; i += kThreads) a.within[i] += s_cnt[bucket_of(a.key[0][i], bshift)];
}

// 3. Bucket starts (an exclusive scan of the counts), the spans (block b
// owns the whole buckets that start in [b tile, (b + 1) tile)), the capacity
// units before each span (from the bucket sums), and every token placed in
// its bucket: key[1] / tok[0] at bucket start + place.
__global__ __launch_bounds__(kThreads) void lite_place_kernel(LiteDev a) {
  const int t = threadIdx.x, blk = blockIdx.x, G = gridDim.x, n = a.n;
  const FrontRange r = front_range(n);
  __shared__ unsigned int s_start[kBuckets];
  __shared__ unsigned long long s_u64[kThreads + 2];
  __shared__ int s_first;
  const int bshift = bucket_shift(int(a.geom[3]));
  unsigned int c[kPerThread];
  unsigned long long vb[kPerThread];
#pragma unroll
  for (int j = 0; j < kPerThread; ++j) {
    c[j] = a.bcnt[t * kPerThread + j];
    vb[j] = a.bval[t * kPerThread + j];
  }
  unsigned long long csum = 0ull;
#pragma unroll
  for (int j = 0; j < kPerThread; ++j) csum += c[j];
  unsigned long long ctot;
  unsigned int st = unsigned(block_excl_sum_u64(csum, s_u64, ctot));
#pragma unroll
  for (int j = 0; j < kPerThread; ++j) {
    s_start[t * kPerThread + j] = st;
    st += c[j];
  }
  __syncthreads();
  if (t <= G) {
    const unsigned int target = unsigned(min(n, t * r.tile));
    int lo = 0, hi = kBuckets;   // first bucket starting at or after target
    while (lo < hi) {
      const int mid = (lo + hi) >> 1;
      if (s_start[mid] < target) lo = mid + 1;
      else hi = mid;
    }
    if (blk == 0) a.span[t] = lo < kBuckets ? int(s_start[lo]) : n;
    if (t == blk) s_first = lo;
  }
  __syncthreads();
  const int fb = s_first;
  unsigned long long below = 0ull, all = 0ull;
#pragma unroll
  for (int j = 0; j < kPerThread; ++j) {
    if (t * kPerThread + j < fb) below += vb[j];
    all += vb[j];
  }
  const unsigned long long run = block_sum_u64(below, s_u64);
  const unsigned long long W = block_sum_u64(all, s_u64);
  if (t == 0) {
    a.span_run[blk] = run;
    if (blk == 0) *reinterpret_cast<unsigned long long*>(a.ctrl + kCtrlW) = W;
  }
  for (int i = r.p0 + t; i < r.p1; i += kThreads) {
    const unsigned long long key = a.key[0][i];
    const unsigned int slot = s_start[bucket_of(key, bshift)] + a.within[i];
    a.key[1][slot] = key;
    a.tok[0][slot] = i;
  }
}

// A span too long for the register sort, or whose keys do not pack with a
// token index: a stable LSD radix sort of its (key, token) pairs in 8-bit
// digits, the token's digits first, inside the block, then the positions'
// tokens, voxels and group offsets chunk by chunk (the same terms as
// span_offsets).  Data moves between (key[1], tok[0]) and (key[0], tok[1])
// over the span's positions, which no other block touches; it ends in
// tok[1].  Returns the thread's minimum tp - p.
__device__ int span_radix(const LiteDev& a, int r0, int m, int kbits, int tokbits, const double (&org)[3],
                          unsigned long long run, unsigned long long W, unsigned long long* s_u64,
                          unsigned int* s_base, unsigned int (*s_wcnt)[kBins]) {
  const int t = threadIdx.x, lane = t & 63, w = t >> 6;
  const int tpass = (tokbits + 7) / 8, passes = tpass + (kbits + 7) / 8;
  for (int pass = 0; pass < passes; ++pass) {
    const int src = pass & 1;
    const unsigned long long* ks = (src ? a.key[0] : a.key[1]) + r0;
    const int* ts = (src ? a.tok[1] : a.tok[0]) + r0;
    unsigned long long* kd = (src ? a.key[1] : a.key[0]) + r0;
    int* td = (src ? a.tok[0] : a.tok[1]) + r0;
    auto digit = [&](unsigned long long k, int tk) {
      return pass < tpass ? unsigned(tk >> (8 * pass)) & 0xffu : unsigned(k >> (8 * (pass - tpass))) & 0xffu;
    };
    // Digit counts over the span, then every digit's first slot.
    s_base[t] = 0u;
    __syncthreads();
    for (int i = t; i < m; i += kThreads) atomicAdd(&s_base[digit(get(ks + i), get(ts + i))], 1u);
    __syncthreads();
    {
      const unsigned int cnt = s_base[t];
      unsigned long long total;
      const unsigned long long ex = block_excl_sum_u64(cnt, s_u64, total);
      s_base[t] = unsigned(ex);
    }
    __syncthreads();
    // Stable scatter, 256 items per round: rank among equal digits inside a
    // wave from ballots, then across the block's waves through LDS.
    for (int c0 = 0; c0 < m; c0 += kThreads) {
      const int i = c0 + t;
      const bool live = i < m;
      const unsigned long long kv = live ? get(ks + i) : 0ull;
      const int tv = live ? get(ts + i) : 0;
      const unsigned int dig = digit(kv, tv);
      unsigned long long same = __ballot(live);
      for (int bit = 0; bit < 8; ++bit) {
        const unsigned long long mb = __ballot(live && ((dig >> bit) & 1u));
        same &= ((dig >> bit) & 1u) ? mb : ~mb;
      }
      const unsigned long long below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
      const int rank = __popcll(same & below);
      for (int q = t; q < kWaves * kBins; q += kThreads) (&s_wcnt[0][0])[q] = 0u;
      __syncthreads();
      if (live && rank == 0) s_wcnt[w][dig] = unsigned(__popcll(same));
      __syncthreads();
      if (live) {
        unsigned int off = s_base[dig];
        for (int q = 0; q < w; ++q) off += s_wcnt[q][dig];
        put(kd + off + rank, kv);
        put(td + off + rank, tv);
      }
      __syncthreads();
      unsigned int add = 0u;
      for (int q = 0; q < kWaves; ++q) add += s_wcnt[q][t];
      s_base[t] += add;
      __syncthreads();
    }
    __builtin_amdgcn_s_waitcnt(0x0F70);   // vmcnt(0): this pass's stores are done before the next reads them
    __syncthreads();
  }
  // An even number of passes left the tokens in tok[0]: move them.
  if ((passes & 1) == 0) {
    for (int i = t; i < m; i += kThreads) put(a.tok[1] + r0 + i, get(a.tok[0] + r0 + i));
    __builtin_amdgcn_s_waitcnt(0x0F70);
    __syncthreads();
  }
  const unsigned long long KK = (unsigned long long)a.k;
  const double kw = W ? double(a.k) / double(W) : 0.0;
  int bmin = INT_MAX;
  for (int c0 = 0; c0 < m; c0 += kThreads) {
    const int i = c0 + t;
    const int pos = r0 + i;
    const int tk = i < m ? get(a.tok[1] + pos) : 0;
    const unsigned long long V = i < m ? capacity_units(a.v[tk]) : 0ull;
    unsigned long long chunk;
    const unsigned long long ex = block_excl_sum_u64(V, s_u64, chunk);
    if (i < m) {
      a.vox_pos[pos] = pack_vox(grid_coord(a.pos[3 * tk], org[0], a.grid_scale) >> kSubBits,
                                grid_coord(a.pos[3 * tk + 1], org[1], a.grid_scale) >> kSubBits,
                                grid_coord(a.pos[3 * tk + 2], org[2], a.grid_scale) >> kSubBits);
      long long tp;
      if (pos == 0) tp = 0;
      else if (W == 0ull) tp = a.k - 1;
      else tp = thresholds_crossed(KK, run + ex, W, kw);
      const int mm = int(tp - pos);
      a.gid[pos] = mm;
      bmin = min(bmin, mm);
    }
    run += chunk;
  }
  return bmin;
}

// 4. Each block sorts its span by (key, token) -- in registers when it holds
// at most kSortCap tokens and key and token pack into 64 bits, else with
// span_radix -- and writes the permutation, the voxels by position and the
// group offsets tp - p of its positions (Eq. 17 in scan form), and its
// minimum offset.
__global__ __launch_bounds__(kThreads) void lite_sort_kernel(LiteDev a) {
  const int t = threadIdx.x, lane = t & 63, w = t >> 6, blk = blockIdx.x;
  __shared__ unsigned long long s_a[kSortCap], s_b[kSortCap];
  __shared__ unsigned long long s_u64[kThreads + 2];
  __shared__ unsigned int s_base[kBins];
  __shared__ unsigned int s_wcnt[kWaves][kBins];
  __shared__ int s_i32[kWaves];
  const int r0 = a.span[blk], m = a.span[blk + 1] - r0;
  const unsigned long long run = a.span_run[blk];
  const unsigned long long W = *reinterpret_cast<const unsigned long long*>(a.ctrl + kCtrlW);
  const double org[3] = {a.geom[0], a.geom[1], a.geom[2]};
  const int kbits = int(a.geom[3]), tokbits = tok_bits(a.n);
  int bmin = INT_MAX;
  if (m > 0) {
    if (m <= kSortCap && kbits + tokbits <= 64) {
      int per = 1;
      while (kThreads * per < m) per <<= 1;
      const int i0 = min(m, t * per), i1 = min(m, t * per + per);
      const unsigned long long tmask = tokbits ? (~0ull >> (64 - tokbits)) : 0ull;
      const unsigned long long* ks = a.key[1] + r0;
      const int* ts = a.tok[0] + r0;
      switch (per) {
        case 1:
          span_sort<1>(ks, ts, tokbits, m, s_a, s_b);
          bmin = span_offsets<1>(a, r0, m, i0, i1, tmask, org, run, W, s_a, s_u64);
          break;
        case 2:
          span_sort<2>(ks, ts, tokbits, m, s_a, s_b);
          bmin = span_offsets<2>(a, r0, m, i0, i1, tmask, org, run, W, s_a, s_u64);
          break;
        case 4:
          span_sort<4>(ks, ts, tokbits, m, s_a, s_b);
          bmin = span_offsets<4>(a, r0, m, i0, i1, tmask, org, run, W, s_a, s_u64);
          break;
        case 8:
          span_sort<8>(ks, ts, tokbits, m, s_a, s_b);
          bmin = span_offsets<8>(a, r0, m, i0, i1, tmask, org, run, W, s_a, s_u64);
          break;
        default:
          span_sort<16>(ks, ts, tokbits, m, s_a, s_b);
          bmin = span_offsets<16>(a, r0, m, i0, i1, tmask, org, run, W, s_a, s_u64);
          break;
      }
    } else {
      bmin = span_radix(a, r0, m, kbits, tokbits, org, run, W, s_u64, s_base, s_wcnt);
    }
  }
  bmin = wave_min(bmin);
  if (lane == 0) s_i32[w] = bmin;
  __syncthreads();
  if (t == 0) {
    int mm = s_i32[0];
    for (int q = 1; q < kWaves; ++q) mm = min(mm, s_i32[q]);
    a.bmin[blk] = mm;
  }
}

// 5. Groups of the span's positions: the prefix minimum of the offsets
// (earlier blocks, earlier threads, then this thread's positions in order)
// gives each position's group (the walk of Eq. 17 in scan form); group
// starts where the group changes; the group output.
__global__ __launch_bounds__(kThreads) void lite_groups_kernel(LiteDev a) {
  const int t = threadIdx.x, blk = blockIdx.x, n = a.n, K = a.k;
  __shared__ int s_i32[kThreads];
  __shared__ int s_minoff;
  const int r0 = a.span[blk], m = a.span[blk + 1] - r0;
  s_i32[t] = t < blk ? a.bmin[t] : INT_MAX;
  __syncthreads();
  if (t == 0) {
    int mm = INT_MAX;
    for (int b = 0; b < blk; ++b) mm = min(mm, s_i32[b]);
    s_minoff = mm;
  }
  __syncthreads();
  if (m <= 0) return;
  const int per = (m + kThreads - 1) / kThreads;
  const int i0 = min(m, t * per), i1 = min(m, t * per + per);
  int lmin = INT_MAX;
  for (int i = i0; i < i1; ++i) lmin = min(lmin, a.gid[r0 + i]);
  const int incl = block_incl_min(lmin, s_i32);
  s_i32[t] = incl;
  __syncthreads();
  int cur = min(s_minoff, t > 0 ? s_i32[t - 1] : INT_MAX);   // prefix minimum before position r0 + i0
  int qprev = r0 + i0 > 0 ? max(K - n + r0 + i0 - 1, r0 + i0 - 1 + cur) : -1;
  for (int i = i0; i < i1; ++i) {
    const int pos = r0 + i;
    cur = min(cur, a.gid[pos]);
    const int q = max(K - n + pos, pos + cur);
    if (q != qprev) a.gstart[q] = pos;
    if (pos == n - 1) a.gstart[K] = n;
    if (a.group) a.group[a.tok[1][pos]] = q;
    qprev = q;
  }
}

// 6. Tiles per group and tiles of big groups, summed per block of groups.
__global__ __launch_bounds__(kThreads) void lite_tile_sums_kernel(LiteDev a) {
  const int t = threadIdx.x, blk = blockIdx.x, G = gridDim.x, K = a.k;
  __shared__ unsigned long long s_u64[kThreads + 2];
  const int gtile = (K + G - 1) / G;
  const int q0 = min(K, blk * gtile), q1 = min(K, q0 + gtile);
  unsigned long long local = 0ull, lbig = 0ull;
  for (int q = q0 + t; q < q1; q += kThreads) {
    const int g = max(0, a.gstart[q + 1] - a.gstart[q]);
    const int nt = (g + kTileRows - 1) / kTileRows;
    local += (unsigned long long)nt;
    lbig += nt > kSplitTiles ? (unsigned long long)nt : 0ull;
  }
  unsigned long long tot, tbig;
  block_excl_sum_u64(local, s_u64, tot);
  block_excl_sum_u64(lbig, s_u64, tbig);
  if (t == 0) {
    a.bsum[blk] = tot;
    a.bsum2[blk] = tbig;
  }
}

// 7. The tile prefix per group, the group of every tile and the list of big
// groups' tiles (work units of the pair kernels).
__global__ __launch_bounds__(kThreads) void lite_tiles_kernel(LiteDev a) {
  const int t = threadIdx.x, blk = blockIdx.x, G = gridDim.x, K = a.k;
  __shared__ unsigned long long s_u64[kThreads + 2];
  const int gtile = (K + G - 1) / G;
  const int q0 = min(K, blk * gtile), q1 = min(K, q0 + gtile);
  unsigned long long run, tot, rbig, tbig;
  block_prefix_u64(a.bsum, G, blk, s_u64, run, tot);
  block_prefix_u64(a.bsum2, G, blk, s_u64, rbig, tbig);
  if (blk == 0 && t == 0) {
    a.ctrl[kCtrlTiles] = unsigned(tot);
    a.ctrl[kCtrlBig] = unsigned(tbig);
  }
  for (int c0 = q0; c0 < q1; c0 += kThreads) {
    const int q = c0 + t;
    int nt = 0;
    if (q < q1) {
      const int g = max(0, a.gstart[q + 1] - a.gstart[q]);
      nt = (g + kTileRows - 1) / kTileRows;
    }
    const int nb = nt > kSplitTiles ? nt : 0;
    unsigned long long chunk, cbig;
    const unsigned long long ex = block_excl_sum_u64((unsigned long long)nt, s_u64, chunk);
    const unsigned long long exb = block_excl_sum_u64((unsigned long long)nb, s_u64, cbig);
    if (q < q1) {
      const int u0 = int(run + ex), b0 = int(rbig + exb);
      a.rt_start[q] = u0;
      for (int x = 0; x < nt; ++x) a.unit_group[u0 + x] = q;
      for (int x = 0; x < nb; ++x) a.big_unit[b0 + x] = u0 + x;
    }
    if (q == K - 1) a.rt_start[K] = int(run + ex + nt);
    run += chunk;
    rbig += cbig;
  }
}

// ---------------------------------------------------------------------------
// Within-group pair pass.  Work unit: one 16-row tile ta of one group,
// multiplied on the matrix cores against every 16-row tile tb of the same
// group over the full feature width.  The same pass raises M_x and M_tau:
// it visits every evaluated pair (same group, adjacent voxels, diagonal
// included), which is the set those maxima range over.  Lane l supplies row l % 16 and feature
// slice 8 (l / 16) .. +8 of each 32-wide K step (bf16), or 4 (l / 16) .. +4 of
// each 16-wide step spread over four MFMAs (f32); the output element
// (4 (l / 16) + r, l % 16) lands in register r of lane l.  A group of at most
// kSplitTiles tiles takes one wave per unit (lite_pair_kernel); a larger one
// takes one block per unit whose waves split the column tiles and add their
// row sums in wave order (lite_pair_split_kernel), so a big group does not
// leave one wave working through all its tiles alone.
struct Unit {
  int p0, g, ntile, ta;
};

// Group and row tile of unit u, from the front's table.
__device__ __forceinline__ bool unit_of(const LiteDev& a, int u, Unit& t) {
  const int q = min(max(a.unit_group[u], 0), a.k - 1);
  t.p0 = clamp_range(a.gstart[q], a.n);
  t.g = max(0, clamp_range(a.gstart[q + 1], a.n) - t.p0);
  t.ntile = (t.g + kTileRows - 1) / kTileRows;
  t.ta = u - a.rt_start[q];
  return t.ta >= 0 && t.ta < t.ntile;
}

// Running maxima of one lane over the pairs it evaluates: squared distance
// (float64) and frame gap.
struct PairMax {
  float df = 0.f;
  double x2 = 0.0;
  int tau = 0;
};

// The maxima over all slots, in a kernel after the pair kernels: lane q of
// the wave reads slot q, then maxima across the wave (every lane active).
struct PairMaxima {
  float df;
  double x2;
  int tau;
};
__device__ __forceinline__ PairMaxima pair_maxima(const LiteDev& a) {
  static_assert(kMaxSlots <= 64, "one slot per lane");
  const int lane = threadIdx.x & 63;
  PairMaxima m{0.f, 0.0, 0};
  if (lane < kMaxSlots) {
    const unsigned int* slot = a.pmax + lane * kSlotWords;
    m.df = __uint_as_float(slot[kSlotMf]);
    m.tau = int(slot[kSlotMt]);
    m.x2 = __longlong_as_double(*reinterpret_cast<const long long*>(slot + kSlotMx2));
  }
  m.df = wave_max(m.df);
  m.x2 = wave_max(m.x2);
  m.tau = wave_max(m.tau);
  return m;
}

// The epilogue of a tile product: acc holds row tile t.ta against column
// tile tb (output element (4 (l / 16) + r, l % 16) in register r of lane l),
// na the squared norm of the lane's row l % 16 of tile ta and nb that of
// column tile tb's row l % 16.  Adds v_j d_f over adjacent pairs to arow
// (the lane's four output rows) and raises the maxima.
__device__ __forceinline__ void pair_epilogue(const LiteDev& a, const int* perm, const Unit& t, int tb,
                                              const f32x4& acc, float na, float nb, double* arow, PairMax& pm) {
  const int lane = threadIdx.x & 63;
  const int row = lane & 15, quad = lane >> 4;
  const int ra = t.ta * kTileRows + row;
  const int cb = tb * kTileRows + row;    // output column of this lane
  const bool cvalid = cb < t.g;
  const int tokb = cvalid ? perm[t.p0 + cb] : 0;
  const unsigned long long vb = cvalid ? a.vox_pos[t.p0 + cb] : 0ull;
  const double wv = cvalid ? double(a.v[tokb]) : 0.0;
  const float xb = a.pos[3 * tokb], yb = a.pos[3 * tokb + 1], zb = a.pos[3 * tokb + 2];
  const int fb = a.frame[tokb];
  // Lane l (l < 16) also holds row l of tile ta's position and frame.
  const int toka = ra < t.g ? perm[t.p0 + ra] : 0;
  const float xa = a.pos[3 * toka], ya = a.pos[3 * toka + 1], za = a.pos[3 * toka + 2];
  const int fa = a.frame[toka];
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int oa = quad * 4 + r;           // output row within tile ta
    const float nra = __shfl(na, oa);
    const float xo = __shfl(xa, oa), yo = __shfl(ya, oa), zo = __shfl(za, oa);
    const int fo = __shfl(fa, oa);
    const int ca = t.ta * kTileRows + oa;
    if (cvalid && ca < t.g && adjacent(a.vox_pos[t.p0 + ca], vb)) {
      const float den = sqrtf(nra) * sqrtf(nb);
      const float cosv = den > 0.f ? acc[r] / den : 0.f;
      float df = fminf(fmaxf(1.f - cosv, 0.f), 2.f);
      if (ca == cb) df = 0.f;
      arow[r] = fma(wv, double(df), arow[r]);
      pm.df = fmaxf(pm.df, df);
      pm.x2 = fmax(pm.x2, sq_dist(xo, yo, zo, xb, yb, zb));
      pm.tau = max(pm.tau, abs(fo - fb));
    }
  }
}


// Row tile t.ta against column tile tb: the product over the feature width,
// then pair_epilogue.
template <bool BF16>
__device__ __forceinline__ void pair_tile(const LiteDev& a, const int* perm, const Unit& t, int tb, double* arow,
                                          PairMax& pm) {
  const int lane = threadIdx.x & 63;
  const int row = lane & 15, quad = lane >> 4;
  const int ra = t.ta * kTileRows + row;  // operand row of this lane in tile ta
  const int rb = tb * kTileRows + row;
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  float na = 0.f, nb = 0.f;
  if (BF16) {
    const uint16_t* Fa = ra < t.g ? static_cast<const uint16_t*>(a.feats) + size_t(perm[t.p0 + ra]) * a.d : nullptr;
    const uint16_t* Fb = rb < t.g ? static_cast<const uint16_t*>(a.feats) + size_t(perm[t.p0 + rb]) * a.d : nullptr;
    // Eight 32-wide K steps per round: all loads first, then the MFMAs.
    constexpr int U = 8;
    const bool same = tb == t.ta;
    for (int k0 = 0; k0 < a.d; k0 += 32 * U) {
      uint4 ua[U], ub[U];
#pragma unroll
      for (int x = 0; x < U; ++x) {
        const int kk = k0 + 32 * x + quad * 8;
        ua[x] = uint4{0u, 0u, 0u, 0u};
        ub[x] = uint4{0u, 0u, 0u, 0u};
        if (Fa && kk < a.d) ua[x] = *reinterpret_cast<const uint4*>(Fa + kk);
        if (!same && Fb && kk < a.d) ub[x] = *reinterpret_cast<const uint4*>(Fb + kk);
      }
#pragma unroll
      for (int x = 0; x < U; ++x) {
        if (same) ub[x] = ua[x];
        const uint32_t wa[4] = {ua[x].x, ua[x].y, ua[x].z, ua[x].w}, wb[4] = {ub[x].x, ub[x].y, ub[x].z, ub[x].w};
#pragma unroll
        for (int h = 0; h < 4; ++h) {
          const float a0 = bf16_bits_to_float(wa[h] & 0xffffu), a1 = bf16_bits_to_float(wa[h] >> 16);
          const float b0 = bf16_bits_to_float(wb[h] & 0xffffu), b1 = bf16_bits_to_float(wb[h] >> 16);
          na = fmaf(a0, a0, fmaf(a1, a1, na));
          nb = fmaf(b0, b0, fmaf(b1, b1, nb));
        }
        bf16x8 va, vb;
        __builtin_memcpy(&va, &ua[x], sizeof va);
        __builtin_memcpy(&vb, &ub[x], sizeof vb);
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(va, vb, acc, 0, 0, 0);
      }
    }
  } else {
    const float* Fa = ra < t.g ? static_cast<const float*>(a.feats) + size_t(perm[t.p0 + ra]) * a.d : nullptr;
    const float* Fb = rb < t.g ? static_cast<const float*>(a.feats) + size_t(perm[t.p0 + rb]) * a.d : nullptr;
    for (int k0 = 0; k0 < a.d; k0 += 16) {
      const int kk = k0 + quad * 4;
      float4 fa = make_float4(0.f, 0.f, 0.f, 0.f), fb = fa;
      if (Fa && kk < a.d) fa = *reinterpret_cast<const float4*>(Fa + kk);
      if (tb == t.ta) fb = fa;
      else if (Fb && kk < a.d) fb = *reinterpret_cast<const float4*>(Fb + kk);
      na = fmaf(fa.x, fa.x, fmaf(fa.y, fa.y, fmaf(fa.z, fa.z, fmaf(fa.w, fa.w, na))));
      nb = fmaf(fb.x, fb.x, fmaf(fb.y, fb.y, fmaf(fb.z, fb.z, fmaf(fb.w, fb.w, nb))));
      acc = __builtin_amdgcn_mfma_f32_16x16x4f32(fa.x, fb.x, acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_16x16x4f32(fa.y, fb.y, acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_16x16x4f32(fa.z, fb.z, acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_16x16x4f32(fa.w, fb.w, acc, 0, 0, 0);
    }
  }
  // Row sums of squares: the four lanes sharing l % 16 hold its slices.
  na += __shfl_xor(na, 16);
  na += __shfl_xor(na, 32);
  nb += __shfl_xor(nb, 16);
  nb += __shfl_xor(nb, 32);
  pair_epilogue(a, perm, t, tb, acc, na, nb, arow, pm);
}

// Row tile t.ta of a group of two tiles against both column tiles, with
// bfloat16 features: the lane's rows of both tiles are read once per K step
// and feed the products ta x ta and ta x tb, which then go through
// pair_epilogue in column-tile order, as the two pair_tile calls they
// replace (the same products and sums, so the same values).  Those calls
// read tile ta's rows twice.
__device__ __forceinline__ void pair_tile_both(const LiteDev& a, const int* perm, const Unit& t, double* arow,
                                               PairMax& pm) {
  const int lane = threadIdx.x & 63;
  const int row = lane & 15, quad = lane >> 4;
  const int tb = 1 - t.ta;
  const int ra = t.ta * kTileRows + row, rb = tb * kTileRows + row;
  const uint16_t* Fa = ra < t.g ? static_cast<const uint16_t*>(a.feats) + size_t(perm[t.p0 + ra]) * a.d : nullptr;
  const uint16_t* Fb = rb < t.g ? static_cast<const uint16_t*>(a.feats) + size_t(perm[t.p0 + rb]) * a.d : nullptr;
  f32x4 caa = {0.f, 0.f, 0.f, 0.f}, cab = caa;
  float na = 0.f, nb = 0.f;
  constexpr int U = 8;
  for (int k0 = 0; k0 < a.d; k0 += 32 * U) {
    uint4 ua[U], ub[U];
#pragma unroll
    for (int x = 0; x < U; ++x) {
      const int kk = k0 + 32 * x + quad * 8;
      ua[x] = uint4{0u, 0u, 0u, 0u};
      ub[x] = uint4{0u, 0u, 0u, 0u};
      if (Fa && kk < a.d) ua[x] = *reinterpret_cast<const uint4*>(Fa + kk);
      if (Fb && kk < a.d) ub[x] = *reinterpret_cast<const uint4*>(Fb + kk);
    }
#pragma unroll
    for (int x = 0; x < U; ++x) {
      const uint32_t wa[4] = {ua[x].x, ua[x].y, ua[x].z, ua[x].w}, wb[4] = {ub[x].x, ub[x].y, ub[x].z, ub[x].w};
#pragma unroll
      for (int h = 0; h < 4; ++h) {
        const float a0 = bf16_bits_to_float(wa[h] & 0xffffu), a1 = bf16_bits_to_float(wa[h] >> 16);
        const float b0 = bf16_bits_to_float(wb[h] & 0xffffu), b1 = bf16_bits_to_float(wb[h] >> 16);
        na = fmaf(a0, a0, fmaf(a1, a1, na));
        nb = fmaf(b0, b0, fmaf(b1, b1, nb));
      }
      bf16x8 va, vb;
      __builtin_memcpy(&va, &ua[x], sizeof va);
      __builtin_memcpy(&vb, &ub[x], sizeof vb);
      caa = __builtin_amdgcn_mfma_f32_16x16x32_bf16(va, va, caa, 0, 0, 0);
      cab = __builtin_amdgcn_mfma_f32_16x16x32_bf16(va, vb, cab, 0, 0, 0);
    }
  }
  na += __shfl_xor(na, 16);
  na += __shfl_xor(na, 32);
  nb += __shfl_xor(nb, 16);
  nb += __shfl_xor(nb, 32);
  if (t.ta == 0) {
    pair_epilogue(a, perm, t, 0, caa, na, na, arow, pm);
    pair_epilogue(a, perm, t, 1, cab, na, nb, arow, pm);
  } else {
    pair_epilogue(a, perm, t, 0, cab, na, nb, arow, pm);
    pair_epilogue(a, perm, t, 1, caa, na, na, arow, pm);
  }
}

// Folds a block's maxima into the control words.  Atomics on one cache line
// from many blocks serialize, so a block first reads the current value (the
// maxima only grow) and issues an atomic only where it holds a larger one.
template <int NW>
__device__ __forceinline__ void pair_max_to(const LiteDev& a, PairMax pm) {
  __shared__ float sf[NW];
  __shared__ double sx[NW];
  __shared__ int st[NW];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  pm.df = wave_max(pm.df);
  pm.x2 = wave_max(pm.x2);
  pm.tau = wave_max(pm.tau);
  if (lane == 0) {
    sf[w] = pm.df;
    sx[w] = pm.x2;
    st[w] = pm.tau;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int q = 1; q < NW; ++q) {
      pm.df = fmaxf(pm.df, sf[q]);
      pm.x2 = fmax(pm.x2, sx[q]);
      pm.tau = max(pm.tau, st[q]);
    }
    unsigned int* slot = a.pmax + (blockIdx.x % kMaxSlots) * kSlotWords;
    unsigned long long* mx2 = reinterpret_cast<unsigned long long*>(slot + kSlotMx2);
    if (pm.df > __uint_as_float(get(slot + kSlotMf))) atomic_max_nonneg(slot + kSlotMf, pm.df);
    if (pm.x2 > __longlong_as_double((long long)get(mx2))) atomic_max_nonneg(mx2, pm.x2);
    if (unsigned(pm.tau) > get(slot + kSlotMt)) atomicMax(slot + kSlotMt, unsigned(pm.tau));
  }
}

// Sum each output row over the 16 lanes (columns) that share it.
__device__ __forceinline__ void row_sums(double* arow) {
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    double x = arow[r];
    x += __shfl_xor(x, 1);
    x += __shfl_xor(x, 2);
    x += __shfl_xor(x, 4);
    x += __shfl_xor(x, 8);
    arow[r] = x;
  }
}

template <bool BF16>
__global__ __launch_bounds__(kThreads, 4) void lite_pair_kernel(LiteDev a) {
  const int lane = threadIdx.x & 63;
  const int gw = blockIdx.x * kWaves + (threadIdx.x >> 6);
  const int nw = gridDim.x * kWaves;
  const int* perm = a.tok[1];
  const int units = int(a.ctrl[kCtrlTiles]);
  const int row = lane & 15, quad = lane >> 4;
  PairMax pm;
  for (int u = gw; u < units; u += nw) {
    Unit t;
    if (!unit_of(a, u, t) || t.ntile > kSplitTiles) continue;
    double arow[4] = {0.0, 0.0, 0.0, 0.0};
    if (BF16 && t.ntile == 2)
      pair_tile_both(a, perm, t, arow, pm);
    else
      for (int tb = 0; tb < t.ntile; ++tb) pair_tile<BF16>(a, perm, t, tb, arow, pm);
    row_sums(arow);
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int ca = t.ta * kTileRows + quad * 4 + r;
      if (row == 0 && ca < t.g) a.A[t.p0 + ca] = arow[r];
    }
  }
  pair_max_to<kWaves>(a, pm);
}

constexpr int kSplitWaves = 16;

template <bool BF16>
__global__ __launch_bounds__(kSplitWaves * 64) void lite_pair_split_kernel(LiteDev a) {
  __shared__ double spart[kSplitWaves][kTileRows];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int* perm = a.tok[1];
  const int nbig = int(a.ctrl[kCtrlBig]);
  const int row = lane & 15, quad = lane >> 4;
  PairMax pm;
  for (int b = blockIdx.x; b < nbig; b += gridDim.x) {
    Unit t;
    if (!unit_of(a, a.big_unit[b], t)) continue;   // the same for the whole block
    double arow[4] = {0.0, 0.0, 0.0, 0.0};
    for (int tb = w; tb < t.ntile; tb += kSplitWaves) pair_tile<BF16>(a, perm, t, tb, arow, pm);
    row_sums(arow);
    if (row == 0) {
#pragma unroll
      for (int r = 0; r < 4; ++r) spart[w][quad * 4 + r] = arow[r];
    }
    __syncthreads();
    if (threadIdx.x < kTileRows) {
      const int ca = t.ta * kTileRows + threadIdx.x;
      if (ca < t.g) {
        double x = 0.0;
#pragma unroll
        for (int q = 0; q < kSplitWaves; ++q) x += spart[q][threadIdx.x];
        a.A[t.p0 + ca] = x;
      }
    }
    __syncthreads();
  }
  pair_max_to<kSplitWaves>(a, pm);
}

// B(p) = sum over the group of v_j (lam_x phi(d_x / M_x) + lam_tau d_tau / M_tau)
// for adjacent pairs and v_j c0 otherwise: every term of the group cost that
// does not involve features.  One wave per 16-row tile of a group (the pair
// kernels' work units): lane l takes row l % 16 of the tile and every fourth
// member of the group from l / 16 on; the four lanes of a row add their sums
// in a fixed order.
__global__ __launch_bounds__(kThreads) void lite_b_kernel(LiteDev a) {
  const int lane = threadIdx.x & 63;
  const int row = lane & 15, quad = lane >> 4;
  const int gw = blockIdx.x * kWaves + (threadIdx.x >> 6);
  const int nw = gridDim.x * kWaves;
  const int units = int(a.ctrl[kCtrlTiles]);
  const int* perm = a.tok[1];
  const PairMaxima mm = pair_maxima(a);
  const double m_x = sqrt(mm.x2);
  const int m_t = mm.tau;
  const double c0 = double(a.lam_f) + double(a.lam_x) + double(a.lam_t);
  for (int u = gw; u < units; u += nw) {
    Unit t;
    if (!unit_of(a, u, t)) continue;
    const int r = t.ta * kTileRows + row;
    const bool rvalid = r < t.g;
    const int i = t.p0 + min(r, t.g - 1);
    const int tokn = perm[i];
    const unsigned long long vi = a.vox_pos[i];
    const double xi = a.pos[3 * tokn], yi = a.pos[3 * tokn + 1], zi = a.pos[3 * tokn + 2];
    const int fi = a.frame[tokn];
    double acc = 0.0;
    // Members jj, jj + 4, jj + 8, jj + 12 per round: their loads go out
    // together, then their terms are added in member order.
    constexpr int R = 4;
    for (int j0 = quad; j0 < t.g; j0 += 4 * R) {
      int tj[R];
      unsigned long long vj[R];
#pragma unroll
      for (int x = 0; x < R; ++x) {
        const int jj = min(j0 + 4 * x, t.g - 1);
        tj[x] = perm[t.p0 + jj];
        vj[x] = a.vox_pos[t.p0 + jj];
      }
      float px[R], py[R], pz[R], cv[R];
      int fr[R];
#pragma unroll
      for (int x = 0; x < R; ++x) {
        px[x] = a.pos[3 * tj[x]];
        py[x] = a.pos[3 * tj[x] + 1];
        pz[x] = a.pos[3 * tj[x] + 2];
        fr[x] = a.frame[tj[x]];
        cv[x] = a.v[tj[x]];
      }
#pragma unroll
      for (int x = 0; x < R; ++x) {
        if (j0 + 4 * x >= t.g) break;
        const double w = double(cv[x]);
        if (!adjacent(vi, vj[x])) {
          acc += w * c0;
          continue;
        }
        const double dist = sqrt(sq_dist(xi, yi, zi, px[x], py[x], pz[x]));
        const double z = m_x > 0.0 ? dist / m_x : 0.0;
        const double ph = a.kappa > 0.f ? log1p(double(a.kappa) * z) * a.inv_log1p_kappa : z;
        const double dt = m_t > 0 ? double(max(0, fi - fr[x])) / double(m_t) : 0.0;
        acc += w * (double(a.lam_x) * ph + double(a.lam_t) * dt);
      }
    }
    acc += __shfl_xor(acc, 16);
    acc += __shfl_xor(acc, 32);
    if (quad == 0 && rvalid) a.B[i] = acc;
  }
}

// One wave per group: prototype = argmin of (lam_f / M_f) A + B over the
// group's members (lanes), ties to the smaller token index.
__global__ __launch_bounds__(kThreads) void lite_select_kernel(LiteDev a) {
  const int lane = threadIdx.x & 63;
  const int q = blockIdx.x * kWaves + (threadIdx.x >> 6);
  if (q >= a.k) return;
  const int* perm = a.tok[1];
  const float m_f = pair_maxima(a).df;
  const double wf = m_f > 0.f ? double(a.lam_f) / double(m_f) : 0.0;
  double best = DBL_MAX;
  int bt = INT_MAX;
  const int i0 = clamp_range(a.gstart[q], a.n), i1 = clamp_range(a.gstart[q + 1], a.n);
  for (int i = i0 + lane; i < i1; i += 64) {
    const double c = fma(wf, a.A[i], a.B[i]);
    const int tk = perm[i];
    if (a.token_cost) a.token_cost[tk] = c;
    if (c < best || (c == best && tk < bt)) {
      best = c;
      bt = tk;
    }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const double oc = __shfl_xor(best, o);
    const int ot = __shfl_xor(bt, o);
    if (oc < best || (oc == best && ot < bt)) {
      best = oc;
      bt = ot;
    }
  }
  if (lane == 0) {
    a.selected[q] = bt == INT_MAX ? -1 : bt;
    a.gcost[q] = bt == INT_MAX ? 0.0 : best;
  }
}

__global__ __launch_bounds__(kThreads) void lite_total_kernel(LiteDev a) {
  __shared__ double sd[kThreads];
  double x = 0.0;
  for (int q = threadIdx.x; q < a.k; q += kThreads) x += a.gcost[q];
  sd[threadIdx.x] = x;
  __syncthreads();
  for (int o = kThreads / 2; o > 0; o >>= 1) {
    if (int(threadIdx.x) < o) sd[threadIdx.x] += sd[threadIdx.x + o];
    __syncthreads();
  }
  if (threadIdx.x == 0) *a.objective = sd[0];
}

}  // namespace

size_t lite_workspace_bytes(int64_t n, int64_t k) { return layout(n, k).total; }

hipError_t launch_lite(const LiteParams& p, hipStream_t stream) {
  const Layout L = layout(p.n, p.k);
  char* w = static_cast<char*>(p.workspace);
  LiteDev a{};
  a.feats = p.feats;
  a.n = p.n;
  a.d = p.d;
  a.k = p.k;
  a.pos = p.pos;
  a.frame = p.frame;
  a.v = p.capacity;
  a.lam_f = p.lambda_f;
  a.lam_x = p.lambda_x;
  a.lam_t = p.lambda_tau;
  a.kappa = p.kappa;
  a.inv_log1p_kappa = p.inv_log1p_kappa;
  a.grid_scale = p.grid_scale;
  a.selected = p.selected;
  a.group = p.group;
  a.objective = p.objective;
  a.token_cost = p.token_cost;
  a.key[0] = reinterpret_cast<unsigned long long*>(w + L.key0);
  a.key[1] = reinterpret_cast<unsigned long long*>(w + L.key1);
  a.tok[0] = reinterpret_cast<int*>(w + L.tok0);
  a.tok[1] = reinterpret_cast<int*>(w + L.tok1);
  a.vox_pos = reinterpret_cast<unsigned long long*>(w + L.vox_pos);
  a.bbox_part = reinterpret_cast<unsigned int*>(w + L.bbox_part);
  a.within = reinterpret_cast<unsigned int*>(w + L.within);
  a.span = reinterpret_cast<int*>(w + L.span);
  a.span_run = reinterpret_cast<unsigned long long*>(w + L.span_run);
  a.geom = reinterpret_cast<double*>(w + L.geom);
  a.bcnt = reinterpret_cast<unsigned int*>(w + L.bcnt);
  a.bval = reinterpret_cast<unsigned long long*>(w + L.bval);
  a.bsum = reinterpret_cast<unsigned long long*>(w + L.bsum);
  a.bmin = reinterpret_cast<int*>(w + L.bmin);
  a.gid = reinterpret_cast<int*>(w + L.gid);
  a.gstart = reinterpret_cast<int*>(w + L.gstart);
  a.rt_start = reinterpret_cast<int*>(w + L.rt_start);
  a.unit_group = reinterpret_cast<int*>(w + L.unit_group);
  a.big_unit = reinterpret_cast<int*>(w + L.big_unit);
  a.bsum2 = reinterpret_cast<unsigned long long*>(w + L.bsum2);
  a.A = reinterpret_cast<double*>(w + L.A);
  a.B = reinterpret_cast<double*>(w + L.B);
  a.gcost = reinterpret_cast<double*>(w + L.gcost);
  a.ctrl = reinterpret_cast<unsigned int*>(w + L.ctrl);
  a.pmax = reinterpret_cast<unsigned int*>(w + L.pmax);

  // The front: seven ordinary launches (a cooperative launch costs about
  // 20 us more than an ordinary one, and no block of the front waits for
  // another).
  const int G = std::max(1, std::min(kFrontBlocks, (p.n + kThreads - 1) / kThreads));
  lite_bbox_kernel<<<G, kThreads, 0, stream>>>(a);
  lite_keys_kernel<<<G, kThreads, 0, stream>>>(a);
  lite_place_kernel<<<G, kThreads, 0, stream>>>(a);
  lite_sort_kernel<<<G, kThreads, 0, stream>>>(a);
  lite_groups_kernel<<<G, kThreads, 0, stream>>>(a);
  lite_tile_sums_kernel<<<G, kThreads, 0, stream>>>(a);
  lite_tiles_kernel<<<G, kThreads, 0, stream>>>(a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  // One wave per 16-row tile; a group has at most n / 16 + 1 tiles in total
  // over all groups, so n / 16 + k waves cover every tile.
  const int units = p.n / kTileRows + p.k;
  const int blocks = std::max(1, std::min((units + kWaves - 1) / kWaves, 65535));
  // Groups of more than kSplitTiles tiles: one block per row tile.
  const int split_blocks = std::max(1, std::min(units, 256));
  if (p.bf16) {
    lite_pair_kernel<true><<<blocks, kThreads, 0, stream>>>(a);
    lite_pair_split_kernel<true><<<split_blocks, kSplitWaves * 64, 0, stream>>>(a);
  } else {
    lite_pair_kernel<false><<<blocks, kThreads, 0, stream>>>(a);
    lite_pair_split_kernel<false><<<split_blocks, kSplitWaves * 64, 0, stream>>>(a);
  }
  if ((e = hipGetLastError()) != hipSuccess) return e;
  // B needs M_x and M_tau, which the pair kernels raise.
  lite_b_kernel<<<blocks, kThreads, 0, stream>>>(a);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  lite_select_kernel<<<(p.k + kWaves - 1) / kWaves, kThreads, 0, stream>>>(a);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if (p.objective) {
    lite_total_kernel<<<1, kThreads, 0, stream>>>(a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace cp
