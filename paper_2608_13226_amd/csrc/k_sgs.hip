// Greedy coverage selection over the target-major cost (Sec. 3.5, Eq. 14-16).
//
// State: b_j, the best cost at which target j is covered so far (c0 while
// uncovered), and the mask of chosen tokens.  Step l picks
//   t_l = argmax_{c not chosen} gain(c),  gain(c) = sum_j v_j max(0, b_j - C_tm[j][c])
// and then b_j <- min(b_j, C_tm[j][t_l]).
//
// One cooperative launch runs all K steps.  The matrix is cut into P row
// panels x S column strips of 256 columns; the item (panel, strip) is owned by
// one block for the whole launch.  Per step the block
//   1. brings its private copy of b for the panel's rows up to date with the
//      previous pick (b = min(b, C_tm[j][t])) and stages b and v in LDS; the
//      strip-0 item of a panel also updates the assignment and folds the
//      panel's share of the objective;
//   2. streams the panel's rows of its strip (a wave reads 1 KB of a row per
//      16-byte non-temporal load) accumulating float64 gains per column, and
//      writes the panel's partial gains;
//   3. arrives at its strip's counter.  The strip's last block sums the P
//      partials of every column in panel order, masks chosen columns, takes
//      the strip's exact argmax (ties to the smaller index), records it, folds
//      it into the step's packed (gain, index) maximum with one 64-bit
//      atomicMax, and arrives at the step counter;
//   4. waits until every strip has arrived and reads the step's winner.
// Data that crosses blocks (partial gains, strip winners, objective shares,
// the mask, the step's key and counters) is written and read only with
// device-scope atomic operations, which are coherent across the chip's L2
// caches without fences.  A block's writes are complete at the workgroup
// barrier that precedes thread 0's counter update, so a block that observes
// the counter also observes the data.  A device-scope fence would instead
// write back the whole L2 and cost about as much as a step's tail.
// Across strips the packed key compares gains truncated to 44 bits (relative
// resolution 2^-32) and breaks ties by the smaller index; within a strip the
// comparison is exact.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <climits>

#include "common.h"
#include "launch.h"

namespace cp {
namespace {

constexpr int kStrip = 256;        // columns per strip: 64 lanes x 4 floats
constexpr int kMaxPanels = 64;
constexpr int kMaxStrips = (1 << 18) / kStrip;
constexpr int kMinPanelRows = 64;
constexpr int kIndexBits = 20;     // packed key: [44-bit gain | 20-bit inverted index]
constexpr unsigned long long kIndexMask = (1ull << kIndexBits) - 1ull;

struct SgsDev {
  const float* C;
  const float* v;
  int n, k;
  float c0;
  int32_t* selected;
  double* step_gain;
  double* step_obj;
  int32_t* assign;
  float* bpriv;              // [items][rows] private best costs
  unsigned int* mask;        // [n] 1 once chosen
  double* partial;           // [P][n]
  double* strip_g;           // [S] exact gain of each strip's winner
  double* obj_part;          // [P]
  unsigned long long* key;   // [k] packed step maxima
  unsigned int* strip_cnt;   // [S]
  unsigned int* step_cnt;
  unsigned int* fin_cnt;
  unsigned int* abort;       // set when the step wait gives up
  unsigned int poll_limit;   // polls before it gives up (WaitPolicy)
  unsigned int abort_init;   // the abort flag's value at launch
  int P, S, rows;            // panels, strips, rows per panel
};

struct Layout {
  size_t bpriv, mask, partial, strip_g, obj_part, key, strip_cnt, ctrl, total;
};

size_t a256(size_t x) { return (x + 255) / 256 * 256; }

// Private best costs: items x rows = S x (P x rows) < S x (n + P) floats.
Layout layout(int64_t n, int64_t k) {
  Layout L;
  const size_t S = size_t((n + kStrip - 1) / kStrip);
  size_t o = 0;
  L.bpriv = o;     o += a256(S * size_t(n + kMaxPanels) * 4);
  L.mask = o;      o += a256(size_t(n) * 4);
  L.partial = o;   o += a256(size_t(kMaxPanels) * size_t(n) * 8);
  L.strip_g = o;   o += a256(size_t(kMaxStrips) * 8);
  L.obj_part = o;  o += a256(size_t(kMaxPanels) * 8);
  L.key = o;       o += a256(size_t(k) * 8);
  L.strip_cnt = o; o += a256(size_t(kMaxStrips) * 4);
  L.ctrl = o;      o += 256;
  L.total = o;
  return L;
}

// The barrier waits for every wave's outstanding memory operations, so the
// block's device-scope stores are complete before thread 0 counts the block
// in.  Returns, block-uniformly, the counter value before this increment.
template <int BT>
__device__ unsigned int block_arrive(unsigned int* counter, unsigned int* s_prev) {
  __syncthreads();
  if (threadIdx.x == 0)
    *s_prev = __hip_atomic_fetch_add(counter, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  __syncthreads();
  return *s_prev;
}

template <int BT>
__device__ void block_argmax(double& g, int& i, double* sg, int* si) {
  constexpr int W = BT / 64;
  wave_argmax(g, i);
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  __syncthreads();
  if (lane == 0) {
    sg[w] = g;
    si[w] = i;
  }
  __syncthreads();
  if (threadIdx.x == 0)
    for (int x = 1; x < W; ++x)
      if (better(sg[x], si[x], g, i)) {
        g = sg[x];
        i = si[x];
      }
}

// Fixed-order block sum, result in thread 0.
template <int BT>
__device__ double block_sum(double x, double* sd) {
  constexpr int W = BT / 64;
  x = wave_sum(x);
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  __syncthreads();
  if (lane == 0) sd[w] = x;
  __syncthreads();
  double s = 0.0;
  if (threadIdx.x == 0)
    for (int q = 0; q < W; ++q) s += sd[q];
  return s;
}

__global__ void sgs_init_kernel(SgsDev a) {
  const int gt = blockIdx.x * blockDim.x + threadIdx.x, nt = gridDim.x * blockDim.x;
  for (int j = gt; j < a.n; j += nt) {
    a.mask[j] = 0u;
    if (a.assign) a.assign[j] = -1;
  }
  for (int s = gt; s < a.S; s += nt) a.strip_cnt[s] = 0u;
  for (int s = gt; s < a.k; s += nt) a.key[s] = 0ull;
  if (gt == 0) {
    *a.step_cnt = 0u;
    *a.fin_cnt = 0u;
    *a.abort = a.abort_init;
  }
}

__device__ __forceinline__ unsigned long long pack_key(double g, int idx) {
  const unsigned long long gb = (unsigned long long)__double_as_longlong(g) >> kIndexBits;
  return (gb << kIndexBits) | (kIndexMask - (unsigned long long)idx);
}

struct RowState {
  float bo, cv, vj;
};

// Row j entering step `step`: previous best cost, cost of the previous pick.
__device__ __forceinline__ RowState fetch_row(const SgsDev& a, const float* bp, int step, int tprev,
                                              int j, int j1) {
  RowState r{0.f, 0.f, 0.f};
  if (j < j1) {
    r.vj = a.v[j];
    if (step == 0) {
      r.bo = a.c0;
      r.cv = a.c0;
    } else {
      r.bo = bp[j];
      r.cv = a.C[size_t(j) * a.n + tprev];
    }
  }
  return r;
}

// Sweep of one item for one step.  Returns the panel's objective share in
// thread 0 for the strip-0 item.
template <int BT, bool VEC4>
__device__ double sweep_item(const SgsDev& a, int step, int tprev, int it, int panel, int strip,
                             float* sb, float* sv, double* red, double* sd) {
  constexpr int W = BT / 64;
  constexpr int U = 16;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int j0 = panel * a.rows, j1 = min(a.n, j0 + a.rows);
  float* bp = a.bpriv + size_t(it) * a.rows - j0;   // bp[j], j in [j0, j1)
  const int col = strip * kStrip + lane * 4;
  const bool owner = strip == 0;
  double g0 = 0.0, g1 = 0.0, g2 = 0.0, g3 = 0.0;
  double objp = 0.0;

  RowState next = fetch_row(a, bp, step, tprev, j0 + tid, j1);
  for (int c0 = j0; c0 < j1; c0 += BT) {
    const RowState cur = next;
    const int j = c0 + tid;
    float bn = 0.f;
    if (j < j1) {
      bn = fminf(cur.bo, cur.cv);
      bp[j] = bn;
      if (owner) {
        if (a.assign && step > 0 && cur.cv < cur.bo) a.assign[j] = tprev;
        objp = fma(double(cur.vj), double(bn), objp);
      }
    }
    sb[tid] = bn;
    sv[tid] = cur.vj;
    __syncthreads();
    if (c0 + BT < j1) next = fetch_row(a, bp, step, tprev, c0 + BT + tid, j1);

    // Wave w streams rows c0 + 64 w .. + 63 of the chunk.
    const int r0 = c0 + w * 64, r1 = min(j1, r0 + 64);
    if (VEC4) {
      if (col < a.n) {
        const float* base = a.C + col;
        int r = r0;
        for (; r + U <= r1; r += U) {
          f32x4 x[U];
#pragma unroll
          for (int u = 0; u < U; ++u)
            x[u] = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(base + size_t(r + u) * a.n));
#pragma unroll
          for (int u = 0; u < U; ++u) {
            const float bj = sb[r + u - c0];
            const double vj = double(sv[r + u - c0]);
            g0 = fma(vj, double(fmaxf(bj - x[u][0], 0.f)), g0);
            g1 = fma(vj, double(fmaxf(bj - x[u][1], 0.f)), g1);
            g2 = fma(vj, double(fmaxf(bj - x[u][2], 0.f)), g2);
            g3 = fma(vj, double(fmaxf(bj - x[u][3], 0.f)), g3);
          }
        }
        for (; r < r1; ++r) {
          const f32x4 x = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(base + size_t(r) * a.n));
          const float bj = sb[r - c0];
          const double vj = double(sv[r - c0]);
          g0 = fma(vj, double(fmaxf(bj - x[0], 0.f)), g0);
          g1 = fma(vj, double(fmaxf(bj - x[1], 0.f)), g1);
          g2 = fma(vj, double(fmaxf(bj - x[2], 0.f)), g2);
          g3 = fma(vj, double(fmaxf(bj - x[3], 0.f)), g3);
        }
      }
    } else {
      for (int r = r0; r < r1; ++r) {
        const float* row = a.C + size_t(r) * a.n;
        const float bj = sb[r - c0];
        const double vj = double(sv[r - c0]);
        if (col < a.n) g0 = fma(vj, double(fmaxf(bj - row[col], 0.f)), g0);
        if (col + 1 < a.n) g1 = fma(vj, double(fmaxf(bj - row[col + 1], 0.f)), g1);
        if (col + 2 < a.n) g2 = fma(vj, double(fmaxf(bj - row[col + 2], 0.f)), g2);
        if (col + 3 < a.n) g3 = fma(vj, double(fmaxf(bj - row[col + 3], 0.f)), g3);
      }
    }
    __syncthreads();
  }

  // The waves' partial gains, summed in wave order: thread c < 256 owns column c.
  red[(w * 64 + lane) * 4 + 0] = g0;
  red[(w * 64 + lane) * 4 + 1] = g1;
  red[(w * 64 + lane) * 4 + 2] = g2;
  red[(w * 64 + lane) * 4 + 3] = g3;
  __syncthreads();
  if (tid < kStrip) {
    const int cc = strip * kStrip + tid;
    if (cc < a.n) {
      const int l = tid >> 2, q = tid & 3;
      double s = 0.0;
#pragma unroll
      for (int x = 0; x < W; ++x) s += red[(x * 64 + l) * 4 + q];
      put(a.partial + size_t(panel) * a.n + cc, s);
    }
  }
  return owner ? block_sum<BT>(objp, sd) : 0.0;
}

template <int BT, bool VEC4>
__global__ __launch_bounds__(BT) void sgs_dense_kernel(SgsDev a) {
  constexpr int W = BT / 64;
  const int tid = threadIdx.x;
  __shared__ float sb[BT], sv[BT];
  __shared__ double red[BT * 4];
  __shared__ double sd[W];
  __shared__ int si[W];
  __shared__ unsigned int s_prev;
  __shared__ int s_t;

  const int items = a.P * a.S;
  int tprev = -1;
  for (int step = 0; step < a.k; ++step) {
    for (int it = blockIdx.x; it < items; it += gridDim.x) {
      const int panel = it / a.S, strip = it - panel * a.S;
      const double objp = sweep_item<BT, VEC4>(a, step, tprev, it, panel, strip, sb, sv, red, sd);
      if (strip == 0 && tid == 0) put(a.obj_part + panel, objp);

      const unsigned int prev = block_arrive<BT>(a.strip_cnt + strip, &s_prev);
      if (prev != unsigned(step + 1) * unsigned(a.P) - 1u) continue;
      // Last block of the strip.
      double g = -1.0;
      int gi = INT_MAX;
      if (tid < kStrip) {
        const int cc = strip * kStrip + tid;
        if (cc < a.n && !get(a.mask + cc)) {
          g = 0.0;
          for (int p = 0; p < a.P; ++p) g += get(a.partial + size_t(p) * a.n + cc);
          gi = cc;
        }
      }
      block_argmax<BT>(g, gi, sd, si);
      double prev_obj = 0.0;
      if (strip == 0 && step > 0) {
        double x = 0.0;
        for (int p = tid; p < a.P; p += BT) x += get(a.obj_part + p);
        prev_obj = block_sum<BT>(x, sd);
      }
      if (tid == 0) {
        put(a.strip_g + strip, g);
        if (gi != INT_MAX)
          __hip_atomic_fetch_max(a.key + step, pack_key(g, gi), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (strip == 0 && step > 0 && a.step_obj) a.step_obj[step - 1] = prev_obj;
      }
      block_arrive<BT>(a.step_cnt, &s_prev);
    }
    // Wait until every strip has reported, then read the winner; -1 when the
    // wait gave up, and the block leaves the loop.
    if (tid == 0) {
      const unsigned int target = unsigned(step + 1) * unsigned(a.S);
      bool ok = true;
      for (unsigned int spins = 0; get(a.step_cnt) < target; ++spins) {
        if (give_up(spins, a.poll_limit, a.abort)) {
          ok = false;
          break;
        }
        __builtin_amdgcn_s_sleep(1);
      }
      int t = -1;
      if (ok) {
        const unsigned long long kk = __hip_atomic_load(a.key + step, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        t = int(kIndexMask - (kk & kIndexMask));
        const int ts = t / kStrip;
        if (int(blockIdx.x) == ts % int(gridDim.x)) put(a.mask + t, 1u);   // owner of item (0, ts)
        if (blockIdx.x == 0) {
          a.selected[step] = t;
          if (a.step_gain) a.step_gain[step] = get(a.strip_g + ts);
        }
      }
      s_t = t;
    }
    __syncthreads();
    tprev = s_t;
    if (tprev < 0) break;
  }

  // Apply the last pick: assignment and the final objective (not when the
  // launch gave up; tprev is the same in every thread of the block).
  for (int it = blockIdx.x; tprev >= 0 && it < items; it += gridDim.x) {
    const int panel = it / a.S, strip = it - panel * a.S;
    if (strip != 0) continue;
    const int j0 = panel * a.rows, j1 = min(a.n, j0 + a.rows);
    const float* bp = a.bpriv + size_t(it) * a.rows - j0;
    double objp = 0.0;
    for (int j = j0 + tid; j < j1; j += BT) {
      const float bo = bp[j];
      const float cv = a.C[size_t(j) * a.n + tprev];
      if (a.assign && cv < bo) a.assign[j] = tprev;
      objp = fma(double(a.v[j]), double(fminf(bo, cv)), objp);
    }
    const double s = block_sum<BT>(objp, sd);
    if (tid == 0) put(a.obj_part + panel, s);
  }
  const unsigned int fprev = block_arrive<BT>(a.fin_cnt, &s_prev);
  if (fprev == gridDim.x - 1u && a.step_obj && !get(a.abort)) {
    double x = 0.0;
    for (int p = tid; p < a.P; p += BT) x += get(a.obj_part + p);
    const double s = block_sum<BT>(x, sd);
    if (tid == 0) a.step_obj[a.k - 1] = s;
  }
}

constexpr int kBlock = 256;

template <bool VEC4>
hipError_t max_coresident(int& blocks) {
  int dev = 0, cus = 0, per_cu = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if ((e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev)) != hipSuccess) return e;
  e = hipOccupancyMaxActiveBlocksPerMultiprocessor(
      &per_cu, reinterpret_cast<const void*>(sgs_dense_kernel<kBlock, VEC4>), kBlock, 0);
  // Two blocks (8 waves) per CU: enough loads in flight to saturate HBM while
  // keeping the per-step arrivals few.
  blocks = std::max(1, cus * std::min(per_cu, 2));
  return e;
}

}  // namespace

size_t sgs_workspace_bytes(int64_t n, int64_t k) { return layout(n, k).total; }

hipError_t launch_sgs_dense(const SgsParams& p, hipStream_t stream) {
  const bool vec4 = (p.n % 4) == 0;
  int max_blocks = 0;
  hipError_t e = vec4 ? max_coresident<true>(max_blocks) : max_coresident<false>(max_blocks);
  if (e != hipSuccess) return e;
  const int n = p.n;
  const int S = (n + kStrip - 1) / kStrip;
  int P = std::max(1, max_blocks / S);
  P = std::min(P, kMaxPanels);
  P = std::min(P, std::max(1, n / kMinPanelRows));
  const int rows = (n + P - 1) / P;
  const int grid = std::min(P * S, max_blocks);

  const Layout L = layout(n, p.k);
  char* w = static_cast<char*>(p.workspace);
  SgsDev a{};
  a.C = p.cost;
  a.v = p.capacity;
  a.n = n;
  a.k = p.k;
  a.c0 = p.c0;
  a.selected = p.selected;
  a.step_gain = p.step_gain;
  a.step_obj = p.step_objective;
  a.assign = p.assign;
  a.bpriv = reinterpret_cast<float*>(w + L.bpriv);
  a.mask = reinterpret_cast<unsigned int*>(w + L.mask);
  a.partial = reinterpret_cast<double*>(w + L.partial);
  a.strip_g = reinterpret_cast<double*>(w + L.strip_g);
  a.obj_part = reinterpret_cast<double*>(w + L.obj_part);
  a.key = reinterpret_cast<unsigned long long*>(w + L.key);
  a.strip_cnt = reinterpret_cast<unsigned int*>(w + L.strip_cnt);
  a.step_cnt = reinterpret_cast<unsigned int*>(w + L.ctrl);
  a.fin_cnt = reinterpret_cast<unsigned int*>(w + L.ctrl + 4);
  a.abort = reinterpret_cast<unsigned int*>(w + L.ctrl + 8);
  const WaitPolicy wp = wait_policy();
  a.poll_limit = wp.limit;
  a.abort_init = wp.preset;
  a.P = P;
  a.S = S;
  a.rows = rows;

  sgs_init_kernel<<<std::min(1024, (std::max(n, p.k) + 255) / 256), 256, 0, stream>>>(a);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  void* args[] = {&a};
  const void* fn = vec4 ? reinterpret_cast<const void*>(sgs_dense_kernel<kBlock, true>)
                        : reinterpret_cast<const void*>(sgs_dense_kernel<kBlock, false>);
  if ((e = hipLaunchCooperativeKernel(fn, dim3(grid), dim3(kBlock), args, 0, stream)) != hipSuccess) return e;
  return launch_mark_aborted(a.abort, a.selected, a.k, stream);
}

}  // namespace cp
