// Greedy coverage selection over the target-major cost (Sec. 3.5, Eq. 14-16).
//
// State: b_j, the best cost at which target j is covered so far (c0 while
// uncovered), and the mask of chosen tokens.  One step:
//   S  sweep    gain(c) = sum_j v_j max(0, b_j - C_tm[j][c]) for every c: a
//               column reduction of the N x N matrix, streamed row by row
//               (each row is one target; a wave reads 1 KB of it per load);
//               waves own (row chunk, 256-column strip) items and write
//               float64 partial gains per row chunk
//   R  argmax   partials summed per column in a fixed order, masked, argmax
//               with ties to the smaller index; the last block to finish
//               publishes the step's winner t*
//   U  update   b_j = min(b_j, C_tm[j][t*]); assign_j = t* on strict
//               improvement; L = sum_j v_j b_j folded per block
// The K steps run inside one cooperative launch; grid barriers separate the
// phases, so the greedy never returns to the host.
#include <hip/hip_runtime.h>
#include <hip/hip_cooperative_groups.h>

#include <algorithm>
#include <climits>

#include "common.h"
#include "launch.h"

namespace cg = cooperative_groups;

namespace cp {
namespace {

constexpr int kThreads = 256;
constexpr int kStrip = 256;        // columns per wave item: 64 lanes x 4 floats
constexpr int kMaxChunks = 64;     // row chunks (partial-gain rows)
constexpr int kMaxBlocks = 4096;
constexpr int kMinRowsPerChunk = 16;

struct SgsDev {
  const float* C;
  const float* v;
  int n, k;
  float c0;
  int32_t* selected;
  double* step_gain;
  double* step_obj;
  int32_t* assign;
  float* b;
  uint8_t* mask;
  double* partial;     // [nrc][n]
  double* bbest_g;     // [grid]
  int* bbest_i;        // [grid]
  double* obj_part;    // [grid]
  unsigned int* counter;
  int* tstar;
  int ncs, nrc, rows;  // column strips, row chunks, rows per chunk
};

struct Layout {
  size_t b, mask, partial, bbest_g, bbest_i, obj_part, ctrl, total;
};

size_t a256(size_t x) { return (x + 255) / 256 * 256; }

Layout layout(int64_t n) {
  Layout L;
  size_t o = 0;
  L.b = o;        o += a256(size_t(n) * 4);
  L.mask = o;     o += a256(size_t(n));
  L.partial = o;  o += a256(size_t(kMaxChunks) * size_t(n) * 8);
  L.bbest_g = o;  o += a256(size_t(kMaxBlocks) * 8);
  L.bbest_i = o;  o += a256(size_t(kMaxBlocks) * 4);
  L.obj_part = o; o += a256(size_t(kMaxBlocks) * 8);
  L.ctrl = o;     o += 256;
  L.total = o;
  return L;
}

// Block-wide reduction of per-thread (gain, index) to thread 0.
__device__ void block_argmax(double& g, int& i, double* sg, int* si) {
  wave_argmax(g, i);
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  __syncthreads();
  if (lane == 0) {
    sg[w] = g;
    si[w] = i;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int x = 1; x < kThreads / 64; ++x)
      if (better(sg[x], si[x], g, i)) {
        g = sg[x];
        i = si[x];
      }
  }
}

// Block-wide float64 sum in a fixed order, result in thread 0.
__device__ double block_sum(double x, double* sd) {
  x = wave_sum(x);
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  __syncthreads();
  if (lane == 0) sd[w] = x;
  __syncthreads();
  double s = 0.0;
  if (threadIdx.x == 0)
    for (int q = 0; q < kThreads / 64; ++q) s += sd[q];
  return s;
}

__device__ __forceinline__ void sweep_item(const SgsDev& a, int it, int lane) {
  const int r = it / a.ncs, strip = it - r * a.ncs;
  const int col = strip * kStrip + lane * 4;
  const int j0 = r * a.rows, j1 = min(a.n, j0 + a.rows);
  double g0 = 0.0, g1 = 0.0, g2 = 0.0, g3 = 0.0;
  const bool full = (a.n & 3) == 0 && col + 3 < a.n;
  if (full) {
    const float* base = a.C + col;
    int j = j0;
    for (; j + 4 <= j1; j += 4) {
      f32x4 x[4];
#pragma unroll
      for (int u = 0; u < 4; ++u)
        x[u] = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(base + size_t(j + u) * a.n));
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const float bj = a.b[j + u];
        const double vj = double(a.v[j + u]);
        g0 = fma(vj, double(fmaxf(bj - x[u][0], 0.f)), g0);
        g1 = fma(vj, double(fmaxf(bj - x[u][1], 0.f)), g1);
        g2 = fma(vj, double(fmaxf(bj - x[u][2], 0.f)), g2);
        g3 = fma(vj, double(fmaxf(bj - x[u][3], 0.f)), g3);
      }
    }
    for (; j < j1; ++j) {
      const f32x4 x = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(base + size_t(j) * a.n));
      const float bj = a.b[j];
      const double vj = double(a.v[j]);
      g0 = fma(vj, double(fmaxf(bj - x[0], 0.f)), g0);
      g1 = fma(vj, double(fmaxf(bj - x[1], 0.f)), g1);
      g2 = fma(vj, double(fmaxf(bj - x[2], 0.f)), g2);
      g3 = fma(vj, double(fmaxf(bj - x[3], 0.f)), g3);
    }
  } else {
    double g[4] = {0.0, 0.0, 0.0, 0.0};
    for (int j = j0; j < j1; ++j) {
      const float bj = a.b[j];
      const double vj = double(a.v[j]);
      const float* row = a.C + size_t(j) * a.n;
#pragma unroll
      for (int q = 0; q < 4; ++q)
        if (col + q < a.n) g[q] = fma(vj, double(fmaxf(bj - row[col + q], 0.f)), g[q]);
    }
    g0 = g[0]; g1 = g[1]; g2 = g[2]; g3 = g[3];
  }
  double* out = a.partial + size_t(r) * a.n + col;
  if (col < a.n) out[0] = g0;
  if (col + 1 < a.n) out[1] = g1;
  if (col + 2 < a.n) out[2] = g2;
  if (col + 3 < a.n) out[3] = g3;
}

__global__ __launch_bounds__(kThreads) void sgs_dense_kernel(SgsDev a) {
  cg::grid_group grid = cg::this_grid();
  const int tid = threadIdx.x, lane = tid & 63;
  const int gw = blockIdx.x * (kThreads / 64) + (tid >> 6), nw = gridDim.x * (kThreads / 64);
  const int gt = blockIdx.x * kThreads + tid, nt = gridDim.x * kThreads;
  __shared__ double sg[kThreads / 64];
  __shared__ int si[kThreads / 64];
  __shared__ int s_last;

  for (int j = gt; j < a.n; j += nt) {
    a.b[j] = a.c0;
    a.mask[j] = 0;
    if (a.assign) a.assign[j] = -1;
  }
  if (gt == 0) *a.counter = 0u;
  grid.sync();

  const int items = a.ncs * a.nrc;
  for (int step = 0; step < a.k; ++step) {
    // S: partial gains.
    for (int it = gw; it < items; it += nw) sweep_item(a, it, lane);
    grid.sync();

    // R: per-column totals, block argmax, last block -> global argmax.
    double bg = -1.0;
    int bi = INT_MAX;
    for (int c = gt; c < a.n; c += nt) {
      if (a.mask[c]) continue;
      double g = 0.0;
      for (int r = 0; r < a.nrc; ++r) g += a.partial[size_t(r) * a.n + c];
      if (better(g, c, bg, bi)) {
        bg = g;
        bi = c;
      }
    }
    block_argmax(bg, bi, sg, si);
    if (tid == 0) {
      a.bbest_g[blockIdx.x] = bg;
      a.bbest_i[blockIdx.x] = bi;
      __threadfence();
      const unsigned int prev = atomicAdd(a.counter, 1u);
      s_last = prev == unsigned(step + 1) * gridDim.x - 1u;
    }
    __syncthreads();
    if (s_last) {
      __threadfence();
      double g = -1.0;
      int i = INT_MAX;
      for (int x = tid; x < int(gridDim.x); x += kThreads)
        if (better(a.bbest_g[x], a.bbest_i[x], g, i)) {
          g = a.bbest_g[x];
          i = a.bbest_i[x];
        }
      block_argmax(g, i, sg, si);
      double prev_obj = 0.0;
      if (step > 0 && a.step_obj) {
        double x = 0.0;
        for (int q = tid; q < int(gridDim.x); q += kThreads) x += a.obj_part[q];
        prev_obj = block_sum(x, sg);
      }
      if (tid == 0) {
        *a.tstar = i;
        a.selected[step] = i;
        if (a.step_gain) a.step_gain[step] = g;
        if (step > 0 && a.step_obj) a.step_obj[step - 1] = prev_obj;
        a.mask[i] = 1;
      }
    }
    grid.sync();

    // U: best-cost update and this step's objective share.
    const int t = *a.tstar;
    double part = 0.0;
    for (int j = gt; j < a.n; j += nt) {
      const float c = a.C[size_t(j) * a.n + t];
      float bj = a.b[j];
      if (c < bj) {
        bj = c;
        a.b[j] = c;
        if (a.assign) a.assign[j] = t;
      }
      part = fma(double(a.v[j]), double(bj), part);
    }
    const double bs = block_sum(part, sg);
    if (tid == 0) a.obj_part[blockIdx.x] = bs;
    grid.sync();
  }
  if (blockIdx.x == 0 && a.step_obj) {
    double x = 0.0;
    for (int q = tid; q < int(gridDim.x); q += kThreads) x += a.obj_part[q];
    const double s = block_sum(x, sg);
    if (tid == 0) a.step_obj[a.k - 1] = s;
  }
}

struct DeviceInfo {
  int cus = 0;
  int blocks_per_cu = 0;
};

hipError_t device_info(DeviceInfo& info) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if ((e = hipDeviceGetAttribute(&info.cus, hipDeviceAttributeMultiprocessorCount, dev)) != hipSuccess) return e;
  return hipOccupancyMaxActiveBlocksPerMultiprocessor(&info.blocks_per_cu,
                                                      reinterpret_cast<const void*>(sgs_dense_kernel),
                                                      kThreads, 0);
}

}  // namespace

size_t sgs_workspace_bytes(int64_t n) { return layout(n).total; }

hipError_t launch_sgs_dense(const SgsParams& p, hipStream_t stream) {
  DeviceInfo info;
  hipError_t e = device_info(info);
  if (e != hipSuccess) return e;
  const int64_t n = p.n;
  const int max_blocks = std::min(kMaxBlocks, info.cus * std::min(info.blocks_per_cu, 4));
  // Aim for at least 64 KB of the matrix per wave per step.
  const int64_t waves_wanted = std::max<int64_t>(1, (4 * n * n + 65535) / 65536);
  const int grid = int(std::max<int64_t>(1, std::min<int64_t>(max_blocks, (waves_wanted + 3) / 4)));
  const int ncs = int((n + kStrip - 1) / kStrip);
  int nrc = std::max(1, (grid * (kThreads / 64)) / ncs);
  nrc = std::min<int>(nrc, kMaxChunks);
  nrc = std::min<int>(nrc, int(std::max<int64_t>(1, n / kMinRowsPerChunk)));
  const int rows = int((n + nrc - 1) / nrc);

  const Layout L = layout(n);
  char* w = static_cast<char*>(p.workspace);
  SgsDev a;
  a.C = p.cost;
  a.v = p.capacity;
  a.n = p.n;
  a.k = p.k;
  a.c0 = p.c0;
  a.selected = p.selected;
  a.step_gain = p.step_gain;
  a.step_obj = p.step_objective;
  a.assign = p.assign;
  a.b = reinterpret_cast<float*>(w + L.b);
  a.mask = reinterpret_cast<uint8_t*>(w + L.mask);
  a.partial = reinterpret_cast<double*>(w + L.partial);
  a.bbest_g = reinterpret_cast<double*>(w + L.bbest_g);
  a.bbest_i = reinterpret_cast<int*>(w + L.bbest_i);
  a.obj_part = reinterpret_cast<double*>(w + L.obj_part);
  a.counter = reinterpret_cast<unsigned int*>(w + L.ctrl);
  a.tstar = reinterpret_cast<int*>(w + L.ctrl + 4);
  a.ncs = ncs;
  a.nrc = nrc;
  a.rows = rows;
  void* args[] = {&a};
  return hipLaunchCooperativeKernel(reinterpret_cast<const void*>(sgs_dense_kernel), dim3(grid),
                                    dim3(kThreads), args, 0, stream);
}

}  // namespace cp
