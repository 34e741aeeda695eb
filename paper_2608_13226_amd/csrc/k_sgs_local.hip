// Greedy coverage selection, spatially local form (Sec. 3.5, Eq. 13-16).
//
// A candidate's gain runs over its neighbour set only,
//   gain(c) = sum_{j in M_g(c)} v_j max(0, b_j - C(c, j)),
// while a pick still lowers the best cost b_j of every target it is cheaper
// for (the residual of Eq. 14 is over all targets) and L(S) sums over all of
// them.  One cooperative launch of one block per compute unit; block b owns
// candidates [b W, (b + 1) W).  Every block keeps all n best costs in LDS,
// together with its candidates' neighbour lists, the costs C(c, j) and the
// capacities v_j of those neighbours (read once at launch), and per step:
//   1. reads every block's candidate and takes the same winner t;
//   2. reads the winner's costs to every target, C(t, j) for all j, as one
//      contiguous row of a source-major copy T of the cost (written by a
//      transposing kernel before the launch), and lowers b_j wherever the
//      winner is cheaper: every block holds the identical b afterwards, and
//      no block exchanges anything but its candidate;
//   3. sums its candidates' local gains afresh from LDS: lanes over
//      candidates, waves over the neighbour list, each term the float64
//      difference b_j - C(c, j) times v_j rounded onto the fixed-point grid;
//   4. publishes the exact argmax of its unchosen candidates.
// L(S) is kept in the same fixed point as one running part per block over
// the block's own targets, stored for every step and added up in block order
// by a second kernel.  n <= kLocalMaxN, g <= kLocalMaxG.
//
// The candidate exchange and the fixed point are in sgs_exchange.h.
#include <hip/hip_runtime.h>

#include <algorithm>

#include "sgs_exchange.h"

namespace cp {
namespace {

constexpr int kLocalMaxN = 16384;
constexpr int kLocalMaxG = 128;
constexpr int kChunkT = 256;                          // targets per wave-load of the winner's row
constexpr int kLoadsT = kLocalMaxN / kChunkT / kWaves;  // such loads per wave and step
constexpr int kTile = 64;                             // transposing kernel's tile

int local_ldt(int64_t n) { return int((n + kChunkT - 1) / kChunkT * kChunkT); }

// T[s][j] = C_tm[j][s] through a 64 x 65 LDS tile: coalesced reads along s,
// coalesced writes along j.  Row padding [n, ldt) is left as it is.
__global__ __launch_bounds__(256) void transpose_kernel(const float* __restrict__ C, int n, float* __restrict__ T,
                                                        int ldt) {
  __shared__ float tile[kTile][kTile + 1];
  const int tj = blockIdx.y * kTile, ts = blockIdx.x * kTile;
  const int c = threadIdx.x & 63, r0 = threadIdx.x >> 6;
#pragma unroll 4
  for (int r = r0; r < kTile; r += 4) {
    const int j = tj + r, s = ts + c;
    if (j < n && s < n) tile[r][c] = C[size_t(j) * n + s];
  }
  __syncthreads();
#pragma unroll 4
  for (int r = r0; r < kTile; r += 4) {
    const int s = ts + r, j = tj + c;
    if (s < n && j < n) T[size_t(s) * ldt + j] = tile[c][r];
  }
}

struct LocalDev {
  IncDev a;
  const int32_t* nbr;
  int g;
  long long* part;     // [k][blocks] running objective part of each block after each step
  int* scale;          // the fixed-point exponent S, for the objective sums
};

__global__ __launch_bounds__(kBlock) void sgs_local_kernel(LocalDev L) {
  const IncDev& a = L.a;
  const int g = L.g;
  extern __shared__ unsigned long long smem[];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int blk = blockIdx.x, nb = gridDim.x;
  const int lo = blk * a.W;
  const int cnt = max(0, min(a.n, lo + a.W) - lo);
  long long* sG = reinterpret_cast<long long*>(smem);             // [W] gains (W rounded up to even)
  float* sball = reinterpret_cast<float*>(sG + ((a.W + 1) & ~1));  // [ldt] b_j, 16-byte aligned; -inf past n
  // The band, neighbour-major ([g][W]: entry q of candidate i at q W + i),
  // so that the lanes of a wave (consecutive candidates) read consecutive
  // words.
  float* scg = sball + a.ldt;                                      // [g][W] C(c, j), j in M_g(c)
  float* snv = scg + size_t(a.W) * g;                              // [g][W] v_j, j in M_g(c)
  float* sv = snv + size_t(a.W) * g;                               // [W] v of the own targets
  unsigned short* snb = reinterpret_cast<unsigned short*>(sv + a.W);   // [g][W] M_g(c)
  unsigned char* ssel = reinterpret_cast<unsigned char*>(snb + size_t(a.W) * g);   // [W]
  __shared__ long long red[kBlock];
  __shared__ long long sg[kWaves];
  __shared__ double sd[kWaves];
  __shared__ int si[kWaves];
  __shared__ unsigned long long su[kWaves];
  __shared__ int sflag;
  __shared__ long long sLw[kWaves];            // this block's objective part, one running share per wave

  for (int j = tid; j < a.ldt; j += kBlock) sball[j] = j < a.n ? a.c0 : -__builtin_inff();
  for (int i = tid; i < cnt; i += kBlock) {
    ssel[i] = 0;
    sv[i] = a.v[lo + i];
  }
  // The band of the own candidates: neighbour lists, C(c, j) = C_tm[j][c]
  // and v_j (indices clamped into range; the table is the caller's).
  for (int e = tid; e < cnt * g; e += kBlock) {
    const int i = e / g, q = e - i * g;
    const int j = min(max(L.nbr[size_t(lo + i) * g + q], 0), a.n - 1);
    const int at = q * a.W + i;
    snb[at] = (unsigned short)j;
    scg[at] = a.C[size_t(j) * a.n + lo + i];
    snv[at] = a.v[j];
  }

  // Fixed-point scale, the same in every block (same sum, same order).
  double vsum;
  {
    // Thread t adds v[t], v[t + kBlock], ... in that order, eight loads in
    // flight at a time.
    double x = 0.0;
    constexpr int U = 8;
    for (int j0 = tid; j0 < a.n; j0 += kBlock * U) {
      float vv[U];
#pragma unroll
      for (int u = 0; u < U; ++u) vv[u] = a.v[min(j0 + u * kBlock, a.n - 1)];
#pragma unroll
      for (int u = 0; u < U; ++u)
        if (j0 + u * kBlock < a.n) x += double(vv[u]);
    }
    vsum = block_sum_all(x, sd);
  }
  const double M = double(a.c0) * vsum;
  int S = 0;
  if (M > 0.0) {
    int e = 0;
    (void)__builtin_frexp(M, &e);
    S = 62 - e;
  }
  if (blk == 0 && tid == 0) *L.scale = S;

  // The objective part of the own targets at b = c0.
  {
    long long x = 0;
    for (int i = tid; i < cnt; i += kBlock) x += fx(double(sv[i]) * double(a.c0), S);
    const long long P0 = block_sum_i64(x, sg);
    if (tid < kWaves) sLw[tid] = tid == 0 ? P0 : 0;
  }

  // Local gains of the own candidates from the current best costs: lane =
  // candidate within a chunk of 64, waves split the neighbour list.
  const int qper = (g + kWaves - 1) / kWaves;
  auto local_gains = [&]() {
    for (int cc = 0; cc < cnt; cc += 64) {
      const int i = cc + lane;
      // Four neighbours at a time: their LDS reads are issued together
      // (index, then best cost) before the terms are formed.
      long long g0 = 0, g1 = 0;
      if (i < cnt) {
        const int q1 = min(g, (w + 1) * qper);
        for (int q = w * qper; q < q1; q += 4) {
          int jj[4];
          float cg[4], nv[4], bj[4];
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            const int e = min(q + u, q1 - 1) * a.W + i;
            jj[u] = snb[e];
            cg[u] = scg[e];
            nv[u] = snv[e];
          }
#pragma unroll
          for (int u = 0; u < 4; ++u) bj[u] = sball[jj[u]];
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            const double d = double(bj[u]) - double(cg[u]);
            if (q + u < q1 && d > 0.0) {
              if (u & 1) g1 += fx(double(nv[u]) * d, S);
              else g0 += fx(double(nv[u]) * d, S);
            }
          }
        }
      }
      red[tid] = g0 + g1;
      __syncthreads();
      if (tid < 64 && cc + tid < cnt) {
        long long s = 0;
#pragma unroll
        for (int q = 0; q < kWaves; ++q) s += red[q * 64 + tid];
        sG[cc + tid] = s;
      }
      __syncthreads();
    }
  };

  __syncthreads();
  local_gains();
  publish_argmax(sG, ssel, lo, cnt, S, cand_slot(a.cand, 0, blk), epoch_of(0), sg, si);

  const int nch = a.ldt / kChunkT;
  for (int step = 0; step < a.k; ++step) {
    const int tw = read_winner(cand_slot(a.cand, step & 1, 0), epoch_of(step), nb, a.abort, a.poll_limit, su, &sflag);
    if (tw < 0) break;
    const int t = min(tw, a.n - 1);
    if (t >= lo && t < lo + cnt && tid == 0) {
      ssel[t - lo] = 1;
      a.selected[step] = t;
      if (a.step_gain) a.step_gain[step] = fx_to_double(sG[t - lo], S);
    }

    // 2. The winner's row against b, the wave's chunks loaded together; each
    // lane lowers its own four targets, and the own targets' changes enter
    // assign and the block's objective part.
    const f32x4* row = reinterpret_cast<const f32x4*>(a.T + size_t(t) * a.ldt);
    f32x4 xr[kLoadsT];
#pragma unroll
    for (int i = 0; i < kLoadsT; ++i)
      if (w + i * kWaves < nch) xr[i] = row[(w + i * kWaves) * (kChunkT / 4) + lane];
    long long dobj = 0;
#pragma unroll
    for (int i = 0; i < kLoadsT; ++i) {
      const int q0 = w + i * kWaves;
      if (q0 < nch) {
        const int j0 = q0 * kChunkT + 4 * lane;
        f32x4 b = *reinterpret_cast<const f32x4*>(sball + j0);
        const f32x4 x = xr[i];
        const bool any = x[0] < b[0] || x[1] < b[1] || x[2] < b[2] || x[3] < b[3];
        if (any) {
#pragma unroll
          for (int c = 0; c < 4; ++c) {
            if (x[c] < b[c]) {
              const int j = j0 + c;
              if (unsigned(j - lo) < unsigned(cnt)) {
                if (a.assign) a.assign[j] = t;
                const double vj = double(sv[j - lo]);
                dobj += fx(vj * double(x[c]), S) - fx(vj * double(b[c]), S);
              }
              b[c] = x[c];
            }
          }
          *reinterpret_cast<f32x4*>(sball + j0) = b;
        }
      }
    }
    dobj = wave_sum_i64(dobj);
    if (lane == 0) sLw[w] += dobj;
    __syncthreads();
    if (tid == 0 && L.part) {
      long long P = 0;
#pragma unroll
      for (int q = 0; q < kWaves; ++q) P += sLw[q];
      L.part[size_t(step) * nb + blk] = P;
    }

    // 3-4. Fresh local gains and this block's candidate for the next step.
    if (step + 1 < a.k) {
      local_gains();
      publish_argmax(sG, ssel, lo, cnt, S, cand_slot(a.cand, (step + 1) & 1, blk),
                     epoch_of(step + 1), sg, si);
    }
  }
}

// L(S) after step l: the blocks' parts added in block order.
__global__ void local_objective_kernel(const long long* part, int nb, int k, const int* scale, double* out) {
  const int l = blockIdx.x * blockDim.x + threadIdx.x;
  if (l >= k) return;
  long long s = 0;
  for (int b = 0; b < nb; ++b) s += part[size_t(l) * nb + b];
  out[l] = fx_to_double(s, *scale);
}

// Exchange slots, then the objective parts (k x kMaxBlocks), the scale, and T.
struct LocalLayout {
  size_t part, scale, T, total;
};
LocalLayout local_layout(int64_t n, int64_t k) {
  LocalLayout L;
  size_t o = layout(n, k).total;
  L.part = o; o += a256(size_t(k) * kMaxBlocks * sizeof(long long));
  L.scale = o; o += 256;
  L.T = o; o += a256(size_t(n) * local_ldt(n) * sizeof(float));
  L.total = o;
  return L;
}

}  // namespace

size_t sgs_local_workspace_bytes(int64_t n, int64_t k) { return local_layout(n, k).total; }

hipError_t launch_sgs_local(const SgsParams& p, const int32_t* nbr, int g, hipStream_t stream) {
  if (p.n < 1 || p.n > kLocalMaxN || g < 1 || g > p.n || g > kLocalMaxG) return hipErrorInvalidValue;
  int dev = 0, cus = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if ((e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev)) != hipSuccess) return e;
  const int nb = blocks_for(p.n, cus);
  const int W = (p.n + nb - 1) / nb;
  const int ldt = local_ldt(p.n);
  const size_t lds = size_t((W + 1) & ~1) * 8 + size_t(ldt) * 4 + size_t(W) * g * (4 + 4 + 2) + size_t(W) * (4 + 1) + 16;
  if ((e = hipFuncSetAttribute(reinterpret_cast<const void*>(sgs_local_kernel),
                               hipFuncAttributeMaxDynamicSharedMemorySize, int(lds))) != hipSuccess)
    return e;
  int per_cu = 0;
  if ((e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, reinterpret_cast<const void*>(sgs_local_kernel),
                                                        kBlock, lds)) != hipSuccess)
    return e;
  if (per_cu < 1) return hipErrorCooperativeLaunchTooLarge;

  const Layout X = layout(p.n, p.k);
  const LocalLayout Y = local_layout(p.n, p.k);
  char* w = static_cast<char*>(p.workspace);
  LocalDev d{};   // value-initialised: fields this launcher does not set stay null
  IncDev& a = d.a;
  a.C = p.cost;
  a.v = p.capacity;
  a.n = p.n;
  a.k = p.k;
  a.c0 = p.c0;
  a.selected = p.selected;
  a.step_gain = p.step_gain;
  a.step_obj = p.step_objective;
  a.assign = p.assign;
  a.list = reinterpret_cast<unsigned long long*>(w + X.list);
  a.lens = reinterpret_cast<unsigned long long*>(w + X.lens);
  a.cand = reinterpret_cast<unsigned long long*>(w + X.cand);
  a.abort = reinterpret_cast<unsigned int*>(w + X.ctrl);
  const WaitPolicy wp = wait_policy();
  a.poll_limit = wp.limit;
  a.abort_init = wp.preset;
  a.W = W;
  a.w_magic = w_magic_of(W);
  a.T = reinterpret_cast<float*>(w + Y.T);
  a.ldt = ldt;
  d.nbr = nbr;
  d.g = g;
  d.part = p.step_objective ? reinterpret_cast<long long*>(w + Y.part) : nullptr;
  d.scale = reinterpret_cast<int*>(w + Y.scale);

  sgs_inc_init_kernel<<<std::min(1024, (std::max(p.n, p.k) + 255) / 256), 256, 0, stream>>>(a);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  const int tiles = (p.n + kTile - 1) / kTile;
  transpose_kernel<<<dim3(tiles, tiles), 256, 0, stream>>>(p.cost, p.n, a.T, ldt);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  void* args[] = {&d};
  if ((e = hipLaunchCooperativeKernel(reinterpret_cast<const void*>(sgs_local_kernel), dim3(nb), dim3(kBlock), args,
                                      lds, stream)) != hipSuccess)
    return e;
  if ((e = launch_mark_aborted(a.abort, a.selected, a.k, stream)) != hipSuccess) return e;
  if (p.step_objective) {
    local_objective_kernel<<<(p.k + 255) / 256, 256, 0, stream>>>(d.part, nb, p.k, d.scale, p.step_objective);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace cp
