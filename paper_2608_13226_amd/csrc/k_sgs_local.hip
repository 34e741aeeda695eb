// Greedy coverage selection, spatially local form (Sec. 3.5, Eq. 13-16).
//
// A candidate's gain runs over its neighbour set only,
//   gain(c) = sum_{j in M_g(c)} v_j max(0, b_j - C(c, j)),
// while a pick still lowers the best cost b_j of every target it is cheaper
// for (the residual of Eq. 14 is over all targets) and L(S) sums over all of
// them.  The pick exchange and the change lists are the incremental form's.
// Every block keeps all n best costs in LDS, updated from the whole change
// list each step, together with its candidates' neighbour lists and costs
// C(c, j), j in M_g(c) (read once at launch), and sums its candidates' local
// gains afresh each step: lanes over candidates, waves over the neighbour
// list, each term the float64 difference b_j - C(c, j) times v_j rounded onto
// the fixed-point grid.  n <= kLocalMaxN, g <= kLocalMaxG.
//
// The exchanges and the fixed point are in sgs_exchange.h.
#include <hip/hip_runtime.h>

#include <algorithm>

#include "sgs_exchange.h"

namespace cp {
namespace {

constexpr int kLocalMaxN = 16384;
constexpr int kLocalMaxG = 128;

__global__ __launch_bounds__(kBlock) void sgs_local_kernel(IncDev a, const int32_t* __restrict__ nbr, int g) {
  extern __shared__ unsigned long long smem[];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int blk = blockIdx.x, nb = gridDim.x;
  const int lo = blk * a.W;
  const int cnt = max(0, min(a.n, lo + a.W) - lo);
  unsigned long long* sGlo = smem;                                 // [W] gains, low words
  long long* sGhi = reinterpret_cast<long long*>(sGlo + a.W);      // [W] high words
  float* sball = reinterpret_cast<float*>(sGhi + a.W);             // [n] best cost of every target
  float* scg = sball + a.n;                                        // [W][g] C(c, j), j in M_g(c)
  int* snb = reinterpret_cast<int*>(scg + size_t(a.W) * g);        // [W][g] M_g(c)
  unsigned char* ssel = reinterpret_cast<unsigned char*>(snb + size_t(a.W) * g);   // [W]
  __shared__ __int128 red[kBlock];
  __shared__ __int128 sg[kWaves];
  __shared__ double sd[kWaves];
  __shared__ int si[kWaves];
  __shared__ int swt[kWaves];
  __shared__ unsigned long long su[kWaves];
  __shared__ int spre[kMaxBlocks + 1];
  __shared__ int sflag;                       // abort seen while waiting for the winner
  __shared__ int slflag;                      // ... or for the slice lengths

  for (int j = tid; j < a.n; j += kBlock) sball[j] = a.c0;
  for (int i = tid; i < cnt; i += kBlock) ssel[i] = 0;
  // The band of the own candidates: neighbour lists and C(c, j) = C_tm[j][c]
  // (indices clamped into range; the table is the caller's).
  for (int e = tid; e < cnt * g; e += kBlock) {
    const int i = e / g;
    const int j = min(max(nbr[size_t(lo + i) * g + (e - i * g)], 0), a.n - 1);
    snb[e] = j;
    scg[e] = a.C[size_t(j) * a.n + lo + i];
  }

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
    (void)__builtin_frexp(M, &e);
    S = 101 - e;
  }

  // Objective in block 0, one running part per wave (as in the incremental
  // form): step l's total is written after the next step's first barrier.
  __shared__ __int128 sLw[kWaves];
  int obj_step = -1;
  if (blk == 0) {
    __int128 x = 0;
    for (int j = tid; j < a.n; j += kBlock) x += fx(double(a.v[j]) * double(a.c0), S);
    const __int128 L0 = block_sum_i128(x, sg);
    if (tid < kWaves) sLw[tid] = tid == 0 ? L0 : 0;
  }

  // Local gains of the own candidates from the current best costs: lane =
  // candidate within a chunk of 64, waves split the neighbour list.
  const int qper = (g + kWaves - 1) / kWaves;
  auto local_gains = [&]() {
    __syncthreads();
    for (int cc = 0; cc < cnt; cc += 64) {
      const int i = cc + lane;
      __int128 gsum = 0;
      if (i < cnt) {
        const int q1 = min(g, (w + 1) * qper);
        for (int q = w * qper; q < q1; ++q) {
          const int j = snb[i * g + q];
          const double d = double(sball[j]) - double(scg[i * g + q]);
          if (d > 0.0) gsum += fx(double(a.v[j]) * d, S);
        }
      }
      red[tid] = gsum;
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
  };

  local_gains();
  publish_argmax(sGlo, sGhi, ssel, lo, cnt, S, cand_slot(a.cand, 0, blk), epoch_of(0), sg, si);

  for (int step = 0; step < a.k; ++step) {
    const int tw = read_winner(cand_slot(a.cand, step & 1, 0), epoch_of(step), nb, a.abort, su, &sflag);
    if (tw < 0) break;
    if (blk == 0 && tid == 0 && obj_step >= 0 && a.step_obj) {
      __int128 L = 0;
#pragma unroll
      for (int q = 0; q < kWaves; ++q) L += sLw[q];
      a.step_obj[obj_step] = fx_to_double(L, S);
    }
    const int t = min(tw, a.n - 1);
    if (t >= lo && t < lo + cnt && tid == 0) {
      ssel[t - lo] = 1;
      a.selected[step] = t;
      if (a.step_gain) a.step_gain[step] = fx_to_double(((__int128)sGhi[t - lo] << 64) | (__int128)sGlo[t - lo], S);
    }

    // 1. Own targets that the pick improves, into the block's slice.
    int base = 0;
    unsigned long long* mine = a.list + size_t(blk) * a.W * 2;
    for (int i0 = 0; i0 < cnt; i0 += kBlock) {
      const int i = i0 + tid;
      float cv = 0.f, bo = 0.f;
      bool hit = false;
      if (i < cnt) {
        cv = a.C[size_t(lo + i) * a.n + t];
        bo = sball[lo + i];
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
            (unsigned long long)(unsigned int)(lo + i) | ((unsigned long long)__float_as_uint(a.v[lo + i]) << 32));
        put(mine + size_t(slot) * 2 + 1,
            (unsigned long long)__float_as_uint(bo) | ((unsigned long long)__float_as_uint(cv) << 32));
        if (a.assign) a.assign[lo + i] = t;
      }
      base += tot;
      __syncthreads();
    }
    if (tid == 0) put(lens_slot(a.lens, blk), ((unsigned long long)(step + 1) << 32) | unsigned(base));
    if (step + 1 == a.k && blk != 0) break;

    // 2. Every block's slice length, then every change applied to the
    // replicated best costs (and, in block 0, to the objective).
    {
      if (tid == 0) slflag = 0;
      __syncthreads();
      int c = 0;
      if (tid < nb) {
        unsigned long long x;
        const unsigned int round = unsigned(step + 1);
        if (wait_slot(lens_slot(a.lens, tid), a.abort, [round](unsigned long long v) { return (v >> 32) == round; }, x))
          c = int(x & 0xffffffffull);
        else
          slflag = 1;
      }
      const int incl = block_inclusive_scan(c, swt);
      if (tid < nb) spre[tid + 1] = incl;
      if (tid == 0) spre[0] = 0;
      __syncthreads();
    }
    if (slflag) break;
    const int total = spre[nb];
    __int128 dobj = 0;
    for (int e = tid; e < total; e += kBlock) {
      int s0 = 0, s1 = nb;   // spre[s0] <= e < spre[s1]
      while (s1 - s0 > 1) {
        const int mid = (s0 + s1) >> 1;
        if (spre[mid] <= e) s0 = mid;
        else s1 = mid;
      }
      const unsigned long long* src = a.list + (size_t(s0) * a.W + size_t(e - spre[s0])) * 2;
      const unsigned long long h0 = get(src), h1 = get(src + 1);
      const int j = int(h0 & 0xffffffffull);
      const float bn = __uint_as_float(unsigned(h1 >> 32));
      sball[j] = bn;
      if (blk == 0) {
        const double vj = double(__uint_as_float(unsigned(h0 >> 32)));
        dobj += fx(vj * double(bn), S) - fx(vj * double(__uint_as_float(unsigned(h1 & 0xffffffffull))), S);
      }
    }
    if (blk == 0) {
      dobj = wave_sum_i128(dobj);
      if (lane == 0) sLw[w] += dobj;
      obj_step = step;
    }

    // 3. Fresh local gains and this block's candidate for the next step.
    if (step + 1 < a.k) {
      local_gains();
      publish_argmax(sGlo, sGhi, ssel, lo, cnt, S, cand_slot(a.cand, (step + 1) & 1, blk),
                     epoch_of(step + 1), sg, si);
    }
  }
  __syncthreads();
  if (blk == 0 && tid == 0 && obj_step >= 0 && a.step_obj) {
    __int128 L = 0;
#pragma unroll
    for (int q = 0; q < kWaves; ++q) L += sLw[q];
    a.step_obj[obj_step] = fx_to_double(L, S);
  }
  if (blk == 0 && get(a.abort))
    for (int s = tid; s < a.k; s += kBlock) a.selected[s] = -1;
}

}  // namespace


size_t sgs_local_workspace_bytes(int64_t n, int64_t k) { return layout(n, k).total; }

hipError_t launch_sgs_local(const SgsParams& p, const int32_t* nbr, int g, hipStream_t stream) {
  if (p.n < 1 || p.n > kLocalMaxN || g < 1 || g > p.n || g > kLocalMaxG) return hipErrorInvalidValue;
  int dev = 0, cus = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if ((e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev)) != hipSuccess) return e;
  const int nb = blocks_for(p.n, cus);
  const int W = (p.n + nb - 1) / nb;
  const size_t lds = size_t(W) * 16 + size_t(p.n) * 4 + size_t(W) * g * 8 + size_t(W) + 16;
  if ((e = hipFuncSetAttribute(reinterpret_cast<const void*>(sgs_local_kernel),
                               hipFuncAttributeMaxDynamicSharedMemorySize, int(lds))) != hipSuccess)
    return e;
  int per_cu = 0;
  if ((e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, reinterpret_cast<const void*>(sgs_local_kernel),
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
  a.lens = reinterpret_cast<unsigned long long*>(w + L.lens);
  a.cand = reinterpret_cast<unsigned long long*>(w + L.cand);
  a.abort = reinterpret_cast<unsigned int*>(w + L.ctrl);
  a.W = W;

  sgs_inc_init_kernel<<<std::min(1024, (std::max(p.n, p.k) + 255) / 256), 256, 0, stream>>>(a);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  void* args[] = {&a, const_cast<int32_t**>(&nbr), &g};
  return hipLaunchCooperativeKernel(reinterpret_cast<const void*>(sgs_local_kernel), dim3(nb), dim3(kBlock), args,
                                    lds, stream);
}

}  // namespace cp
