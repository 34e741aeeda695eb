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
// One cooperative launch, one block of eight waves per compute unit.  Block b owns the rows
// and the columns [b W, (b + 1) W): the best costs b_j and capacities of its
// rows and the running gains of its columns stay in LDS for the whole launch.
// Per step:
//   1. every block reads all blocks' candidates for the step (each block's
//      best unchosen column, published at the end of the previous step) and
//      takes the same winner;
//   2. it tests its own rows against the winner's column and writes the rows
//      that improve, compacted, to its slice of the change list (row, v,
//      old b, new b), then publishes the slice's length;
//   3. it reads every block's length, walks the whole change list (slices
//      in block order) and applies the changes to its columns' gains,
//      reading each changed row's segment over its columns (one coalesced
//      256-byte read per row and 64 columns); block 0 also applies them to the
//      objective, kept in the same fixed point;
//   4. it publishes the exact argmax of its unchosen columns.
//
// The exchanges and the fixed point are in sgs_exchange.h.
#include <hip/hip_runtime.h>

#include <algorithm>

#include "sgs_exchange.h"

namespace cp {
namespace {

constexpr int kBatch = 64;         // change-list entries a wave fetches per round
constexpr int kChunk = 16;         // of which the rows read together
constexpr int kInitRows = 16;      // rows a wave has in flight in the full pass

// The greedy of one scene as run by block `blk` of the scene's `nb` blocks.
__device__ __forceinline__ void inc_body(const IncDev& a, int blk, int nb) {
  extern __shared__ unsigned long long smem[];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int lo = blk * a.W;
  const int cnt = max(0, min(a.n, lo + a.W) - lo);
  unsigned long long* sGlo = smem;                                 // [W] running gains, low words
  long long* sGhi = reinterpret_cast<long long*>(sGlo + a.W);      // [W] high words
  float* sb = reinterpret_cast<float*>(sGhi + a.W);                // [W] best costs of own rows
  float* sv = sb + a.W;                                            // [W] capacities of own rows
  unsigned char* ssel = reinterpret_cast<unsigned char*>(sv + a.W);       // [W] chosen columns
  __shared__ __int128 red[kBlock];
  __shared__ __int128 sg[kWaves];
  __shared__ double sd[kWaves];
  __shared__ int si[kWaves];
  __shared__ int swt[kWaves];
  __shared__ unsigned long long su[kWaves];
  __shared__ int spre[kMaxBlocks + 1];        // slice offsets
  __shared__ int sflag;                       // abort seen while waiting for the winner
  __shared__ int slflag;                      // ... or for the slice lengths

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
  // 16-row chunks w, w + kWaves, ...; the waves' sums are added in wave order.
  for (int cc = 0; cc < cnt; cc += 64) {
    const bool colok = cc + lane < cnt;
    const int col = lo + cc + lane;
    __int128 g = 0;
    for (int j0 = w * kInitRows; j0 < a.n; j0 += kWaves * kInitRows) {
      float x[kInitRows], vj[kInitRows];
#pragma unroll
      for (int u = 0; u < kInitRows; ++u) {
        const int j = j0 + u;
        x[u] = (colok && j < a.n) ? __builtin_nontemporal_load(a.C + size_t(j) * a.n + col) : a.c0;
        vj[u] = j < a.n ? a.v[j] : 0.f;
      }
#pragma unroll
      for (int u = 0; u < kInitRows; ++u) g += fx(double(vj[u]) * double(fmaxf(a.c0 - x[u], 0.f)), S);
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

  // Block 0 keeps the objective L = sum_j v_j b_j in the gains' fixed point,
  // starting from b = c0, as one running part per wave: a wave adds its share
  // of a step's changes without a barrier, and thread 0 totals the parts for
  // step l after the next step's first barrier (after the loop for the last).
  __shared__ __int128 sLw[kWaves];
  int obj_step = -1;
  if (blk == 0) {
    __int128 x = 0;
    for (int j = tid; j < a.n; j += kBlock) x += fx(double(a.v[j]) * double(a.c0), S);
    const __int128 L0 = block_sum_i128(x, sg);
    if (tid < kWaves) sLw[tid] = tid == 0 ? L0 : 0;
  }

  publish_argmax(sGlo, sGhi, ssel, lo, cnt, S, cand_slot(a.cand, 0, blk), epoch_of(0), sg, si);

  for (int step = 0; step < a.k; ++step) {
    // Some block has a candidate while unchosen columns remain; the clamp
    // only keeps a broken slot from addressing past the matrix.
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
    // The barrier above completed this block's list writes.
    if (tid == 0) put(lens_slot(a.lens, blk), ((unsigned long long)(step + 1) << 32) | unsigned(base));

    // The last step's changes only feed the objective, kept by block 0.
    if (step + 1 == a.k && blk != 0) break;

    // 2. Every block's slice length (thread i waits for block i), and the
    // slices' offsets in the flattened change list.
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

    // 3. Apply the changes to the own columns' gains.  Each lane of a round
    // locates and fetches one entry; the entries are then broadcast and every
    // lane reads its column of each entry's row.
    __int128 dobj = 0;
    for (int cc = 0; cc < cnt; cc += 64) {
      const bool colok = cc + lane < cnt;
      const int col = lo + cc + lane;
      __int128 g = 0;
      // Rounds of up to kBatch entries per wave, the list split evenly over
      // the waves.
      const int per = min(kBatch, (total + kWaves - 1) / kWaves);
      for (int e0 = w * per; e0 < total; e0 += kWaves * per) {
        const int e = e0 + lane;
        unsigned long long h0 = 0ull, h1 = 0ull;
        if (lane < per && e < total) {
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
        const int m = min(per, total - e0);
        // Entry u is broadcast from lane u with readlane (u is uniform), in
        // chunks of kChunk whose row reads are in flight together.
        const int hj = int(h0 & 0xffffffffull), hv = int(h0 >> 32);
        const int hbo = int(h1 & 0xffffffffull), hbn = int(h1 >> 32);
        for (int u0 = 0; u0 < m; u0 += kChunk) {
          float x[kChunk];
#pragma unroll
          for (int i = 0; i < kChunk; ++i) {
            x[i] = 0.f;
            if (u0 + i < m && colok) {
              const int j = __builtin_amdgcn_readlane(hj, u0 + i);
              x[i] = a.C[size_t(j) * a.n + col];
            }
          }
#pragma unroll
          for (int i = 0; i < kChunk; ++i) {
            if (u0 + i < m) {
              // A column that cost at least the old best contributes 0 before
              // and after (new best < old best).
              const float bo = __int_as_float(__builtin_amdgcn_readlane(hbo, u0 + i));
              if (x[i] < bo) {
                const float bn = __int_as_float(__builtin_amdgcn_readlane(hbn, u0 + i));
                const double vj = double(__int_as_float(__builtin_amdgcn_readlane(hv, u0 + i)));
                g += fx(vj * double(fmaxf(bn - x[i], 0.f)), S) - fx(vj * double(bo - x[i]), S);
              }
            }
          }
        }
        if (blk == 0 && cc == 0 && lane < per && e < total) {
          const double vj = double(__uint_as_float(unsigned(h0 >> 32)));
          const float bo = __uint_as_float(unsigned(h1 & 0xffffffffull));
          const float bn = __uint_as_float(unsigned(h1 >> 32));
          dobj += fx(vj * double(bn), S) - fx(vj * double(bo), S);
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
#pragma unroll
      for (int o = 32; o > 0; o >>= 1) {
        const unsigned long long olo = __shfl_xor((unsigned long long)dobj, o);
        const long long ohi = __shfl_xor((long long)(dobj >> 64), o);
        dobj += ((__int128)ohi << 64) | (__int128)olo;
      }
      if (lane == 0) sLw[w] += dobj;
      obj_step = step;
    }

    // 4. This block's candidate for the next step.
    if (step + 1 < a.k)
      publish_argmax(sGlo, sGhi, ssel, lo, cnt, S, cand_slot(a.cand, (step + 1) & 1, blk),
                     epoch_of(step + 1), sg, si);
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

__global__ __launch_bounds__(kBlock) void sgs_inc_kernel(IncDev a) { inc_body(a, blockIdx.x, gridDim.x); }

// Several scenes in one launch: scene s runs on blocks [g0[s], g0[s + 1])
// with its own slots, change lists and abort flag, so the scenes' greedies
// proceed independently side by side.
constexpr int kMaxBatch = 16;

struct IncBatch {
  int count;
  int g0[kMaxBatch + 1];
  IncDev scene[kMaxBatch];
};

__global__ __launch_bounds__(kBlock) void sgs_inc_batch_kernel(IncBatch b) {
  int s = 0;
  while (s + 1 < b.count && int(blockIdx.x) >= b.g0[s + 1]) ++s;
  inc_body(b.scene[s], int(blockIdx.x) - b.g0[s], b.g0[s + 1] - b.g0[s]);
}

IncDev inc_dev(const SgsParams& p, char* w, int W) {
  const Layout L = layout(p.n, p.k);
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
  return a;
}

size_t lds_for(int W) { return size_t(W) * (16 + 4 + 4 + 1) + 16; }

}  // namespace

size_t sgs_inc_workspace_bytes(int64_t n, int64_t k) { return layout(n, k).total; }

hipError_t launch_sgs_incremental(const SgsParams& p, hipStream_t stream) {
  int dev = 0, cus = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if ((e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev)) != hipSuccess) return e;
  const int nb = blocks_for(p.n, cus);
  const int W = (p.n + nb - 1) / nb;
  const size_t lds = lds_for(W);
  int per_cu = 0;
  if ((e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, reinterpret_cast<const void*>(sgs_inc_kernel),
                                                        kBlock, lds)) != hipSuccess)
    return e;
  if (per_cu < 1) return hipErrorCooperativeLaunchTooLarge;

  IncDev a = inc_dev(p, static_cast<char*>(p.workspace), W);
  sgs_inc_init_kernel<<<std::min(1024, (std::max(p.n, p.k) + 255) / 256), 256, 0, stream>>>(a);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  void* args[] = {&a};
  return hipLaunchCooperativeKernel(reinterpret_cast<const void*>(sgs_inc_kernel), dim3(nb), dim3(kBlock), args,
                                    lds, stream);
}

size_t sgs_inc_batch_workspace_bytes(const int64_t* n, const int64_t* k, int count) {
  size_t total = 0;
  for (int s = 0; s < count; ++s) total += layout(n[s], k[s]).total;
  return total;
}

hipError_t launch_sgs_incremental_batch(const SgsParams* p, int count, void* workspace, hipStream_t stream) {
  if (count < 1 || count > kMaxBatch) return hipErrorInvalidValue;
  int dev = 0, cus = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if ((e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev)) != hipSuccess) return e;
  if (count > cus) return hipErrorInvalidValue;
  // One block per compute unit in all: every scene starts with one, then the
  // scene with the most tokens per block gains one (up to its own cap of one
  // block per 64 tokens, at most kMaxBlocks) until the units run out.
  int nb[kMaxBatch], cap[kMaxBatch];
  int used = count;
  for (int s = 0; s < count; ++s) {
    nb[s] = 1;
    cap[s] = blocks_for(p[s].n, cus);
  }
  while (used < cus) {
    int best = -1;
    long long bw = 0;
    for (int s = 0; s < count; ++s) {
      if (nb[s] >= cap[s]) continue;
      const long long w = (p[s].n + nb[s] - 1) / nb[s];
      if (w > bw) {
        bw = w;
        best = s;
      }
    }
    if (best < 0) break;
    ++nb[best];
    ++used;
  }
  IncBatch b;
  b.count = count;
  b.g0[0] = 0;
  size_t lds = 0, off = 0;
  char* w = static_cast<char*>(workspace);
  for (int s = 0; s < count; ++s) {
    const int W = (p[s].n + nb[s] - 1) / nb[s];
    b.scene[s] = inc_dev(p[s], w + off, W);
    b.g0[s + 1] = b.g0[s] + nb[s];
    lds = std::max(lds, lds_for(W));
    off += layout(p[s].n, p[s].k).total;
  }
  int per_cu = 0;
  if ((e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, reinterpret_cast<const void*>(sgs_inc_batch_kernel),
                                                        kBlock, lds)) != hipSuccess)
    return e;
  if (per_cu < 1) return hipErrorCooperativeLaunchTooLarge;
  for (int s = 0; s < count; ++s) {
    sgs_inc_init_kernel<<<std::min(1024, (std::max(p[s].n, p[s].k) + 255) / 256), 256, 0, stream>>>(b.scene[s]);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  void* args[] = {&b};
  return hipLaunchCooperativeKernel(reinterpret_cast<const void*>(sgs_inc_batch_kernel), dim3(used), dim3(kBlock),
                                    args, lds, stream);
}

}  // namespace cp
