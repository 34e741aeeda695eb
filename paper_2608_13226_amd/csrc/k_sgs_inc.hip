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
// that c0 sum(v) stays below 2^62; gains are sums of these integers in 64
// bits.  Integer sums do not depend on their order, so the running gains are
// bit-identical to gains summed afresh from the current b (a gain that has
// dropped to zero is exactly zero), and equal gains go to the smaller index.
// The grid, about 2^-62 c0 sum(v), is finer than the rounding of a float64
// sum of the same terms.
//
// The fixed-point scale and the step-0 gains (b = c0) come from two ordinary
// kernels ahead of the greedy (inc_scale_kernel, inc_first_pass_kernel), which
// run with many more waves in flight than the greedy itself.  The greedy is
// one cooperative launch, one block of eight waves per compute unit.  Block b
// owns the rows and the columns [b W, (b + 1) W): the best costs b_j and
// capacities of its rows and the running gains of its columns stay in LDS for
// the whole launch.  Per step:
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

// The greedy of one scene as run by block `blk` of the scene's `nb` blocks.
__device__ __forceinline__ void inc_body(const IncDev& a, int blk, int nb) {
  extern __shared__ unsigned long long smem[];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int lo = blk * a.W;
  const int cnt = max(0, min(a.n, lo + a.W) - lo);
  long long* sG = reinterpret_cast<long long*>(smem);             // [W] running gains
  float* sb = reinterpret_cast<float*>(sG + a.W);                  // [W] best costs of own rows
  float* sv = sb + a.W;                                            // [W] capacities of own rows
  unsigned char* ssel = reinterpret_cast<unsigned char*>(sv + a.W);       // [W] chosen columns
  __shared__ long long red[kBlock];
  __shared__ long long sg[kWaves];
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

  // The fixed-point scale and the step-0 gains of the own columns (every row
  // at b = c0) come from the first-pass kernels: the gains as P partial sums
  // over row ranges, whose integer total does not depend on the split.
  const int S = *a.scale;
  for (int i = tid; i < cnt; i += kBlock) {
    long long g = 0;
    for (int q = 0; q < a.P; ++q) g += a.part[size_t(q) * a.n + lo + i];
    sG[i] = g;
  }
  __syncthreads();

  // Block 0 keeps the objective L = sum_j v_j b_j in the gains' fixed point,
  // starting from b = c0, as one running part per wave: a wave adds its share
  // of a step's changes without a barrier, and thread 0 totals the parts for
  // step l after the next step's first barrier (after the loop for the last).
  __shared__ long long sLw[kWaves];
  int obj_step = -1;
  if (blk == 0) {
    const long long x = fx_capacity_part(a.v, a.n, a.c0, S);
    const long long L0 = block_sum_i64(x, sg);
    if (tid < kWaves) sLw[tid] = tid == 0 ? L0 : 0;
  }

  publish_argmax(sG, ssel, lo, cnt, S, cand_slot(a.cand, 0, blk), epoch_of(0), sg, si);

  for (int step = 0; step < a.k; ++step) {
    // Some block has a candidate while unchosen columns remain; the clamp
    // only keeps a broken slot from addressing past the matrix.
    const int tw = read_winner(cand_slot(a.cand, step & 1, 0), epoch_of(step), nb, a.abort, a.poll_limit, su, &sflag);
    if (tw < 0) break;
    if (blk == 0 && tid == 0 && obj_step >= 0 && a.step_obj) {
      long long L = 0;
#pragma unroll
      for (int q = 0; q < kWaves; ++q) L += sLw[q];
      a.step_obj[obj_step] = fx_to_double(L, S);
    }
    const int t = min(tw, a.n - 1);
    if (t >= lo && t < lo + cnt && tid == 0) {
      ssel[t - lo] = 1;
      a.selected[step] = t;
      if (a.step_gain) a.step_gain[step] = fx_to_double(sG[t - lo], S);
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
        if (wait_slot(lens_slot(a.lens, tid), a.abort, a.poll_limit,
                      [round](unsigned long long v) { return (v >> 32) == round; }, x))
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
    long long dobj = 0;
    for (int cc = 0; cc < cnt; cc += 64) {
      const bool colok = cc + lane < cnt;
      const int col = lo + cc + lane;
      long long g = 0;
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
        const int hj = int(h0 & 0xffffffffull);
        const int hbo = int(h1 & 0xffffffffull), hbn = int(h1 >> 32);
        // Each lane's entry capacity scaled once for fx_scaled.
        const long long hvs = __double_as_longlong(fx_scale(double(__uint_as_float(unsigned(h0 >> 32))), S));
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
                const double vs = __longlong_as_double(
                    (long long)(((unsigned long long)(unsigned)__builtin_amdgcn_readlane(int(hvs >> 32), u0 + i) << 32) |
                                (unsigned)__builtin_amdgcn_readlane(int(hvs), u0 + i)));
                g += (long long)(fx_scaled(vs, fmaxf(bn - x[i], 0.f)) - fx_scaled(vs, bo - x[i]));
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
        long long s = sG[cc + tid];
#pragma unroll
        for (int q = 0; q < kWaves; ++q) s += red[q * 64 + tid];
        sG[cc + tid] = s;
      }
      __syncthreads();
    }
    if (blk == 0) {
      dobj = wave_sum_i64(dobj);
      if (lane == 0) sLw[w] += dobj;
      obj_step = step;
    }

    // 4. This block's candidate for the next step.
    if (step + 1 < a.k)
      publish_argmax(sG, ssel, lo, cnt, S, cand_slot(a.cand, (step + 1) & 1, blk),
                     epoch_of(step + 1), sg, si);
  }
  __syncthreads();
  if (blk == 0 && tid == 0 && obj_step >= 0 && a.step_obj) {
    long long L = 0;
#pragma unroll
    for (int q = 0; q < kWaves; ++q) L += sLw[q];
    a.step_obj[obj_step] = fx_to_double(L, S);
  }
}

// ---------------------------------------------------------------------------
// Rows form of the same greedy, for scenes whose n best costs fit in LDS.
//
// The exchange form learns J_l from the owners of the rows (a pass over the
// own rows, an exchange of slice lengths, a walk of the change list).  Here
// every block keeps all n best costs b_j in LDS and finds J_l itself: it
// reads the winner's costs to every target, C(t_l, j) for all j, as one
// contiguous row of a source-major copy T of the cost (T[s][j] = C(s, j)),
// tests each against b_j, and applies the rows that improve straight away.
// Every block then holds the identical J_l and the identical b, a step needs
// one exchange (the candidates) instead of two, and no block reads another's
// list.  T is written by the first-pass kernel, which reads the whole cost in
// column strips for the step-0 gains anyway.
//
// Per step and wave: the wave's chunks of the winner's row (256 targets a
// load, 16 bytes a lane) are loaded together; a chunk without a hit costs one
// LDS read and four compares; hits are compacted into the wave's list in LDS
// (target, old b, new b) and their rows' segments over the block's columns
// are read 16 rows at a time.  The block's columns' deltas are then summed
// over the waves in wave order, as in the exchange form, and are the same
// integers, so both forms take the same picks.
constexpr int kRowsMaxN = 32768;   // 128 KB of best costs in LDS
constexpr int kRowsMaxW = 128;     // columns per block: two per lane
constexpr int kRowChunk = 256;     // targets per wave-load of the winner's row
constexpr int kList = 128;         // hits a wave collects before applying them (dense steps)
constexpr int kCap = kList * kWaves;   // hits a block lists in one step

int rows_ldt(int64_t n) { return int((n + kRowChunk - 1) / kRowChunk * kRowChunk); }

// Fixed-point scale, the same in every block (same sum, same order): every
// partial gain is at most c0 sum(v) < 2^(62 - S), and every single term
// v_j d 2^S (0 <= d <= c0) at most c0 max(v) 2^S < 2^52, which fx_diff
// needs.
__device__ __forceinline__ int fixed_scale(const IncDev& a, double* sd) {
  double x = 0.0, m = 0.0;
  // Thread t adds v[t], v[t + kBlock], ... in that order; the loads of
  // eight of them go out together (indices past n read v[n - 1], unused).
  constexpr int U = 8;
  for (int j0 = threadIdx.x; j0 < a.n; j0 += kBlock * U) {
    float vv[U];
#pragma unroll
    for (int u = 0; u < U; ++u) vv[u] = a.v[min(j0 + u * kBlock, a.n - 1)];
#pragma unroll
    for (int u = 0; u < U; ++u)
      if (j0 + u * kBlock < a.n) {
        x += double(vv[u]);
        m = fmax(m, double(vv[u]));
      }
  }
  const double M = double(a.c0) * block_sum_all(x, sd);
  const double Mt = double(a.c0) * block_max_all(m, sd);
  int S = 0;
  if (M > 0.0) {
    int e = 0;
    (void)__builtin_frexp(M, &e);   // M < 2^e
    S = 62 - e;
    (void)__builtin_frexp(Mt, &e);  // 0 < Mt <= M
    S = min(S, 52 - e);
  }
  return S;
}

// Predicting the next winner (rows schedule, at most 64 columns a block).
// Each block publishes two words in its slot: its best key (word 0) and its
// second-best key (word 1), each with the exchange's epoch bit.  After a
// step's exchange every block knows, for the runner-up r (the best candidate
// outside the winner's block), a lower bound on its fixed-point gain (from
// its key), and an upper bound U on every other candidate's truncated gain:
// the best keys of all blocks but the winner's and r's, and the second-best
// keys of those two (a block's other columns gain at most its second best,
// and gains only fall).  While applying the step's hits every block also sums
// r's changes from the same terms, so every block holds the same lower bound
// on r's gain after the step; if its truncated gain is strictly above U, r is
// the next winner (whatever the indices), every block knows it, and the next
// step runs without an exchange, on r's row of T loaded during this step.
// The same holds down a chain: with r_1, r_2, ... the best candidates of
// distinct blocks in key order (the winner's block left out), r_m follows
// r_(m-1) when its bound beats the best key of the remaining blocks, r_(m+1),
// and the second-best keys of the winner's block and of r_1 .. r_m; every
// block tracks the changes of all of r_1 .. r_kChain since the exchange.
__device__ __forceinline__ void publish_rows(const long long* sG, const unsigned char* ssel, int lo, int cnt, int S,
                                             unsigned long long* slot, unsigned long long epoch) {
  if (threadIdx.x >= 64) return;
  const int i = threadIdx.x;
  const bool ok = i < cnt && !ssel[i];
  long long g1 = ok ? sG[i] : -1;
  int i1 = ok ? lo + i : INT_MAX;
  const long long mine = g1;
  const int mi = i1;
  wave_argmax(g1, i1);
  long long g2 = mi == i1 ? -1 : mine;
  int i2 = mi == i1 ? INT_MAX : mi;
  wave_argmax(g2, i2);
  if (i == 0) {
    put(slot + 1, (i2 != INT_MAX ? pack_key(fx_to_double(g2, S), i2) : kNoCandidate) | epoch);
    put(slot, (i1 != INT_MAX ? pack_key(fx_to_double(g1, S), i1) : kNoCandidate) | epoch);
  }
}

// A lower bound on the fixed-point gain g behind a key: the key keeps the
// top bits of the float64 value of g 2^-S (rounded to nearest from 64 bits,
// then truncated), so scaling it back can exceed g by at most half a unit in
// the 53rd bit, which the bound takes off.
__device__ __forceinline__ long long key_gain_floor(unsigned long long key, int S) {
  const double d = __longlong_as_double((long long)((key >> kIndexBits) << (kIndexBits + 1)));
  const long long G = (long long)__builtin_ldexp(d, S);
  return max(0ll, G - (G >> 52) - 1);
}

// read_winner for two-word slots: thread i < nb polls both words of block
// i's slot and stores them (epoch bits cleared) in sk1 and sk2.  Returns the
// winner's index, -1 when the launch is aborting.
__device__ int read_winner_rows(const unsigned long long* slots, unsigned long long epoch, int nb, unsigned int* abort,
                                unsigned int limit, unsigned long long* su, int* sflag, unsigned long long* sk1,
                                unsigned long long* sk2) {
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  unsigned long long best = 0ull;
  if (tid == 0) *sflag = 0;
  __syncthreads();
  if (tid < nb) {
    const unsigned long long* p = slots + size_t(tid) * kSlotStride;
    bool done = false;
    for (unsigned int spins = 0; !done; ++spins) {
      const unsigned long long x0 = get(p), x1 = get(p + 1);
      if ((x0 & kEpoch) == epoch && (x1 & kEpoch) == epoch) {
        best = x0 & ~kEpoch;
        sk1[tid] = best;
        sk2[tid] = x1 & ~kEpoch;
        done = true;
      } else {
        if (give_up(spins, limit, abort)) {
          *sflag = 1;
          break;
        }
        __builtin_amdgcn_s_sleep(1);
      }
    }
  }
  best = wave_max_u64(best);
  if (lane == 0) su[w] = best;
  __syncthreads();
  unsigned long long m = su[0];
#pragma unroll
  for (int q = 1; q < kWaves; ++q) m = su[q] > m ? su[q] : m;
  const bool aborting = *sflag != 0;
  __syncthreads();
  return aborting ? -1 : int(kIndexMask - (m & kIndexMask));
}

constexpr int kChain = 1;   // predicted steps in a row at most (deeper chains measured slower)
constexpr int kTrackMax = 256;   // hits of a step that still tracks the chain

// The step-0 gains of a block's columns [lo, lo + cnt) from the P partial
// sums part[q][column] (64-bit integers, so the split does not matter):
// thread (column tid % 64, group tid / 64) adds partials group, group +
// kWaves, ..., eight loads in flight, then the groups' sums are added in
// LDS.  P is 3 after the first pass, n / 64 after the fused epilogue.
__device__ __forceinline__ void init_gains(const IncDev& a, long long* sG, int lo, int cnt, long long* red) {
  const int tid = threadIdx.x, g = tid >> 6;
  for (int i0 = 0; i0 < cnt; i0 += 64) {
    const int i = i0 + (tid & 63);
    const int col = lo + min(i, cnt - 1);
    long long x = 0;
    for (int q0 = g; q0 < a.P; q0 += 8 * kWaves) {
      long long v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) v[u] = a.part[size_t(min(q0 + u * kWaves, a.P - 1)) * a.n + col];
#pragma unroll
      for (int u = 0; u < 8; ++u)
        if (q0 + u * kWaves < a.P) x += v[u];
    }
    red[tid] = x;
    __syncthreads();
    if (tid < 64 && i0 + tid < cnt) {
      long long t = 0;
#pragma unroll
      for (int r = 0; r < kWaves; ++r) t += red[r * 64 + tid];
      sG[i0 + tid] = t;
    }
    __syncthreads();
  }
}

// NG 64-column groups per block (W <= 64 NG); RL chunk loads per wave and
// step (n <= kRowChunk kWaves RL).
template <int NG, int RL>
__device__ __forceinline__ void rows_body(const IncDev& a, int blk, int nb) {
  extern __shared__ unsigned long long smem[];
  // Hits a block lists in one step: with one column group the list is four
  // times kCap (48 KB of LDS beside the 64 KB of best costs), which puts all
  // but the first dense steps in one round; two groups keep 128 KB of best
  // costs and the short list.
  constexpr int kCapR = (NG == 1 ? 4 : 1) * kCap;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int lo = blk * a.W;
  const int cnt = max(0, min(a.n, lo + a.W) - lo);
  long long* sG = reinterpret_cast<long long*>(smem);             // [W] running gains (W rounded up to even)
  float* sball = reinterpret_cast<float*>(sG + ((a.W + 1) & ~1));  // [ldt] b_j, 16-byte aligned; -inf past n
  unsigned char* ssel = reinterpret_cast<unsigned char*>(sball + a.ldt);   // [W] chosen columns
  __shared__ long long red[kBlock];
  __shared__ long long sg[kWaves];
  __shared__ int si[kWaves];
  __shared__ unsigned long long su[kWaves];
  __shared__ int sflag;
  __shared__ int lj[kCapR];                    // hit list: target
  __shared__ float lbo[kCapR];                 // old best cost
  __shared__ float lbn[kCapR];                 // new best cost
  __shared__ int scnt[2];                     // hits listed in steps of each parity
  __shared__ int schunk[kRowsMaxN / kRowChunk];   // dense steps: hits per chunk, then their offsets
  if (tid == 0) scnt[0] = scnt[1] = 0;
  // Prediction of the next winners (one column group only): every block's
  // two slot words of the last exchange and the waves' parts of the chain
  // candidates' changes in the step.
  constexpr bool kSpec = NG == 1;
  __shared__ unsigned long long sk1[kSpec ? kMaxBlocks : 1], sk2[kSpec ? kMaxBlocks : 1];
  __shared__ long long sdr[kWaves][kChain];

  // A launch that continues another one runs only when its gate says so
  // (the same word for every block), and then starts from the state the
  // previous launch handed over.
  if (a.gate && *a.gate != a.gate_val) return;
  // After the early kernel the first step is the one it stopped before.
  if (a.start && *a.abort) return;
  const int k_begin = a.start ? int(*a.start) : a.k_begin;
  const bool resume = k_begin > 0;
  if (resume && *a.abort) return;             // the launch before it gave up
  // The fixed-point scale, the step-0 gains (as P partial sums over row
  // ranges) and T come from the first-pass kernels.
  const int S = *a.scale;
  if (resume) {
    for (int j = tid; j < a.ldt; j += kBlock) sball[j] = a.ho_b[j];
    for (int i = tid; i < cnt; i += kBlock) {
      ssel[i] = a.ho_sel[lo + i];
      sG[i] = a.ho_gain[lo + i];
    }
  } else {
    for (int j = tid; j < a.ldt; j += kBlock) sball[j] = j < a.n ? a.c0 : -__builtin_inff();
    for (int i = tid; i < cnt; i += kBlock) ssel[i] = 0;
    init_gains(a, sG, lo, cnt, red);
  }
  __syncthreads();

  // Block 0 keeps the objective as one running part per wave (as in the
  // exchange form).
  __shared__ long long sLw[kWaves];
  int obj_step = k_begin - 1;
  if (blk == 0) {
    long long L0 = 0;
    if (resume) {
      L0 = a.ho_misc[0];
    } else {
      const long long x = fx_capacity_part(a.v, a.n, a.c0, S);
      L0 = block_sum_i64(x, sg);
    }
    if (tid < kWaves) sLw[tid] = tid == 0 ? L0 : 0;
  }

  // Slot sets and epochs count exchanges, which predicted steps skip.  A
  // continuing launch finds its first exchange's candidates published.
  int xc = resume ? int(a.ho_misc[1]) : 0;
  if (!resume) {
    if (kSpec)
      publish_rows(sG, ssel, lo, cnt, S, cand_slot(a.cand, 0, blk), epoch_of(0));
    else
      publish_argmax(sG, ssel, lo, cnt, S, cand_slot(a.cand, 0, blk), epoch_of(0), sg, si);
  }

  const int nch = a.ldt / kRowChunk;
  bool predicted = false;     // this step's winner was predicted (no exchange)
  int tpred = -1;
  f32x4 xr2[RL];              // the predicted winner's row, loaded during the previous step
  // The chain since the last exchange, the same in every wave and block:
  // candidates r_1 .. (-1 past the last), lower bounds on their gains (with
  // their changes since the exchange), the bounds they must beat (truncated
  // gain bits), and the position (steps predicted since the exchange).
  int rc[kChain];
  long long acc[kChain];
  unsigned long long ub[kChain];
  int chain = 0;
#pragma unroll
  for (int m = 0; m < kChain; ++m) {
    rc[m] = -1;
    acc[m] = 0;
    ub[m] = 0ull;
  }
  for (int step = k_begin; step < a.k_end; ++step) {
    int tw;
    if (predicted) {
      __syncthreads();
      tw = tpred;
    } else {
      tw = kSpec ? read_winner_rows(cand_slot(a.cand, xc & 1, 0), epoch_of(xc), nb, a.abort, a.poll_limit, su,
                                    &sflag, sk1, sk2)
                 : read_winner(cand_slot(a.cand, xc & 1, 0), epoch_of(xc), nb, a.abort, a.poll_limit, su, &sflag);
      ++xc;
    }
    if (tw < 0) break;
    if (blk == 0 && tid == 0 && obj_step >= 0 && a.step_obj) {
      long long L = 0;
#pragma unroll
      for (int q = 0; q < kWaves; ++q) L += sLw[q];
      a.step_obj[obj_step] = fx_to_double(L, S);
    }
    const int t = min(tw, a.n - 1);
    if (t >= lo && t < lo + cnt && tid == 0) {
      ssel[t - lo] = 1;
      a.selected[step] = t;
      if (a.step_gain) a.step_gain[step] = fx_to_double(sG[t - lo], S);
    }

    // The wave's chunks of the winner's row, all loads in flight together
    // (already loaded when the winner was predicted).
    const f32x4* row = reinterpret_cast<const f32x4*>(a.T + size_t(t) * a.ldt);
    f32x4 xr[RL];
#pragma unroll
    for (int i = 0; i < RL; ++i)
      if (w + i * kWaves < nch) xr[i] = predicted ? xr2[i] : row[(w + i * kWaves) * (kRowChunk / 4) + lane];

    // After an exchange every wave builds the chain while the row is in
    // flight: the best keys of distinct blocks in order, each taken out in
    // turn.  Blocks own W consecutive columns, so the winner's block is t / W.
    if (kSpec && !predicted) {
      const int bt = block_of(a, t);
      unsigned long long k[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int b = lane + 64 * q;
        k[q] = (b < nb && b != bt) ? sk1[b] : 0ull;
      }
      unsigned long long u2 = sk2[bt];
      int bprev = -1;
#pragma unroll
      for (int m = 0; m <= kChain; ++m) {
        const unsigned long long kr = wave_max_u64(max(max(k[0], k[1]), max(k[2], k[3])));
        const bool real = kr > kNoCandidate && (m == 0 || bprev >= 0);
        const int r = real ? int(kIndexMask - (kr & kIndexMask)) : -1;
        const int br = real ? block_of(a, r) : -1;
        if (m > 0) ub[m - 1] = max(real ? kr : 0ull, u2) >> kIndexBits;
        if (m < kChain) {
          rc[m] = r;
          acc[m] = real ? key_gain_floor(kr, S) : 0;
          if (real) u2 = max(u2, sk2[br]);
#pragma unroll
          for (int q = 0; q < 4; ++q) k[q] = (lane + 64 * q) == br ? 0ull : k[q];
        }
        bprev = br;
      }
      chain = 0;
    }

    long long g[NG];
#pragma unroll
    for (int q = 0; q < NG; ++q) g[q] = 0;
    long long dobj = 0;
    long long dr[kChain];       // this wave's parts of the chain candidates' changes
#pragma unroll
    for (int m = 0; m < kChain; ++m) dr[m] = 0;
    // Candidates still ahead in the chain: r_(chain+1) ..
    auto live = [&](int m) { return kSpec && m >= chain && rc[m] >= 0; };
    // Applies listed hits base .. base + m to the wave's partial gains (and,
    // in block 0, to the objective), and records them in assign and (with
    // setb) in b.
    auto apply = [&](int base, int m, bool setb) {
      // Lane u < kChunk of a batch holds entry e0 + u and its capacity; the
      // entries are broadcast with readlane.  The next batch's entries and
      // row reads are issued before the current batch's terms are summed.
      int jl = 0;
      float bol = 0.f, bnl = 0.f, vl = 0.f;
      float rl[kChain];
      float xc[kChunk][NG];
      auto fetch = [&](int e0) {
        const int nbt = min(kChunk, base + m - e0);
        jl = 0;
        bol = bnl = vl = 0.f;
#pragma unroll
        for (int c = 0; c < kChain; ++c) rl[c] = 0.f;
        if (lane < nbt) {
          jl = lj[e0 + lane];
          bol = lbo[e0 + lane];
          bnl = lbn[e0 + lane];
          vl = a.v[jl];
#pragma unroll
          for (int c = 0; c < kChain; ++c)
            if (live(c)) rl[c] = a.C[size_t(jl) * a.n + rc[c]];   // C(r_c, j): a candidate's cost to the entry
        }
#pragma unroll
        for (int u = 0; u < kChunk; ++u) {
          const int j = __builtin_amdgcn_readlane(jl, u);
#pragma unroll
          for (int q = 0; q < NG; ++q)
            xc[u][q] = (u < nbt && q * 64 + lane < cnt) ? a.C[size_t(j) * a.n + lo + q * 64 + lane] : 0.f;
        }
      };
      if (m > 0) fetch(base);
      for (int e0 = base; e0 < base + m; e0 += kChunk) {
        const int nbt = min(kChunk, base + m - e0);
        const int cj = jl;
        const float cbo = bol, cbn = bnl;
        // Each lane's entry capacity scaled once for fx_diff (0 past the
        // batch, where v was not read).
        const double cvs = fx_scale(double(vl), S);
        const long long cvb = __double_as_longlong(cvs);
        float cr[kChain];
#pragma unroll
        for (int c = 0; c < kChain; ++c) cr[c] = rl[c];
        float cx[kChunk][NG];
#pragma unroll
        for (int u = 0; u < kChunk; ++u)
#pragma unroll
          for (int q = 0; q < NG; ++q) cx[u][q] = xc[u][q];
        if (e0 + kChunk < base + m) fetch(e0 + kChunk);
#pragma unroll
        for (int u = 0; u < kChunk; ++u) {
          if (u < nbt) {
            const float bo = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(cbo), u));
            const float bn = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(cbn), u));
            const double vs = __longlong_as_double(
                (long long)(((unsigned long long)(unsigned)__builtin_amdgcn_readlane(int(cvb >> 32), u) << 32) |
                            (unsigned)__builtin_amdgcn_readlane(int(cvb), u)));
#pragma unroll
            for (int q = 0; q < NG; ++q) {
              // A column that cost at least the old best contributes 0
              // before and after.
              const float xx = cx[u][q];
              if (q * 64 + lane < cnt && xx < bo) g[q] += fx_diff(vs, fmaxf(bn - xx, 0.f), bo - xx);
            }
          }
        }
        // The batch's targets, one lane each: objective (block 0), the chain
        // candidates' changes, b and assign.
        if (lane < nbt) {
#pragma unroll
          for (int c = 0; c < kChain; ++c)
            if (live(c) && cr[c] < cbo)
              dr[c] += fx_diff(cvs, fmaxf(cbn - cr[c], 0.f), cbo - cr[c]);
          if (blk == 0) dobj += fx_diff(cvs, cbn, cbo);
          if (setb) sball[cj] = cbn;
          if (a.assign && unsigned(cj - lo) < unsigned(cnt)) a.assign[cj] = t;
        }
      }
    };

    // Fast path: the waves list the hits of their chunks in one block-wide
    // list (a chunk's hits reserve their places with one LDS atomic), and
    // after a barrier each wave applies an equal share of it: the targets a
    // pick improves lie close together, in few chunks of few waves.
    const int par = step & 1;
#pragma unroll
    for (int i = 0; i < RL; ++i) {
      const int q0 = w + i * kWaves;
      if (q0 < nch) {
        const int j0 = q0 * kRowChunk + 4 * lane;     // this lane's four targets
        const f32x4 bo = *reinterpret_cast<const f32x4*>(sball + j0);
        const f32x4 x = xr[i];
        const unsigned long long m0 = __ballot(x[0] < bo[0]), m1 = __ballot(x[1] < bo[1]);
        const unsigned long long m2 = __ballot(x[2] < bo[2]), m3 = __ballot(x[3] < bo[3]);
        if ((m0 | m1 | m2 | m3) != 0ull) {
          const unsigned long long lt = (1ull << lane) - 1ull;
          const int tot = __popcll(m0) + __popcll(m1) + __popcll(m2) + __popcll(m3);
          int at = 0;
          if (lane == 0) at = atomicAdd(&scnt[par], tot);
          at = __builtin_amdgcn_readlane(at, 0);
#pragma unroll
          for (int c = 0; c < 4; ++c) {
            const unsigned long long mk = c == 0 ? m0 : c == 1 ? m1 : c == 2 ? m2 : m3;
            const int e = at + __popcll(mk & lt);
            if (((mk >> lane) & 1ull) && e < kCapR) {
              lj[e] = j0 + c;
              lbo[e] = bo[c];
              lbn[e] = x[c];
            }
            at += __popcll(mk);
          }
        }
      }
    }
    __syncthreads();
    const int total = scnt[par];
    // Early steps improve many targets; tracking the chain there costs more
    // than it saves, so a step with many hits ends the chain.
    if (total > kTrackMax) chain = kChain;
    if (tid == 0) scnt[par ^ 1] = 0;   // last read in the previous step, next used in the next
    if (total <= kCapR) {
      const int per = (total + kWaves - 1) / kWaves;
      const int e0 = min(total, w * per);
      apply(e0, min(total, e0 + per) - e0, true);
    } else {
      // Dense step (early in the greedy): the list is built and applied in
      // rounds of kCapR entries, each entry's place fixed by the hit counts
      // of the chunks before it, and every round is shared evenly by the
      // waves.  b keeps its old values until the last round (the hit test is
      // repeated each round), then takes the new ones.
      for (int q0 = w; q0 < nch; q0 += kWaves) {
        const int j0 = q0 * kRowChunk + 4 * lane;
        const f32x4 bo = *reinterpret_cast<const f32x4*>(sball + j0);
        const f32x4 x = row[q0 * (kRowChunk / 4) + lane];
        const int c = __popcll(__ballot(x[0] < bo[0])) + __popcll(__ballot(x[1] < bo[1])) +
                      __popcll(__ballot(x[2] < bo[2])) + __popcll(__ballot(x[3] < bo[3]));
        if (lane == 0) schunk[q0] = c;
      }
      __syncthreads();
      if (w == 0) {
        // Exclusive prefix of the chunk counts, two chunks a lane.
        const int c0 = 2 * lane < nch ? schunk[2 * lane] : 0;
        const int c1 = 2 * lane + 1 < nch ? schunk[2 * lane + 1] : 0;
        const int incl = wave_scan_incl(c0 + c1);
        if (2 * lane < nch) schunk[2 * lane] = incl - c0 - c1;
        if (2 * lane + 1 < nch) schunk[2 * lane + 1] = incl - c1;
      }
      __syncthreads();
      for (int r0 = 0; r0 < total; r0 += kCapR) {
        for (int q0 = w; q0 < nch; q0 += kWaves) {
          const int j0 = q0 * kRowChunk + 4 * lane;
          const f32x4 bo = *reinterpret_cast<const f32x4*>(sball + j0);
          const f32x4 x = row[q0 * (kRowChunk / 4) + lane];
          int at = schunk[q0] - r0;
          for (int c = 0; c < 4; ++c) {
            const bool hit = x[c] < bo[c];
            const unsigned long long mk = __ballot(hit);
            const int e = at + __popcll(mk & ((1ull << lane) - 1ull));
            if (hit && e >= 0 && e < kCapR) {
              lj[e] = j0 + c;
              lbo[e] = bo[c];
              lbn[e] = x[c];
            }
            at += __popcll(mk);
          }
        }
        __syncthreads();
        const int m = min(kCapR, total - r0);
        const int per = (m + kWaves - 1) / kWaves;
        const int e0 = min(m, w * per);
        apply(e0, min(m, e0 + per) - e0, false);
        __syncthreads();
      }
      for (int q0 = w; q0 < nch; q0 += kWaves) {
        const int j0 = q0 * kRowChunk + 4 * lane;
        f32x4 b = *reinterpret_cast<const f32x4*>(sball + j0);
        const f32x4 x = row[q0 * (kRowChunk / 4) + lane];
#pragma unroll
        for (int c = 0; c < 4; ++c) b[c] = x[c] < b[c] ? x[c] : b[c];
        *reinterpret_cast<f32x4*>(sball + j0) = b;
      }
    }

    // The next candidate, r_(chain+1), and its row for the next step if it
    // is confirmed: issued after the step's own loads so that none of their
    // waits includes it.
    int rn = -1;
#pragma unroll
    for (int c = 0; c < kChain; ++c)
      if (c == chain) rn = rc[c];
    if (kSpec && rn >= 0) {
#pragma unroll
      for (int c = 0; c < kChain; ++c)
        if (live(c)) {
          const long long d = wave_sum_i64(dr[c]);
          if (lane == 0) sdr[w][c] = d;
        }
      const f32x4* rowr = reinterpret_cast<const f32x4*>(a.T + size_t(rn) * a.ldt);
#pragma unroll
      for (int i = 0; i < RL; ++i)
        if (w + i * kWaves < nch) xr2[i] = rowr[(w + i * kWaves) * (kRowChunk / 4) + lane];
    }
    // The waves' partial gains, added in wave order by wave 0.  With one
    // column group wave 0 then publishes the candidate on its own (the next
    // step begins with a barrier); with two the general publish reads every
    // column after a barrier.
#pragma unroll
    for (int q = 0; q < NG; ++q) {
      red[tid] = g[q];
      __syncthreads();
      if (tid < 64 && q * 64 + tid < cnt) {
        const int c = q * 64 + tid;
        long long s = sG[c];
#pragma unroll
        for (int r = 0; r < kWaves; ++r) s += red[r * 64 + tid];
        sG[c] = s;
      }
      if (NG > 1) __syncthreads();
    }
    if (blk == 0) {
      dobj = wave_sum_i64(dobj);
      if (lane == 0) sLw[w] += dobj;
      obj_step = step;
    }

    // The lower bounds on the candidates' gains after the step, the same in
    // every block: when the next candidate's truncated gain beats its bound
    // on all others, it is the next winner.
    bool next = false;
    if (kSpec && rn >= 0) {
#pragma unroll
      for (int c = 0; c < kChain; ++c)
        if (live(c))
#pragma unroll
          for (int q = 0; q < kWaves; ++q) acc[c] += sdr[q][c];
      long long gr = 0;
      unsigned long long u = 0ull;
#pragma unroll
      for (int c = 0; c < kChain; ++c)
        if (c == chain) {
          gr = acc[c];
          u = ub[c];
        }
      next = step + 1 < a.k_end && gr > 0 && (pack_key(fx_to_double(gr, S), rn) >> kIndexBits) > u;
    }
    if (step + 1 < a.k && !next) {
      if (kSpec)
        publish_rows(sG, ssel, lo, cnt, S, cand_slot(a.cand, xc & 1, blk), epoch_of(xc));
      else
        publish_argmax(sG, ssel, lo, cnt, S, cand_slot(a.cand, xc & 1, blk), epoch_of(xc), sg, si);
    }
    predicted = next;
    tpred = rn;
    chain += next ? 1 : 0;
  }
  __syncthreads();
  if (blk == 0 && tid == 0 && obj_step >= 0 && a.step_obj) {
    long long L = 0;
#pragma unroll
    for (int q = 0; q < kWaves; ++q) L += sLw[q];
    a.step_obj[obj_step] = fx_to_double(L, S);
  }
  // Hand the state over to the launch that continues (the last step
  // published the candidates of the next exchange).
  if (a.k_end < a.k) {
    for (int i = tid; i < cnt; i += kBlock) {
      a.ho_gain[lo + i] = sG[i];
      a.ho_sel[lo + i] = ssel[i];
    }
    if (blk == 0) {
      for (int j = tid; j < a.ldt; j += kBlock) a.ho_b[j] = sball[j];
      if (tid == 0) {
        long long L = 0;
#pragma unroll
        for (int q = 0; q < kWaves; ++q) L += sLw[q];
        a.ho_misc[0] = L;
        a.ho_misc[1] = xc;
      }
    }
  }
}

__global__ __launch_bounds__(kBlock) void sgs_inc_kernel(IncDev a) { inc_body(a, blockIdx.x, gridDim.x); }

template <int NG, int RL>
__global__ __launch_bounds__(kBlock) void sgs_rows_kernel(IncDev a) { rows_body<NG, RL>(a, blockIdx.x, gridDim.x); }

// ---------------------------------------------------------------------------
// The rows schedule's early steps.
//
// A pick early in the greedy lowers the best cost of thousands of targets
// (about a fifth of all targets in each of the first 16 steps at N = 16384),
// and the rows kernel has every block read its own 64 columns of each such
// target's row of the cost: a 256-byte piece of thousands of rows per block
// and step, which the memory system serves at well under half its streaming
// rate.  Here the step's hits are split instead.  Every block still finds all
// of them from the winner's row of T (each block keeps every best cost);
// block b then takes the b-th equal share of the hit list (in target order),
// reads its targets' whole rows of the cost (contiguous, 64 KB each at
// N = 16384) and sums the gain changes of all n columns, the same 64-bit
// fixed-point terms as the rows kernel, into registers.  It writes the sums
// to its row of a [blocks] x [n] table, with the objective's change of its
// share after them, and raises its flag for the step; every block then adds,
// for its own columns, the rows of all blocks whose share was not empty.  The
// gains are the same integers as in the rows kernel (integer sums do not
// depend on their order), so the picks are the same.
//
// The kernel runs while a step improves at least kEarlyMinHits targets, and
// at most until the lists take over (or to the end), then hands its state
// to the rows kernel as the rows kernel hands it to the list kernel, with the
// next step in ho_misc[2].  One column group only (n <= kEarlyMaxN): a
// thread holds the changes of n / kBlock columns.
constexpr int kEarlyMaxN = kRowChunk * kWaves * 8;    // 16384, the one-group rows kernel's reach
constexpr int kEarlyCols = kEarlyMaxN / kBlock;       // columns per thread: 32
constexpr int kEarlyPass = 8;                         // of which one pass over the share sums
constexpr int kEarlyDepth = 4;                        // rows whose loads are in flight
constexpr int kEarlyShare = 64;                       // hits a block takes per step at most (W <= 64)
constexpr int kEarlyMinHits = 512;                    // steps with fewer hits go back to the rows kernel

int early_ldp(int64_t n) { return int((n + 1 + 63) / 64 * 64); }
bool early_for(int64_t n, int W) { return n <= kEarlyMaxN && W <= 64; }

__global__ __launch_bounds__(kBlock) void sgs_early_kernel(IncDev a) {
  extern __shared__ unsigned long long smem[];
  constexpr int RL = 8;                               // chunk loads per wave: n <= kRowChunk kWaves RL
  const int blk = blockIdx.x, nb = gridDim.x;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int lo = blk * a.W;
  const int cnt = max(0, min(a.n, lo + a.W) - lo);
  long long* sG = reinterpret_cast<long long*>(smem);             // [W] running gains (W rounded up to even)
  float* sball = reinterpret_cast<float*>(sG + ((a.W + 1) & ~1));  // [ldt] b_j; -inf past n
  unsigned char* ssel = reinterpret_cast<unsigned char*>(sball + a.ldt);   // [W] chosen columns
  __shared__ long long red[kBlock];
  __shared__ unsigned long long su[kWaves];
  __shared__ unsigned long long sk1[kMaxBlocks], sk2[kMaxBlocks];
  __shared__ int sflag;
  __shared__ int schunk[kEarlyMaxN / kRowChunk];     // hits per chunk of the winner's row, then their offsets
  __shared__ int stot;
  __shared__ int sj[kEarlyShare];                     // the block's share: target, old and new best cost,
  __shared__ float sbo[kEarlyShare], sbn[kEarlyShare];
  __shared__ double svs[kEarlyShare];                 // and its capacity scaled for fx_diff

  const int S = *a.scale;
  for (int j = tid; j < a.ldt; j += kBlock) sball[j] = j < a.n ? a.c0 : -__builtin_inff();
  for (int i = tid; i < cnt; i += kBlock) ssel[i] = 0;
  init_gains(a, sG, lo, cnt, red);
  // Block 0 keeps the objective (in wave 1 after the start).
  long long L = 0;
  if (blk == 0) {
    const long long x = fx_capacity_part(a.v, a.n, a.c0, S);
    L = block_sum_i64(x, red);
  }
  publish_rows(sG, ssel, lo, cnt, S, cand_slot(a.cand, 0, blk), epoch_of(0));

  const int nch = a.ldt / kRowChunk;
  const int k_stop = a.k_end;                         // steps [0, k_stop) at most
  long long* mine = a.epart + size_t(blk) * a.ldp;
  int xc = 0;
  for (int step = 0; step < k_stop; ++step) {
    const int tw = read_winner_rows(cand_slot(a.cand, xc & 1, 0), epoch_of(xc), nb, a.abort, a.poll_limit, su,
                                    &sflag, sk1, sk2);
    ++xc;
    if (tw < 0) return;
    const int t = min(tw, a.n - 1);
    if (t >= lo && t < lo + cnt && tid == 0) {
      ssel[t - lo] = 1;
      a.selected[step] = t;
      if (a.step_gain) a.step_gain[step] = fx_to_double(sG[t - lo], S);
    }

    // The winner's row of T: every wave its chunks, all loads in flight.
    const f32x4* row = reinterpret_cast<const f32x4*>(a.T + size_t(t) * a.ldt);
    f32x4 xr[RL];
#pragma unroll
    for (int i = 0; i < RL; ++i)
      if (w + i * kWaves < nch) xr[i] = row[(w + i * kWaves) * (kRowChunk / 4) + lane];
    // Hits per chunk, their offsets in target order, and the total.
#pragma unroll
    for (int i = 0; i < RL; ++i) {
      const int q0 = w + i * kWaves;
      if (q0 < nch) {
        const f32x4 bo = *reinterpret_cast<const f32x4*>(sball + q0 * kRowChunk + 4 * lane);
        const f32x4 x = xr[i];
        const int c = __popcll(__ballot(x[0] < bo[0])) + __popcll(__ballot(x[1] < bo[1])) +
                      __popcll(__ballot(x[2] < bo[2])) + __popcll(__ballot(x[3] < bo[3]));
        if (lane == 0) schunk[q0] = c;
      }
    }
    __syncthreads();
    if (w == 0) {
      const int c0 = 2 * lane < nch ? schunk[2 * lane] : 0;
      const int c1 = 2 * lane + 1 < nch ? schunk[2 * lane + 1] : 0;
      const int incl = wave_scan_incl(c0 + c1);
      if (2 * lane < nch) schunk[2 * lane] = incl - c0 - c1;
      if (2 * lane + 1 < nch) schunk[2 * lane + 1] = incl - c1;
      if (lane == 63) stot = incl;
    }
    __syncthreads();
    const int H = stot;
    const int per = (H + nb - 1) / nb;                // at most ceil(n / nb) <= W
    const int e_lo = min(H, blk * per), e_hi = min(H, e_lo + per);
    const int nshare = per > 0 ? (H + per - 1) / per : 0;   // blocks with a share
    // The block's share of the list; every target's new best cost; assign
    // for the own targets.
#pragma unroll
    for (int i = 0; i < RL; ++i) {
      const int q0 = w + i * kWaves;
      if (q0 < nch) {
        const int j0 = q0 * kRowChunk + 4 * lane;
        f32x4 bo = *reinterpret_cast<const f32x4*>(sball + j0);
        const f32x4 x = xr[i];
        int at = schunk[q0];
#pragma unroll
        for (int c = 0; c < 4; ++c) {
          const bool hit = x[c] < bo[c];
          const unsigned long long mk = __ballot(hit);
          const int e = at + __popcll(mk & ((1ull << lane) - 1ull));
          if (hit) {
            const int j = j0 + c;
            if (e >= e_lo && e < e_hi) {
              sj[e - e_lo] = j;
              sbo[e - e_lo] = bo[c];
              sbn[e - e_lo] = x[c];
              svs[e - e_lo] = fx_scale(double(a.v[j]), S);
            }
            if (a.assign && unsigned(j - lo) < unsigned(cnt)) a.assign[j] = t;
            bo[c] = x[c];
          }
          at += __popcll(mk);
        }
        *reinterpret_cast<f32x4*>(sball + j0) = bo;
      }
    }
    __syncthreads();

    // The share's rows of the cost, in passes over kEarlyPass of the
    // thread's columns at a time, with the next kEarlyDepth rows' loads in
    // flight while a row is summed.  Loads past the share repeat its last
    // row and columns past n read column n - 1, so that every load is issued
    // unconditionally (the waits then count them exactly); such values are
    // never summed.
    const int nsh = e_hi - e_lo;
    if (nsh > 0) {
#pragma unroll 1
      for (int h = 0; h < kEarlyCols; h += kEarlyPass) {
        long long acc[kEarlyPass];
        float buf[kEarlyDepth][kEarlyPass];
#pragma unroll
        for (int q = 0; q < kEarlyPass; ++q) acc[q] = 0;
        auto load = [&](float* dst, int e) {
          const float* r = a.C + size_t(sj[min(e, nsh - 1)]) * a.n;
#pragma unroll
          for (int q = 0; q < kEarlyPass; ++q)
            dst[q] = __builtin_nontemporal_load(r + min(tid + kBlock * (h + q), a.n - 1));
        };
#pragma unroll
        for (int d = 0; d < kEarlyDepth; ++d) load(buf[d], d);
        for (int e = 0; e < nsh; e += kEarlyDepth) {
#pragma unroll
          for (int d = 0; d < kEarlyDepth; ++d) {
            float x[kEarlyPass];
#pragma unroll
            for (int q = 0; q < kEarlyPass; ++q) x[q] = buf[d][q];
            load(buf[d], e + d + kEarlyDepth);
            if (e + d < nsh) {
              const float bo = sbo[e + d], bn = sbn[e + d];
              const double vs = svs[e + d];
#pragma unroll
              for (int q = 0; q < kEarlyPass; ++q) {
                // A column that cost at least the old best contributes 0
                // before and after.
                if (tid + kBlock * (h + q) < a.n && x[q] < bo)
                  acc[q] += fx_diff(vs, fmaxf(bn - x[q], 0.f), bo - x[q]);
              }
            }
          }
        }
#pragma unroll
        for (int q = 0; q < kEarlyPass; ++q) {
          const int c = tid + kBlock * (h + q);
          if (c < a.n) put(reinterpret_cast<unsigned long long*>(mine + c), (unsigned long long)acc[q]);
        }
      }
      if (w == 0) {
        long long d = 0;
        if (lane < nsh) d = fx_diff(svs[lane], sbn[lane], sbo[lane]);
        d = wave_sum_i64(d);
        if (lane == 0) put(reinterpret_cast<unsigned long long*>(mine + a.n), (unsigned long long)d);
      }
      __builtin_amdgcn_s_waitcnt(0x0F70);   // vmcnt(0): this wave's stores are done
    }
    __syncthreads();
    if (nsh > 0 && tid == 0) put(lens_slot(a.lens, blk), (unsigned long long)(step + 1));

    // Every share's sums, once its block has raised its flag for the step.
    if (tid == 0) sflag = 0;
    __syncthreads();
    if (tid < nshare) {
      unsigned long long f;
      const unsigned long long want = (unsigned long long)(step + 1);
      if (!wait_slot(lens_slot(a.lens, tid), a.abort, a.poll_limit, [want](unsigned long long v) { return v == want; },
                     f))
        sflag = 1;
    }
    __syncthreads();
    if (sflag) return;
    {
      // All of a thread's loads are issued before any is used (a row past
      // nshare, or a column past cnt, is read from a valid address and not
      // summed).
      constexpr int kRead = 16;                       // loads in flight: two rounds for 256 blocks
      const int col = min(lo + min(lane, max(cnt - 1, 0)), a.n - 1);
      long long s = 0;
      for (int b0 = 0; b0 < nshare; b0 += kRead * kWaves) {
        unsigned long long x[kRead];
#pragma unroll
        for (int m = 0; m < kRead; ++m)
          x[m] = get(reinterpret_cast<const unsigned long long*>(
              a.epart + size_t(min(b0 + w + kWaves * m, nb - 1)) * a.ldp + col));
#pragma unroll
        for (int m = 0; m < kRead; ++m)
          if (lane < cnt && b0 + w + kWaves * m < nshare) s += (long long)x[m];
      }
      red[tid] = s;
    }
    if (blk == 0 && w == 1) {
      constexpr int kRead = kMaxBlocks / 64;
      unsigned long long x[kRead];
#pragma unroll
      for (int m = 0; m < kRead; ++m)
        x[m] = get(reinterpret_cast<const unsigned long long*>(a.epart + size_t(min(lane + 64 * m, nb - 1)) * a.ldp + a.n));
      long long s = 0;
#pragma unroll
      for (int m = 0; m < kRead; ++m)
        if (lane + 64 * m < nshare) s += (long long)x[m];
      L += wave_sum_i64(s);
      if (lane == 0 && a.step_obj) a.step_obj[step] = fx_to_double(L, S);
    }
    __syncthreads();
    if (tid < 64 && tid < cnt) {
      long long s = sG[tid];
#pragma unroll
      for (int r = 0; r < kWaves; ++r) s += red[r * 64 + tid];
      sG[tid] = s;
    }
    // The next exchange's candidates (wave 0, which also wrote the gains),
    // unless this was the last step.
    if (step + 1 < a.k) publish_rows(sG, ssel, lo, cnt, S, cand_slot(a.cand, xc & 1, blk), epoch_of(xc));
    if (step + 1 == k_stop || H < kEarlyMinHits) {
      // Hand over before step + 1.
      __syncthreads();
      for (int i = tid; i < cnt; i += kBlock) {
        a.ho_gain[lo + i] = sG[i];
        a.ho_sel[lo + i] = ssel[i];
      }
      if (blk == 0) {
        for (int j = tid; j < a.ldt; j += kBlock) a.ho_b[j] = sball[j];
        if (tid == 64) {
          a.ho_misc[0] = L;
          a.ho_misc[1] = xc;
          a.ho_misc[2] = step + 1;
        }
      }
      return;
    }
  }
}

// ---------------------------------------------------------------------------
// The rows schedule's later steps from candidate lists.
//
// Best costs only fall, so a pair (candidate c, target j) with C(c, j) >= b_j
// never changes a gain again.  After kListStep steps few pairs are left (at
// N = 16384, K = 1638: 44 per candidate on average, at most 5391 among one
// block's 64 candidates).  The rows schedule then runs in two launches: the
// first stops after kListStep steps and hands its state over (best costs,
// running gains, chosen flags, objective, exchange count); list_build_kernel
// writes every candidate's pairs (target, cost, the target's capacity) into
// a list of at most kListMax entries; sgs_list_kernel runs the remaining steps
// from the lists.  Per step a block reads the winner's list (a few KB, from
// L2 for all but the first block of an XCD) instead of its 64 KB row of T, and
// keeps the block's own pairs (up to kEntMax) in LDS indexed by target: the
// thread that lowers a target's best cost from the winner's list also adds
// the changes of the own candidates paired with that target, instead of
// reading each hit row's segment over its columns from memory.  The terms are the fixed-point terms of the rows of T, so the picks
// are the same.  When the lists do not fit (a candidate with more than
// kListMax pairs, or a block with more than kEntMax), the build raises lfail
// and the rows kernel continues instead (its launch is gated on lfail).
constexpr int kListStep = 128;                        // steps before the lists
constexpr int kListSlots = 256;                       // per candidate: a header and kListMax pairs
constexpr int kListMax = kListSlots - 1;
constexpr int kListMaxN = kRowChunk * kWaves * 8;     // 16384, the one-group rows kernel's reach
constexpr int kOwnSets = 16;                          // own pairs a thread places at the start
constexpr int kEntMax = kOwnSets * kBlock;            // own pairs a block holds: 8192

bool lists_for(int64_t n, int64_t k, int W) { return n <= kListMaxN && W <= 64 && k > kListStep; }

// The list kernel's LDS: the best costs, the own pairs' first index per
// target (16 bits each, targets 0 .. n), their costs and candidates.
__host__ __device__ __forceinline__ int list_off_words(int n) { return (n + 2) / 2; }
size_t list_lds(int64_t n) {
  return size_t(rows_ldt(n)) * 4 + size_t(list_off_words(int(n))) * 4 + size_t(kEntMax) * 5;
}

// One wave per candidate: its pairs from its row of T against the handed
// over best costs.  Also counts the pairs of each block of the list kernel.
__global__ __launch_bounds__(256) void list_build_kernel(IncDev a) {
  if (*a.abort) return;
  const int lane = threadIdx.x & 63;
  const int c = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (c >= a.n) return;
  const f32x4* row = reinterpret_cast<const f32x4*>(a.T + size_t(c) * a.ldt);
  const f32x4* bb = reinterpret_cast<const f32x4*>(a.ho_b);
  unsigned long long* dst = a.lists + size_t(c) * (2 * kListSlots);
  const int nch = a.ldt / kRowChunk;
  const unsigned long long lt = (1ull << lane) - 1ull;
  int m = 0;
  for (int q0 = 0; q0 < nch; q0 += 8) {
    f32x4 x[8], b[8];
#pragma unroll
    for (int u = 0; u < 8; ++u)
      if (q0 + u < nch) {
        x[u] = __builtin_nontemporal_load(row + (q0 + u) * (kRowChunk / 4) + lane);   // T is read once here
        b[u] = bb[(q0 + u) * (kRowChunk / 4) + lane];
      }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      if (q0 + u >= nch) break;
#pragma unroll
      for (int cc = 0; cc < 4; ++cc) {
        const bool hit = x[u][cc] < b[u][cc];         // never past n, where b = -inf
        const unsigned long long mk = __ballot(hit);
        if (hit) {
          const int pos = m + __popcll(mk & lt);
          const int j = (q0 + u) * kRowChunk + 4 * lane + cc;
          if (pos < kListMax) {
            dst[2 * (1 + pos)] = (unsigned long long)(unsigned)j | ((unsigned long long)__float_as_uint(x[u][cc]) << 32);
            dst[2 * (1 + pos) + 1] = (unsigned long long)__float_as_uint(a.v[j]);
          }
        }
        m += __popcll(mk);
      }
    }
  }
  if (lane == 0) {
    dst[0] = (unsigned long long)m;
    const unsigned int tot = atomicAdd(a.lblock + c / a.W, unsigned(m)) + unsigned(m);
    if (m > kListMax || tot > unsigned(kEntMax)) atomicOr(a.lfail, 1u);
  }
}

// The greedy's steps kListStep .. k - 1 from the lists (one block of eight
// waves per compute unit, block b owning candidates [b W, (b + 1) W) as in
// the rows kernel, W <= 64).
//
// Predicted steps, as in the rows kernel but up to kListChain in a row: after
// an exchange the chain r_1, r_2, ... are the best candidates of distinct
// blocks in key order (the winner's block left out).  r_m is the next winner
// when a lower bound on its gain (its key, plus its exact changes since the
// exchange) beats the key of r_(m+1) and the second-best keys of the
// winner's block and of r_1 .. r_m's blocks.  Every block holds the lists of
// the exchange's winner and of the chain in registers, so it sums the chain's
// changes itself (an entry's target was hit when its best cost fell in the
// step: the same terms as the owner applies), and a predicted step finds its
// winner's hits in registers: no exchange and no memory latency.
//
// A step: the waves holding the winner's list lower the best costs of its
// hits in LDS; after a barrier every thread compares its own pairs' and its
// chain entries' last seen best costs with LDS and sums the changes (own
// candidates into LDS, chain candidates per wave); after a second barrier
// every thread updates the chain bounds and decides whether the next step is
// predicted, and wave 0 folds the gains and publishes when it is not.
constexpr int kListChain = 3;                         // predicted steps in a row at most
constexpr int kSlotsPerSet = kBlock / kListSlots;    // lists the block's threads hold side by side
constexpr int kListSets = (kListChain + kSlotsPerSet) / kSlotsPerSet;   // chain list entries a thread holds

__global__ __launch_bounds__(kBlock) void sgs_list_kernel(IncDev a) {
  if (*a.lfail || *a.abort) return;
  extern __shared__ unsigned long long smem[];
  const int blk = blockIdx.x, nb = gridDim.x;
  const int tid = threadIdx.x, lane = tid & 63;
  const int lo = blk * a.W;
  const int cnt = max(0, min(a.n, lo + a.W) - lo);
  float* sball = reinterpret_cast<float*>(smem);                   // [ldt] best costs
  // The block's own pairs by target: pairs [off(j), off(j + 1)) have target
  // j, each with its cost and its candidate (own index); off as 16-bit
  // values, two to a word.
  unsigned int* soffw = reinterpret_cast<unsigned int*>(sball + a.ldt);   // [n / 2 + 1]
  float* spc = reinterpret_cast<float*>(soffw + list_off_words(a.n));     // [kEntMax]
  unsigned char* spk = reinterpret_cast<unsigned char*>(spc + kEntMax);   // [kEntMax]
  auto off = [&](int j) { return int((soffw[j >> 1] >> ((j & 1) * 16)) & 0xffffu); };
  __shared__ long long sG[64];
  __shared__ unsigned char ssel[64];
  __shared__ unsigned long long sdelta[2][64];                      // own gain changes, by step parity
  __shared__ int soff[65];                                          // each own candidate's first pair
  __shared__ int swt[kWaves];
  __shared__ unsigned long long su[kWaves], sk1[kMaxBlocks], sk2[kMaxBlocks];
  __shared__ int sflag;
  __shared__ unsigned long long sL;                                 // objective (block 0)
  __shared__ unsigned long long sacc[kListChain + 1];               // chain changes since the exchange
  const int S = *a.scale;

  for (int j = tid; j < a.ldt; j += kBlock) sball[j] = a.ho_b[j];
  for (int i = tid; i < list_off_words(a.n); i += kBlock) soffw[i] = 0u;
  if (tid < 64) {
    ssel[tid] = tid < cnt ? a.ho_sel[lo + tid] : 1;
    sG[tid] = tid < cnt ? a.ho_gain[lo + tid] : 0;
    sdelta[0][tid] = sdelta[1][tid] = 0ull;
    // Where each own candidate's pairs start among the block's.
    const int m = tid < cnt ? min(int(a.lists[size_t(lo + tid) * (2 * kListSlots)]), kListMax) : 0;
    const int incl = wave_scan_incl(m);
    soff[tid + 1] = incl;
    if (tid == 0) soff[0] = 0;
  }
  if (tid == 0) sL = (unsigned long long)(blk == 0 ? a.ho_misc[0] : 0);
  __syncthreads();
  const int npairs = min(soff[64], kEntMax);
  {
    // Pair p = q kBlock + tid of the block (candidates in order, each with
    // its list's entries): its candidate by a search of soff, its entry from
    // the list; all loads issued before any is used.
    int ci[kOwnSets], e[kOwnSets];
#pragma unroll
    for (int q = 0; q < kOwnSets; ++q) {
      const int pq = q * kBlock + tid;
      int c = 0;
#pragma unroll
      for (int st = 32; st > 0; st >>= 1)
        if (c + st < 64 && soff[c + st] <= pq) c += st;
      ci[q] = c;
      e[q] = pq < npairs ? 1 + pq - soff[c] : 0;
    }
    uint2 ev[kOwnSets];
#pragma unroll
    for (int q = 0; q < kOwnSets; ++q)
      ev[q] = reinterpret_cast<const uint2*>(a.lists + size_t(min(lo + ci[q], a.n - 1)) * (2 * kListSlots))[2 * e[q]];
    // Pairs per target (16-bit counts, two to a word), their inclusive
    // prefix over the targets, then each pair placed at its target's end,
    // which moves down to the target's first pair.
#pragma unroll
    for (int q = 0; q < kOwnSets; ++q)
      if (q * kBlock + tid < npairs) {
        const int j = min(int(ev[q].x), a.n - 1);
        atomicAdd(&soffw[j >> 1], 1u << ((j & 1) * 16));
      }
    __syncthreads();
    const int per = (list_off_words(a.n) + kBlock - 1) / kBlock;   // words a thread scans
    int sum = 0;
    for (int i = tid * per; i < min((tid + 1) * per, list_off_words(a.n)); ++i)
      sum += int(soffw[i] & 0xffffu) + int(soffw[i] >> 16);
    int run = block_inclusive_scan(sum, swt) - sum;
    for (int i = tid * per; i < min((tid + 1) * per, list_off_words(a.n)); ++i) {
      const unsigned int wv = soffw[i];
      const int lo16 = run + int(wv & 0xffffu);
      const int hi16 = lo16 + int(wv >> 16);
      soffw[i] = unsigned(lo16) | (unsigned(hi16) << 16);
      run = hi16;
    }
    __syncthreads();
#pragma unroll
    for (int q = 0; q < kOwnSets; ++q)
      if (q * kBlock + tid < npairs) {
        const int j = min(int(ev[q].x), a.n - 1);
        const unsigned int sh = (j & 1) * 16;
        const int pos = int((atomicSub(&soffw[j >> 1], 1u << sh) >> sh) & 0xffffu) - 1;
        spc[pos] = __uint_as_float(ev[q].y);
        spk[pos] = (unsigned char)ci[q];
      }
    __syncthreads();
  }

  // Chain slots: 0 the exchange's winner, m = 1 .. kListChain the candidate
  // r_m (-1 past the last), with lower bounds on their gains at the exchange
  // and the key bits they must beat.  Entry set q of a thread is entry
  // tid % kListSlots of slot q kSlotsPerSet + tid / kListSlots's list:
  // target, cost, scaled capacity, and the target's best cost as last seen
  // (entry 0 of a list is its header).
  const int half = tid / kListSlots, ent = tid % kListSlots;
  int rc[kListChain + 1];
  long long acc[kListChain + 1];
  unsigned long long ub[kListChain + 1];
  int ej[kListSets];
  float ec[kListSets], eb[kListSets];
  double evs[kListSets];
  bool eok[kListSets];
#pragma unroll
  for (int m = 0; m <= kListChain; ++m) {
    rc[m] = -1;
    acc[m] = 0;
    ub[m] = 0ull;
  }
#pragma unroll
  for (int q = 0; q < kListSets; ++q) {
    ej[q] = 0;
    ec[q] = eb[q] = 0.f;
    evs[q] = 0.0;
    eok[q] = false;
  }
  int xc = int(a.ho_misc[1]);
  int obj_step = a.k_begin - 1;
  bool predicted = false;
  int pos = 0;                 // the step's place in the chain (0: after an exchange)
  for (int step = a.k_begin; step < a.k; ++step) {
    int t = -1;
    const int par = step & 1;
    if (!predicted) {
      const int tw = read_winner_rows(cand_slot(a.cand, xc & 1, 0), epoch_of(xc), nb, a.abort, a.poll_limit, su,
                                      &sflag, sk1, sk2);
      ++xc;
      if (tw < 0) break;
      t = min(tw, a.n - 1);
      if (tid <= kListChain) sacc[tid] = 0ull;
      // The chain from the exchange's keys (every wave the same).
      const int bt = block_of(a, t);
      unsigned long long kq[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int bq = lane + 64 * q;
        kq[q] = (bq < nb && bq != bt) ? sk1[bq] : 0ull;
      }
      unsigned long long u2 = sk2[bt];
      rc[0] = t;
#pragma unroll
      for (int m = 1; m <= kListChain + 1; ++m) {
        const unsigned long long kr = wave_max_u64(max(max(kq[0], kq[1]), max(kq[2], kq[3])));
        const bool real = kr > kNoCandidate && (m == 1 || rc[m - 1] >= 0);
        const int r = real ? int(kIndexMask - (kr & kIndexMask)) : -1;
        const int br = real ? block_of(a, r) : -1;
        if (m >= 2) ub[m - 1] = max(real ? kr : 0ull, u2) >> kIndexBits;
        if (m <= kListChain) {
          rc[m] = r;
          acc[m] = real ? key_gain_floor(kr, S) : 0;
          if (real) u2 = max(u2, sk2[br]);
#pragma unroll
          for (int q = 0; q < 4; ++q) kq[q] = (lane + 64 * q) == br ? 0ull : kq[q];
        }
      }
      pos = 0;
      // The lists of the winner and of the chain, all loads in flight
      // together (plain loads: the lists are fixed since the build).
      uint4 hv[kListSets], ev[kListSets];
#pragma unroll
      for (int q = 0; q < kListSets; ++q) {
        const int sl = q * kSlotsPerSet + half;
        int r = -1;
#pragma unroll
        for (int m = 0; m <= kListChain; ++m)
          if (m == sl) r = rc[m];
        const uint4* lw = reinterpret_cast<const uint4*>(a.lists + size_t(max(r, 0)) * (2 * kListSlots));
        hv[q] = lw[0];
        ev[q] = lw[ent];
        eok[q] = r >= 0;
      }
#pragma unroll
      for (int q = 0; q < kListSets; ++q) {
        eok[q] = eok[q] && ent >= 1 && ent <= min(int(hv[q].x), kListMax);
        ej[q] = eok[q] ? min(int(ev[q].x), a.n - 1) : 0;
        ec[q] = __uint_as_float(ev[q].y);
        evs[q] = fx_scale(double(__uint_as_float(ev[q].z)), S);
      }
      // The entries' best costs before the step's hits lower them.
#pragma unroll
      for (int q = 0; q < kListSets; ++q) eb[q] = eok[q] ? sball[ej[q]] : 0.f;
      __syncthreads();
    } else {
#pragma unroll
      for (int m = 1; m <= kListChain; ++m)
        if (m == pos) t = rc[m];
    }
    if (blk == 0 && tid == 0 && obj_step >= 0 && a.step_obj) a.step_obj[obj_step] = fx_to_double((long long)sL, S);
    if (t >= lo && t < lo + cnt && tid == 0) {
      ssel[t - lo] = 1;
      a.selected[step] = t;
      if (a.step_gain) a.step_gain[step] = fx_to_double(sG[t - lo], S);
    }
    // The winner's hits, from the waves that hold its list (slot pos): each
    // lowers its target's best cost (a target appears once in a list).
    long long dobj = 0;
#pragma unroll
    for (int q = 0; q < kListSets; ++q) {
      if (q * kSlotsPerSet + half != pos) continue;   // uniform over the wave
      if (eok[q]) {
        const int j = ej[q];
        const float x = ec[q], bo = sball[j];
        if (x < bo) {
          sball[j] = x;
          if (blk == 0) dobj = fx_diff(evs[q], x, bo);
          if (a.assign && unsigned(j - lo) < unsigned(cnt)) a.assign[j] = t;
          // The own candidates with a pair on j: their gain changes, added
          // up in LDS as 64-bit integers.
          const int p1 = off(j + 1);
          for (int p = off(j); p < p1; ++p) {
            const float cv = spc[p];
            if (cv < bo)
              atomicAdd(&sdelta[par][spk[p]], (unsigned long long)fx_diff(evs[q], fmaxf(x - cv, 0.f), bo - cv));
          }
        }
      }
    }
    __syncthreads();
    if (dobj != 0) atomicAdd(&sL, (unsigned long long)dobj);
    obj_step = step;
    // The chain candidates still ahead (slots above pos): their changes in
    // the step, from the entries whose best cost fell, into LDS.
#pragma unroll
    for (int q = 0; q < kListSets; ++q) {
      const int sl = q * kSlotsPerSet + half;
      if (sl <= pos || sl > kListChain) continue;   // uniform over the wave
      long long d = 0;
      if (eok[q]) {
        const float bn = sball[ej[q]], bo = eb[q];
        if (bn < bo) {
          const float cv = ec[q];
          if (cv < bo) d = fx_diff(evs[q], fmaxf(bn - cv, 0.f), bo - cv);
          eb[q] = bn;
        }
      }
      if (__ballot(d != 0)) {
        d = wave_sum_i64(d);
        if (lane == 0) atomicAdd(&sacc[sl], (unsigned long long)d);
      }
    }
    __syncthreads();
    // Wave 0 folds the step's own changes.  A predicted next step starts
    // without a barrier, so its hits add into the other parity's buffer
    // while this one is read and cleared.
    if (tid < 64) {
      if (tid < cnt) sG[tid] += (long long)sdelta[par][tid];
      sdelta[par][tid] = 0ull;
    }
    bool next = false;
    if (pos < kListChain && step + 1 < a.k) {
      int rn = -1;
      long long gr = 0;
      unsigned long long u = 0ull;
#pragma unroll
      for (int m = 1; m <= kListChain; ++m)
        if (m == pos + 1) {
          rn = rc[m];
          gr = acc[m];
          u = ub[m];
        }
      gr += (long long)sacc[pos + 1];
      next = rn >= 0 && gr > 0 && (pack_key(fx_to_double(gr, S), rn) >> kIndexBits) > u;
    }
    // Wave 0 folded the gains itself, so it publishes without a barrier.
    if (step + 1 < a.k && !next) publish_rows(sG, ssel, lo, cnt, S, cand_slot(a.cand, xc & 1, blk), epoch_of(xc));
    predicted = next;
    pos += next ? 1 : 0;
  }
  __syncthreads();
  if (blk == 0 && tid == 0 && obj_step >= 0 && a.step_obj) a.step_obj[obj_step] = fx_to_double((long long)sL, S);
}

// The fixed-point scale of a scene (one block; the sum in the same order as
// every block of the greedy would take it).
__global__ __launch_bounds__(kBlock) void inc_scale_kernel(IncDev a, int* scale) {
  __shared__ double sd[kWaves];
  const int S = fixed_scale(a, sd);
  if (threadIdx.x == 0) *scale = S;
}

// Step-0 gains, every row at b = c0, split over a grid of (column strip,
// row range) blocks so that the pass runs with many more waves in flight than
// the greedy's one block per compute unit: block (b, p) sums rows
// [p R, (p + 1) R) of columns [b W, (b + 1) W) into part[p][column], 64-bit
// fixed point, four waves adding in wave order.  A round covers 64 rows, 16
// per wave.  With WT the round's 64 x 64 tile also goes to T through LDS:
// lane `col` of a wave holds C_tm[j0 .. j0 + 16)[col], i.e. a piece of row
// `col` of T; after a barrier each store instruction writes four rows of T,
// 256 contiguous bytes each (16 lanes of 16 bytes), so every line written is
// whole.  R is a multiple of 16 and rows of T are only written below the
// range's end (n, padding aside, for the last range).
constexpr int kPassThreads = 256;
constexpr int kPassWaves = kPassThreads / 64;
constexpr int kPassRows = 16;
constexpr int kPassTile = kPassWaves * kPassRows;   // rows per round
constexpr int kPassLd = kPassTile + 4;               // LDS row of the tile: 16-byte aligned, banks spread

__host__ __device__ __forceinline__ int pass_rows(int n, int P) {
  return ((n + P - 1) / P + kPassRows - 1) / kPassRows * kPassRows;
}

template <bool WT>
__global__ __launch_bounds__(kPassThreads) void inc_first_pass_kernel(IncDev a, long long* part) {
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int lo = blockIdx.x * a.W, cnt = max(0, min(a.n, lo + a.W) - lo);
  const int R = pass_rows(a.n, a.P), r0 = blockIdx.y * R, r1 = min(a.n, r0 + R);
  const int S = *a.scale;
  __shared__ long long red[kPassThreads];
  __shared__ __attribute__((aligned(16))) float tile[WT ? 64 : 1][WT ? kPassLd : 1];   // [column][row of the round]
  for (int cc = 0; cc < cnt; cc += 64) {
    const bool colok = cc + lane < cnt;
    const int col = lo + cc + lane;
    // The next round's loads are issued before the current round's terms
    // are formed; two accumulators.
    long long g0 = 0, g1 = 0;
    float xn[kPassRows], vn[kPassRows];
    auto load = [&](int j0) {
#pragma unroll
      for (int u = 0; u < kPassRows; ++u) {
        const int j = j0 + u;
        xn[u] = (colok && j < r1) ? __builtin_nontemporal_load(a.C + size_t(j) * a.n + col) : a.c0;
        vn[u] = j < r1 ? a.v[j] : 0.f;
      }
    };
    load(r0 + w * kPassRows);
    for (int jr = r0; jr < r1; jr += kPassTile) {   // uniform over the block
      const int j0 = jr + w * kPassRows;
      float x[kPassRows], vj[kPassRows];
#pragma unroll
      for (int u = 0; u < kPassRows; ++u) {
        x[u] = xn[u];
        vj[u] = vn[u];
      }
      if (jr + kPassTile < r1) load(j0 + kPassTile);   // rows past r1 load as zero terms
#pragma unroll
      for (int u = 0; u < kPassRows; u += 2) {
        g0 += fx(double(vj[u]) * double(fmaxf(a.c0 - x[u], 0.f)), S);
        g1 += fx(double(vj[u + 1]) * double(fmaxf(a.c0 - x[u + 1], 0.f)), S);
      }
      if (WT) {
#pragma unroll
        for (int q = 0; q < kPassRows / 4; ++q)
          *reinterpret_cast<f32x4*>(&tile[lane][w * kPassRows + 4 * q]) =
              f32x4{x[4 * q], x[4 * q + 1], x[4 * q + 2], x[4 * q + 3]};
        __syncthreads();
        // Instruction q: columns 16 q .. 16 q + 15, lane piece (tid % 16) of
        // four rows; a piece starting below r1 lies below ldt.
#pragma unroll
        for (int q = 0; q < 64 / (kPassThreads / 16); ++q) {
          const int c = q * (kPassThreads / 16) + tid / 16, r = (tid % 16) * 4;
          if (cc + c < cnt && jr + r < r1)
            *reinterpret_cast<f32x4*>(a.T + size_t(lo + cc + c) * a.ldt + jr + r) =
                *reinterpret_cast<const f32x4*>(&tile[c][r]);
        }
        __syncthreads();
      }
    }
    red[tid] = g0 + g1;
    __syncthreads();
    if (tid < 64 && cc + tid < cnt) {
      long long s = 0;
#pragma unroll
      for (int q = 0; q < kPassWaves; ++q) s += red[q * 64 + tid];
      part[size_t(blockIdx.y) * a.n + lo + cc + tid] = s;
    }
    __syncthreads();
  }
}

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

template <int NG, int RL>
__global__ __launch_bounds__(kBlock) void sgs_rows_batch_kernel(IncBatch b) {
  int s = 0;
  while (s + 1 < b.count && int(blockIdx.x) >= b.g0[s + 1]) ++s;
  rows_body<NG, RL>(b.scene[s], int(blockIdx.x) - b.g0[s], b.g0[s + 1] - b.g0[s]);
}

// The rows form runs when the scene's best costs fit in LDS and a block has
// at most two columns per lane; otherwise the exchange form.
bool use_rows(int64_t n, int W) { return n <= kRowsMaxN && W <= kRowsMaxW; }

// The instance for the largest n and W of a launch.
constexpr int kRowsSmallN = kRowChunk * kWaves * 8;
const void* rows_kernel(int64_t n, int W) {
  if (n <= kRowsSmallN)
    return W <= 64 ? reinterpret_cast<const void*>(sgs_rows_kernel<1, 8>)
                   : reinterpret_cast<const void*>(sgs_rows_kernel<2, 8>);
  return reinterpret_cast<const void*>(sgs_rows_kernel<2, 16>);
}
const void* rows_batch_kernel(int64_t n, int W) {
  if (n <= kRowsSmallN)
    return W <= 64 ? reinterpret_cast<const void*>(sgs_rows_batch_kernel<1, 8>)
                   : reinterpret_cast<const void*>(sgs_rows_batch_kernel<2, 8>);
  return reinterpret_cast<const void*>(sgs_rows_batch_kernel<2, 16>);
}

// Exchange slots and lists, the first pass's partial gains and scale, then
// (when the rows form may run) T.
constexpr int kPassParts = 3;   // row ranges of the first pass (three blocks per compute unit fit at once)
struct IncLayout {
  size_t part, scale, T, epart, lists, ho_gain, ho_sel, ho_b, misc, total;
};
IncLayout inc_layout(int64_t n, int64_t k, bool compact) {
  IncLayout L;
  size_t o = layout(n, k).total;
  L.part = o; o += a256(size_t(kPassParts) * n * sizeof(long long));
  L.scale = o; o += 256;
  L.T = o;
  if (!compact && n <= kRowsMaxN) o += a256(size_t(n) * rows_ldt(n) * sizeof(float));
  // The early kernel's partial sums (rows schedule, n <= kEarlyMaxN), for
  // as many blocks as the scene can have.
  L.epart = o;
  const bool early = !compact && n <= kEarlyMaxN;
  if (early) o += a256(size_t(std::min<int64_t>(kMaxBlocks, (n + 63) / 64)) * early_ldp(n) * 8);
  // The candidate lists (n <= kListMaxN, more than kListStep picks) and the
  // hand-over between launches (lists or the early kernel).
  L.lists = L.ho_gain = L.ho_sel = L.ho_b = L.misc = o;
  const bool lists = !compact && n <= kListMaxN && k > kListStep;
  if (lists) {
    L.lists = o;   o += a256(size_t(n) * kListSlots * 16);
  }
  if (lists || early) {
    L.ho_gain = o; o += a256(size_t(n) * 8);
    L.ho_sel = o;  o += a256(size_t(n));
    L.ho_b = o;    o += a256(size_t(rows_ldt(n)) * 4);
    L.misc = o;    o += a256(24 + 4 + size_t(kMaxBlocks) * 4);   // objective, exchanges, next step; lfail; lblock
  }
  L.total = o;
  return L;
}
size_t inc_bytes(int64_t n, int64_t k, bool compact) { return inc_layout(n, k, compact).total; }

IncDev inc_dev(const SgsParams& p, char* w, int W, bool rows) {
  const Layout L = layout(p.n, p.k);
  IncDev a{};
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
  const WaitPolicy wp = wait_policy();
  a.poll_limit = wp.limit;
  a.abort_init = wp.preset;
  a.W = W;
  a.w_magic = w_magic_of(W);
  const IncLayout M = inc_layout(p.n, p.k, !rows);
  a.T = rows ? reinterpret_cast<float*>(w + M.T) : nullptr;
  a.ldt = rows ? rows_ldt(p.n) : 0;
  a.part = reinterpret_cast<const long long*>(w + M.part);
  a.P = kPassParts;
  a.scale = reinterpret_cast<const int*>(w + M.scale);
  a.k_begin = 0;
  a.k_end = p.k;
  a.gate = nullptr;
  a.gate_val = 0u;
  const bool lists = rows && lists_for(p.n, p.k, W);
  const bool early = rows && early_for(p.n, W);
  const bool ho = lists || early;
  a.lists = lists ? reinterpret_cast<unsigned long long*>(w + M.lists) : nullptr;
  a.ho_gain = ho ? reinterpret_cast<long long*>(w + M.ho_gain) : nullptr;
  a.ho_sel = ho ? reinterpret_cast<unsigned char*>(w + M.ho_sel) : nullptr;
  a.ho_b = ho ? reinterpret_cast<float*>(w + M.ho_b) : nullptr;
  a.ho_misc = ho ? reinterpret_cast<long long*>(w + M.misc) : nullptr;
  a.lfail = lists ? reinterpret_cast<unsigned int*>(w + M.misc + 24) : nullptr;
  a.lblock = lists ? reinterpret_cast<unsigned int*>(w + M.misc + 28) : nullptr;
  a.epart = early ? reinterpret_cast<long long*>(w + M.epart) : nullptr;
  a.ldp = early ? early_ldp(p.n) : 0;
  a.start = nullptr;
  return a;
}

// The scale and the step-0 pass of one scene, ahead of the greedy's launch.
hipError_t launch_first_pass(const IncDev& a, int nb, hipStream_t stream) {
  inc_scale_kernel<<<1, kBlock, 0, stream>>>(a, const_cast<int*>(a.scale));
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  long long* part = const_cast<long long*>(a.part);
  if (a.T)
    inc_first_pass_kernel<true><<<dim3(nb, a.P), kPassThreads, 0, stream>>>(a, part);
  else
    inc_first_pass_kernel<false><<<dim3(nb, a.P), kPassThreads, 0, stream>>>(a, part);
  return hipGetLastError();
}

size_t lds_for(int W) { return size_t(W) * (8 + 4 + 4 + 1) + 16; }
size_t lds_rows(int W, int64_t n) { return size_t((W + 1) & ~1) * 8 + size_t(rows_ldt(n)) * 4 + size_t(W) + 16; }

hipError_t fits(const void* kernel, size_t lds) {
  int per_cu = 0;
  hipError_t e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kernel, kBlock, lds);
  if (e != hipSuccess) return e;
  return per_cu < 1 ? hipErrorCooperativeLaunchTooLarge : hipSuccess;
}

int device_cus(int* cus) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  return hipDeviceGetAttribute(cus, hipDeviceAttributeMultiprocessorCount, dev);
}

// The greedy's launches; with `fused` the step-0 gains and T were written by
// fst_epilogue_sgs_kernel (and the scale before it), so the first pass is
// skipped and the gains come from its partial sums.
hipError_t run_incremental(const SgsParams& p, bool compact, const SgsFused* fused, hipStream_t stream) {
  int cus = 0;
  hipError_t e = hipError_t(device_cus(&cus));
  if (e != hipSuccess) return e;
  const int nb = blocks_for(p.n, cus);
  const int W = (p.n + nb - 1) / nb;
  const bool rows = !compact && use_rows(p.n, W);
  if (fused && !rows) return hipErrorInvalidValue;
  const void* kernel = rows ? rows_kernel(p.n, W) : reinterpret_cast<const void*>(sgs_inc_kernel);
  const size_t lds = rows ? lds_rows(W, p.n) : lds_for(W);
  if ((e = fits(kernel, lds)) != hipSuccess) return e;

  IncDev a = inc_dev(p, static_cast<char*>(p.workspace), W, rows);
  if (fused) {
    a.part = fused->part;
    a.P = fused->P;
  }
  // Scenes the list phase serves: the rows kernel stops after kListStep
  // steps, the lists are built, and the list kernel (or, when the lists do
  // not fit, the rows kernel again) runs the rest.
  const bool lists = a.lists != nullptr;
  if (lists) {
    a.k_end = kListStep;
    if ((e = fits(reinterpret_cast<const void*>(sgs_list_kernel), list_lds(p.n))) != hipSuccess) return e;
  }
  // The early kernel runs the first steps, while they improve many targets;
  // the rows kernel continues from the step it stopped before.
  const bool early = a.epart != nullptr;
  if (early && (e = fits(reinterpret_cast<const void*>(sgs_early_kernel), lds)) != hipSuccess) return e;
  sgs_inc_init_kernel<<<std::min(1024, (std::max(p.n, p.k) + 255) / 256), 256, 0, stream>>>(a);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if (!fused && (e = launch_first_pass(a, nb, stream)) != hipSuccess) return e;
  if (early) {
    void* eargs[] = {&a};
    if ((e = hipLaunchCooperativeKernel(reinterpret_cast<const void*>(sgs_early_kernel), dim3(nb), dim3(kBlock), eargs,
                                        lds, stream)) != hipSuccess)
      return e;
    a.start = a.ho_misc + 2;
  }
  void* args[] = {&a};
  if ((e = hipLaunchCooperativeKernel(kernel, dim3(nb), dim3(kBlock), args, lds, stream)) != hipSuccess) return e;
  if (lists) {
    list_build_kernel<<<(p.n + 3) / 4, 256, 0, stream>>>(a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    IncDev b = a;
    b.start = nullptr;
    b.k_begin = kListStep;
    b.k_end = p.k;
    void* bargs[] = {&b};
    if ((e = hipLaunchCooperativeKernel(reinterpret_cast<const void*>(sgs_list_kernel), dim3(nb), dim3(kBlock), bargs,
                                        list_lds(p.n), stream)) != hipSuccess)
      return e;
    IncDev c = b;
    c.gate = a.lfail;
    c.gate_val = 1u;
    void* cargs[] = {&c};
    if ((e = hipLaunchCooperativeKernel(kernel, dim3(nb), dim3(kBlock), cargs, lds, stream)) != hipSuccess) return e;
  }
  return launch_mark_aborted(a.abort, a.selected, a.k, stream);
}

}  // namespace

size_t sgs_inc_workspace_bytes(int64_t n, int64_t k, bool compact) { return inc_bytes(n, k, compact); }

hipError_t launch_sgs_incremental(const SgsParams& p, bool compact, hipStream_t stream) {
  return run_incremental(p, compact, nullptr, stream);
}

// coverprune_prune: the rows schedule's workspace, then the epilogue's
// partial gains, [n / 64][n] 64-bit integers.
bool sgs_fused_fits(int64_t n) {
  int cus = 0;
  if (device_cus(&cus) != hipSuccess || n < 64 || n % 64 != 0) return false;
  const int nb = blocks_for(n, cus);
  return use_rows(n, int((n + nb - 1) / nb));
}

size_t sgs_fused_workspace_bytes(int64_t n, int64_t k) {
  return inc_bytes(n, k, false) + a256(size_t(n / 64) * size_t(n) * 8);
}

hipError_t sgs_fused_prepare(const SgsParams& p, SgsFused* f, hipStream_t stream) {
  int cus = 0;
  hipError_t e = hipError_t(device_cus(&cus));
  if (e != hipSuccess) return e;
  const int nb = blocks_for(p.n, cus);
  IncDev a = inc_dev(p, static_cast<char*>(p.workspace), (p.n + nb - 1) / nb, true);
  f->T = a.T;
  f->ldt = a.ldt;
  f->part = reinterpret_cast<long long*>(static_cast<char*>(p.workspace) + inc_bytes(p.n, p.k, false));
  f->P = p.n / 64;
  f->scale = const_cast<int*>(a.scale);
  inc_scale_kernel<<<1, kBlock, 0, stream>>>(a, f->scale);
  return hipGetLastError();
}

hipError_t launch_sgs_fused(const SgsParams& p, const SgsFused& f, hipStream_t stream) {
  return run_incremental(p, false, &f, stream);
}

size_t sgs_inc_batch_workspace_bytes(const int64_t* n, const int64_t* k, int count, bool compact) {
  size_t total = 0;
  for (int s = 0; s < count; ++s) total += inc_bytes(n[s], k[s], compact);
  return total;
}

hipError_t launch_sgs_incremental_batch(const SgsParams* p, int count, bool compact, void* workspace,
                                        hipStream_t stream) {
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
  // The rows form when every scene allows it (one form per launch).
  bool rows = !compact;
  int wmax = 0, nmax = 0;
  for (int s = 0; s < count; ++s) {
    const int W = (p[s].n + nb[s] - 1) / nb[s];
    rows = rows && use_rows(p[s].n, W);
    wmax = std::max(wmax, W);
    nmax = std::max(nmax, p[s].n);
  }
  IncBatch b{};
  b.count = count;
  b.g0[0] = 0;
  size_t lds = 0, off = 0;
  char* w = static_cast<char*>(workspace);
  for (int s = 0; s < count; ++s) {
    const int W = (p[s].n + nb[s] - 1) / nb[s];
    b.scene[s] = inc_dev(p[s], w + off, W, rows);
    b.g0[s + 1] = b.g0[s] + nb[s];
    lds = std::max(lds, rows ? lds_rows(W, p[s].n) : lds_for(W));
    off += inc_bytes(p[s].n, p[s].k, compact);
  }
  const void* kernel = rows ? rows_batch_kernel(nmax, wmax) : reinterpret_cast<const void*>(sgs_inc_batch_kernel);
  if ((e = fits(kernel, lds)) != hipSuccess) return e;
  for (int s = 0; s < count; ++s) {
    sgs_inc_init_kernel<<<std::min(1024, (std::max(p[s].n, p[s].k) + 255) / 256), 256, 0, stream>>>(b.scene[s]);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if ((e = launch_first_pass(b.scene[s], b.g0[s + 1] - b.g0[s], stream)) != hipSuccess) return e;
  }
  void* args[] = {&b};
  if ((e = hipLaunchCooperativeKernel(kernel, dim3(used), dim3(kBlock), args, lds, stream)) != hipSuccess) return e;
  for (int s = 0; s < count; ++s)
    if ((e = launch_mark_aborted(b.scene[s].abort, b.scene[s].selected, b.scene[s].k, stream)) != hipSuccess) return e;
  return hipSuccess;
}

}  // namespace cp
