// Shared parts of the persistent greedy kernels that keep their gains in
// exact fixed point: the incremental form (k_sgs_inc.hip) and the local form
// (k_sgs_local.hip), Sec. 3.5.  Both run one cooperative launch of one block
// per compute unit; block b owns tokens [b W, (b + 1) W).
//
// The exchanges are per-block slots rather than counters: a slot holds the
// value together with the step it belongs to, every block reads all slots in
// parallel (one thread per slot), and no address takes more than one writer,
// so a step costs two round trips through memory instead of two grid
// barriers of serialized atomic increments.  Slots, lists and lengths are
// written and read with device-scope atomic operations, coherent across the
// chip's L2 caches without fences; a block's list writes are complete at the
// workgroup barrier before its thread 0 publishes the length.  A slot is only
// rewritten after every block has read it: a block can publish step l + 1's
// values only after reading every block's step-l + 1 candidate, which each
// block publishes only after it has consumed step l.
#pragma once

#include <hip/hip_runtime.h>

#include <climits>

#include "common.h"
#include "fixed_point.h"
#include "launch.h"

namespace cp {
namespace {

constexpr int kBlock = 512;
constexpr int kWaves = kBlock / 64;
constexpr int kMaxBlocks = 256;    // at most one block per compute unit
// Exchange slots sit one per 128-byte line: packed 8 bytes apart, 16 blocks
// on different XCDs would write into the line that every block is polling.
constexpr int kSlotStride = 16;
constexpr int kIndexBits = 20;     // candidate: [epoch | 43-bit gain | 20-bit inverted index]
constexpr unsigned long long kIndexMask = (1ull << kIndexBits) - 1ull;
constexpr unsigned long long kEpoch = 1ull << 63;
constexpr unsigned long long kNoCandidate = 1ull;   // below every real candidate
// Every wait in the kernel is bounded (give_up in common.h): a wait that
// gives up raises the abort flag, every block leaves its waits and returns,
// and a kernel after the launch fills selected[] with -1.

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
  unsigned long long* lens;   // [blocks] (step + 1) << 32 | slice length
  unsigned long long* cand;   // [2][blocks] packed candidate | epoch << 63
  unsigned int* abort;        // set when a wait gives up
  unsigned int poll_limit;    // polls before a wait gives up (WaitPolicy)
  unsigned int abort_init;    // the abort flag's value at launch (WaitPolicy)
  int W;                      // rows and columns per block
  unsigned int w_magic;       // floor(2^32 / W) + 1: block_of(c) = c / W by one high multiply
  float* T;                   // rows form only: [n][ldt] source-major copy, T[s][t] = C(s, t)
  int ldt;                    // its row stride, n rounded up to a whole 256-row chunk
  const long long* part;      // incremental form: [P][n] step-0 gains summed over P row ranges
  int P;
  const int* scale;           // incremental form: the fixed-point exponent S
  // Rows schedule in two launches with a hand-over (see k_sgs_inc.hip): the
  // steps of this launch, the word that decides whether it runs, and the
  // state handed from one launch to the next.
  int k_begin, k_end;         // steps [k_begin, k_end); [0, k) for a single launch
  const unsigned int* gate;   // the launch runs only if *gate == gate_val (null: always)
  unsigned int gate_val;
  long long* ho_gain;         // [n] running gains
  unsigned char* ho_sel;      // [n] chosen flags
  float* ho_b;                // [ldt] best costs
  long long* ho_misc;         // [0] objective in fixed point, [1] exchanges so far, [2] next step
  unsigned long long* lists;  // [n][kListSlots][2] candidate lists
  unsigned int* lfail;        // the lists do not fit
  unsigned int* lblock;       // [blocks] pairs of each block's candidates
  // Early steps of the rows schedule (sgs_early_kernel): each block's partial
  // gain changes of every column, and the step a launch after it starts from
  // (null: k_begin).
  long long* epart;           // [blocks][ldp]: columns 0 .. n - 1, then the objective's change
  int ldp;
  const long long* start;
};

// The block that owns column c: c / W as the high word of c times
// floor(2^32 / W) + 1, exact for c < 2^18 and 2 <= W <= 2^13 (the product
// exceeds 2^32 c / W by less than c, which moves c / W by less than 2^-14,
// below the gap 1 / W to the next integer).  W = 1 only with n = 1 (the
// grid has one block per 64 tokens at most), where the multiplier wraps to
// 0 and column 0's block is 0.
__device__ __forceinline__ int block_of(const IncDev& a, int c) { return int(__umulhi(unsigned(c), a.w_magic)); }
inline unsigned int w_magic_of(int W) { return unsigned(0xffffffffu / unsigned(W)) + 1u; }

struct Layout {
  size_t list, lens, cand, ctrl, total;
};

size_t a256(size_t x) { return (x + 255) / 256 * 256; }

int blocks_for(int64_t n, int cus) {
  return int(std::max<int64_t>(1, std::min<int64_t>(std::min(cus, kMaxBlocks), (n + 63) / 64)));
}

// Sized for the largest grid (kMaxBlocks blocks of W = ceil(n / blocks) rows).
Layout layout(int64_t n, int64_t k) {
  (void)k;
  Layout L;
  size_t o = 0;
  L.list = o; o += a256(size_t(n + kMaxBlocks) * 16);
  L.lens = o; o += a256(size_t(kMaxBlocks) * kSlotStride * 8);
  L.cand = o; o += a256(size_t(2 * kMaxBlocks) * kSlotStride * 8);
  L.ctrl = o; o += 256;
  L.total = o;
  return L;
}

// Block b's candidate slot of slot set `set` (set = step % 2), and its
// slice-length slot.
__host__ __device__ __forceinline__ unsigned long long* cand_slot(unsigned long long* cand, int set, int b) {
  return cand + (size_t(set) * kMaxBlocks + b) * kSlotStride;
}
__host__ __device__ __forceinline__ unsigned long long* lens_slot(unsigned long long* lens, int b) {
  return lens + size_t(b) * kSlotStride;
}

// Nonnegative gain truncated to its top 43 bits (relative resolution 2^-31),
// then the inverted index: larger gain first, then smaller index.  Indices
// are below 2^18, so every real candidate exceeds kNoCandidate.
__device__ __forceinline__ unsigned long long pack_key(double g, int idx) {
  const unsigned long long gb = (unsigned long long)__double_as_longlong(g) >> (kIndexBits + 1);
  return (gb << kIndexBits) | (kIndexMask - (unsigned long long)idx);
}

// Epoch bit of the candidates of exchange l (the step, unless steps skip
// their exchange), kept in slot set l % 2: it flips between consecutive uses
// of a set and is never the zero of a fresh workspace for exchanges 0 and 1.
__device__ __forceinline__ unsigned long long epoch_of(int step) {
  return ((step >> 1) & 1) ? 0ull : kEpoch;
}

__global__ void sgs_inc_init_kernel(IncDev a) {
  const int gt = blockIdx.x * blockDim.x + threadIdx.x, nt = gridDim.x * blockDim.x;
  for (int s = gt; s < kMaxBlocks; s += nt) {
    a.lens[size_t(s) * kSlotStride] = 0ull;
    // Word 0 of a candidate slot holds the key; the rows schedule also
    // writes word 1 (the second key).
    for (int w = 0; w < 2; ++w) {
      a.cand[size_t(s) * kSlotStride + w] = 0ull;
      a.cand[size_t(kMaxBlocks + s) * kSlotStride + w] = 0ull;
    }
  }
  for (int j = gt; j < a.n; j += nt)
    if (a.assign) a.assign[j] = -1;
  if (a.lfail) {
    for (int s = gt; s < kMaxBlocks; s += nt) a.lblock[s] = 0u;
    if (gt == 0) *a.lfail = 0u;
  }
  if (gt == 0) *a.abort = a.abort_init;
}

// Wave reductions without LDS traffic: DPP moves within each row of 16
// lanes, in the pattern swap neighbours, swap pairs, mirror halves of 8,
// mirror the row (after each step every lane of a group of 2, 4, 8, 16 holds
// the group's result), then the four row results read from lanes 0, 16, 32
// and 48.  Every lane of the wave must be active.
constexpr int kDppSteps[4] = {0xB1, 0x4E, 0x141, 0x140};   // quad_perm [1,0,3,2], [2,3,0,1], row_half_mirror, row_mirror

__device__ __forceinline__ unsigned long long lane_u64(unsigned long long x, int r) {
  return ((unsigned long long)__builtin_amdgcn_readlane(unsigned(x >> 32), r) << 32) |
         unsigned(__builtin_amdgcn_readlane(unsigned(x), r));
}


__device__ __forceinline__ unsigned wave_max_u32(unsigned x) {
  x = max(x, unsigned(__builtin_amdgcn_mov_dpp(int(x), kDppSteps[0], 0xf, 0xf, false)));
  x = max(x, unsigned(__builtin_amdgcn_mov_dpp(int(x), kDppSteps[1], 0xf, 0xf, false)));
  x = max(x, unsigned(__builtin_amdgcn_mov_dpp(int(x), kDppSteps[2], 0xf, 0xf, false)));
  x = max(x, unsigned(__builtin_amdgcn_mov_dpp(int(x), kDppSteps[3], 0xf, 0xf, false)));
  return max(max(unsigned(__builtin_amdgcn_readlane(int(x), 0)), unsigned(__builtin_amdgcn_readlane(int(x), 16))),
             max(unsigned(__builtin_amdgcn_readlane(int(x), 32)), unsigned(__builtin_amdgcn_readlane(int(x), 48))));
}

// The 64-bit maximum as 32-bit ones: the largest high word, then the low
// word of the one lane that holds it, or, when several do, the largest of
// their low words (32-bit steps take one compare-select where a 64-bit step
// takes three).
__device__ __forceinline__ unsigned long long wave_max_u64(unsigned long long x) {
  const unsigned hi = unsigned(x >> 32);
  const unsigned hm = wave_max_u32(hi);
  const unsigned long long tie = __ballot(hi == hm);
  unsigned lm;
  if (__popcll(tie) == 1)
    lm = unsigned(__builtin_amdgcn_readlane(int(unsigned(x)), __builtin_ctzll(tie)));
  else
    lm = wave_max_u32(hi == hm ? unsigned(x) : 0u);
  return ((unsigned long long)hm << 32) | lm;
}

__device__ __forceinline__ long long wave_max_i64(long long x) {
  long long y;
  y = (long long)dpp_u64<kDppSteps[0]>((unsigned long long)x); x = y > x ? y : x;
  y = (long long)dpp_u64<kDppSteps[1]>((unsigned long long)x); x = y > x ? y : x;
  y = (long long)dpp_u64<kDppSteps[2]>((unsigned long long)x); x = y > x ? y : x;
  y = (long long)dpp_u64<kDppSteps[3]>((unsigned long long)x); x = y > x ? y : x;
  long long m = (long long)lane_u64((unsigned long long)x, 0);
#pragma unroll
  for (int r = 16; r < 64; r += 16) {
    y = (long long)lane_u64((unsigned long long)x, r);
    m = y > m ? y : m;
  }
  return m;
}

__device__ __forceinline__ long long wave_sum_i64(long long x) {
  x += (long long)dpp_u64<kDppSteps[0]>((unsigned long long)x);
  x += (long long)dpp_u64<kDppSteps[1]>((unsigned long long)x);
  x += (long long)dpp_u64<kDppSteps[2]>((unsigned long long)x);
  x += (long long)dpp_u64<kDppSteps[3]>((unsigned long long)x);
  return (long long)(lane_u64((unsigned long long)x, 0) + lane_u64((unsigned long long)x, 16) +
                     lane_u64((unsigned long long)x, 32) + lane_u64((unsigned long long)x, 48));
}

__device__ __forceinline__ int wave_min_i32(int x) {
  int y;
  y = __builtin_amdgcn_mov_dpp(x, kDppSteps[0], 0xf, 0xf, false); x = y < x ? y : x;
  y = __builtin_amdgcn_mov_dpp(x, kDppSteps[1], 0xf, 0xf, false); x = y < x ? y : x;
  y = __builtin_amdgcn_mov_dpp(x, kDppSteps[2], 0xf, 0xf, false); x = y < x ? y : x;
  y = __builtin_amdgcn_mov_dpp(x, kDppSteps[3], 0xf, 0xf, false); x = y < x ? y : x;
  int m = __builtin_amdgcn_readlane(x, 0);
#pragma unroll
  for (int r = 16; r < 64; r += 16) {
    y = __builtin_amdgcn_readlane(x, r);
    m = y < m ? y : m;
  }
  return m;
}

// Inclusive prefix sum over the lanes of a wave (every lane active).
__device__ __forceinline__ int wave_scan_incl(int x) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(x, o);
    if (lane >= o) x += y;
  }
  return x;
}

// Sum over the block of 64-bit integers, result in every thread.
__device__ long long block_sum_i64(long long x, long long* sg) {
  x = wave_sum_i64(x);
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  __syncthreads();
  if (lane == 0) sg[w] = x;
  __syncthreads();
  long long s = 0;
#pragma unroll
  for (int q = 0; q < kWaves; ++q) s += sg[q];
  __syncthreads();
  return s;
}

// Poll *p until pred(value) holds; false if the launch is aborting (this
// wait gave up, or another one did).
template <class Pred>
__device__ bool wait_slot(const unsigned long long* p, unsigned int* abort, unsigned int limit, Pred pred,
                          unsigned long long& x) {
  for (unsigned int spins = 0;; ++spins) {
    x = get(p);
    if (pred(x)) return true;
    if (give_up(spins, limit, abort)) return false;
    __builtin_amdgcn_s_sleep(1);
  }
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

// Thread t's part of sum_j fx(v_j c0, S), the objective at b = c0 (exact
// integers, so the parts and their total do not depend on the order): j = t,
// t + kBlock, ..., eight loads in flight at a time (a load whose result the
// next iteration needs waits for itself otherwise).
__device__ __forceinline__ long long fx_capacity_part(const float* v, int n, float c0, int S) {
  long long x = 0;
  constexpr int U = 8;
  for (int j0 = threadIdx.x; j0 < n; j0 += kBlock * U) {
    float vv[U];
#pragma unroll
    for (int u = 0; u < U; ++u) vv[u] = v[min(j0 + u * kBlock, n - 1)];
#pragma unroll
    for (int u = 0; u < U; ++u)
      if (j0 + u * kBlock < n) x += fx(double(vv[u]) * double(c0), S);
  }
  return x;
}

// Block maximum, result in every thread.
__device__ double block_max_all(double x, double* sd) {
  x = wave_max(x);
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  __syncthreads();
  if (lane == 0) sd[w] = x;
  __syncthreads();
  double s = sd[0];
#pragma unroll
  for (int q = 1; q < kWaves; ++q) s = fmax(s, sd[q]);
  __syncthreads();
  return s;
}

// Argmax of (g, gi) over a whole wave (every lane active), in every lane:
// the largest gain, then the smallest index among the lanes that hold it.
// g = -1 marks no candidate (gi = INT_MAX).
__device__ __forceinline__ void wave_argmax(long long& g, int& gi) {
  const long long top = wave_max_i64(g);
  gi = wave_min_i32(g == top ? gi : INT_MAX);
  g = top;
}

// Exact argmax (ties to the smaller index) of the block's unchosen columns,
// published as the block's candidate for the step; across blocks the gains
// compare as doubles truncated to 43 bits.  With at most 64 columns wave 0
// does it alone, one column per lane, and no barrier follows: the callers'
// next step begins with one (read_winner), and the gains and chosen flags it
// reads were last written by wave 0 itself.
__device__ __forceinline__ void publish_argmax(const long long* sG, const unsigned char* ssel, int lo, int cnt,
                                               int S, unsigned long long* slot, unsigned long long epoch,
                                               long long* sg, int* si) {
  if (cnt <= 64) {
    if (threadIdx.x >= 64) return;
    const int i = threadIdx.x;
    long long g = -1;
    int gi = INT_MAX;
    if (i < cnt && !ssel[i]) {
      g = sG[i];
      gi = lo + i;
    }
    wave_argmax(g, gi);
    if (i == 0) put(slot, (gi != INT_MAX ? pack_key(fx_to_double(g, S), gi) : kNoCandidate) | epoch);
    return;
  }
  long long g = -1;
  int gi = INT_MAX;
  for (int i = threadIdx.x; i < cnt; i += kBlock)
    if (!ssel[i] && sG[i] > g) {   // increasing i: ties keep the smaller index
      g = sG[i];
      gi = lo + i;
    }
  wave_argmax(g, gi);
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
    put(slot, (gi != INT_MAX ? pack_key(fx_to_double(g, S), gi) : kNoCandidate) | epoch);
  }
  __syncthreads();
}

// The step's winner: thread i < nb waits for block i's candidate of this
// epoch; the largest wins (the same in every block).  Returns -1 when the
// launch is aborting.
__device__ int read_winner(const unsigned long long* slots, unsigned long long epoch, int nb,
                           unsigned int* abort, unsigned int limit, unsigned long long* su, int* sflag) {
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  unsigned long long best = 0ull;
  if (tid == 0) *sflag = 0;
  __syncthreads();
  if (tid < nb) {
    unsigned long long x;
    if (wait_slot(slots + size_t(tid) * kSlotStride, abort, limit,
                  [epoch](unsigned long long v) { return (v & kEpoch) == epoch; }, x))
      best = x & ~kEpoch;
    else
      *sflag = 1;
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

}  // namespace
}  // namespace cp
