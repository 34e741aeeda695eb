// The greedy step solved as the paper writes it (Sec. 3.5, Eq. 11-15).
//
// Step l retains S_l = {s_0 .. s_{l-1}}, each with source mass u = 1/K, and
// solves the entropic semi-relaxed transport to all targets (Eq. 12:
// P 1 = u, P^T 1 <= v) by alternating scalings P = diag(a) E diag(b),
// E_ji = exp(-C(s_i, j) / eps):
//   a_i <- u / sum_j E_ji b_j,   b_j <- min(1, v_j / t_j),  t_j = sum_i E_ji a_i
// (b_j = 1 where t_j = 0), from b = 1, for a fixed number of rounds.  The
// residual r_j = max(0, v_j - b_j t_j) (Eq. 14) weights the score
// score(c) = sum_j r_j C(c, j) (Eq. 15 with every target a neighbour), and
// the unselected token with the smallest score is retained next (ties to the
// smaller index).  Step 0 has no source and r = v.  After K picks the same
// solve over all of S gives the plan whose cost <P, C_S> is reported.
//
// Layout: E is a compact [n, kp] float64 matrix (kp = k rounded up to 4)
// whose column i is filled when s_i is retained, target-major like the
// cost, so a round is one pass over the first l columns.  Kernels, per step:
//   lit_append_kernel   E[:, l-1] = exp(-C_tm[:, s_{l-1}] / eps) in float64
//                       (float32 would flush exp(-C / eps) to zero once C / eps
//                       passes about 103, cutting sources off from targets
//                       they must reach; float64 holds it to about 708)
//   lit_rows_kernel     64 rows per block: t_j (one wave per row), b_j, and
//                       the block's column sums sum_j E_ji b_j (one thread per
//                       column); b = 1 on the first round
//   lit_a_kernel        a_i = u / (sum of the row blocks' column sums, in
//                       block order)
//   lit_rows_kernel     (last round) r_j instead of column sums
//   lit_score_kernel    row panels x 256-column strips: partial sum_j r_j C_tm[j][c]
//   lit_select_kernel   one block: panel sums in panel order, argmin over the
//                       unselected tokens, residual mass
// Every sum is float64 in a fixed order, so results are deterministic.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cfloat>

#include "common.h"
#include "launch.h"

namespace cp {
namespace {

constexpr int kLitBlock = 256;
constexpr int kLitWaves = kLitBlock / kWave;
constexpr int kLitRows = 64;          // rows per block of lit_rows_kernel
constexpr int kLitMaxK = 4096;        // a (float64) and the picks stay in LDS
constexpr int kSelectBlock = 1024;

struct LitDev {
  const float* C;          // [n, n] target-major
  const float* v;          // [n]
  int n, k, kp;
  double eps, u;
  double* E;               // [n, kp]
  double* a;               // [k]
  double* b;               // [n]
  double* r;               // [n]
  double* colpart;         // [kp, nrb]: column i's partial sums, one per row block
  double* scorepart;       // [panels, n]
  double* objpart;         // [nrb]
  unsigned char* chosen;   // [n]
  int32_t* selected;       // [k]
  const int32_t* follow;   // [k] or nullptr
  double* step_score;      // [k] or nullptr
  double* step_residual;   // [k] or nullptr
  double* objective;       // [1] or nullptr
  int nrb, panels, strips;
};

__global__ void lit_init_kernel(LitDev p) {
  for (int j = blockIdx.x * blockDim.x + threadIdx.x; j < p.n; j += gridDim.x * blockDim.x) {
    p.chosen[j] = 0;
    p.r[j] = double(p.v[j]);
  }
}

// Column l - 1 of E from the pick of step l - 1.
__global__ void lit_append_kernel(LitDev p, int l) {
  const int s = min(max(int(p.selected[l - 1]), 0), p.n - 1);
  if (blockIdx.x == 0 && threadIdx.x == 0) p.chosen[s] = 1;
  for (int j = blockIdx.x * blockDim.x + threadIdx.x; j < p.n; j += gridDim.x * blockDim.x)
    p.E[size_t(j) * p.kp + (l - 1)] = exp(-double(p.C[size_t(j) * p.n + s]) / p.eps);
}

// mode 0: first round (b = 1): column sums only.
// mode 1: t_j, b_j, then column sums with the new b.
// mode 2: last round: t_j, b_j and the residual r_j.
__global__ __launch_bounds__(kLitBlock) void lit_rows_kernel(LitDev p, int l, int mode) {
  __shared__ double sa[kLitMaxK];
  __shared__ double sb[kLitRows];
  const int lane = threadIdx.x & (kWave - 1), w = threadIdx.x >> 6;
  const int j0 = blockIdx.x * kLitRows;
  const int rows = min(kLitRows, p.n - j0);
  if (mode == 0) {
    for (int q = threadIdx.x; q < rows; q += kLitBlock) sb[q] = 1.0;
  } else {
    for (int i = threadIdx.x; i < l; i += kLitBlock) sa[i] = p.a[i];
    __syncthreads();
    for (int q = w; q < rows; q += kLitWaves) {
      const int j = j0 + q;
      const double* e = p.E + size_t(j) * p.kp;
      double t = 0.0;
#pragma unroll 4
      for (int i = lane; i < l; i += kWave) t = fma(e[i], sa[i], t);
      t = wave_sum(t);
      const double vj = double(p.v[j]);
      const double bj = t > 0.0 ? fmin(1.0, vj / t) : 1.0;
      if (lane == 0) {
        sb[q] = bj;
        p.b[j] = bj;
        if (mode == 2) p.r[j] = fmax(vj - bj * t, 0.0);
      }
    }
  }
  if (mode == 2) return;
  __syncthreads();
  for (int i = threadIdx.x; i < l; i += kLitBlock) {
    double s = 0.0;
#pragma unroll 8
    for (int q = 0; q < rows; ++q) s = fma(p.E[size_t(j0 + q) * p.kp + i], sb[q], s);
    p.colpart[size_t(i) * p.nrb + blockIdx.x] = s;
  }
}

// One wave per column: its row-block partials, lane-strided then a fixed
// butterfly, so the sum's order does not depend on timing.
__global__ __launch_bounds__(kLitBlock) void lit_a_kernel(LitDev p, int l) {
  const int lane = threadIdx.x & (kWave - 1);
  const int i = blockIdx.x * kLitWaves + (threadIdx.x >> 6);
  if (i >= l) return;
  const double* c = p.colpart + size_t(i) * p.nrb;
  double s = 0.0;
  for (int rb = lane; rb < p.nrb; rb += kWave) s += c[rb];
  s = wave_sum(s);
  if (lane == 0) p.a[i] = p.u / s;
}

// Partial scores: block (strip, panel) sums r_j C_tm[j][c] over the panel's
// rows for the strip's 256 columns, eight rows in flight per thread.
__global__ __launch_bounds__(kLitBlock) void lit_score_kernel(LitDev p) {
  __shared__ double sr[kLitBlock];
  const int c = blockIdx.x * kLitBlock + threadIdx.x;
  const int per = (p.n + p.panels - 1) / p.panels;
  const int r0 = blockIdx.y * per, r1 = min(p.n, r0 + per);
  double acc = 0.0;
  for (int base = r0; base < r1; base += kLitBlock) {
    const int cnt = min(kLitBlock, r1 - base);
    __syncthreads();
    if (threadIdx.x < cnt) sr[threadIdx.x] = p.r[base + threadIdx.x];
    __syncthreads();
    if (c < p.n) {
      int q = 0;
      for (; q + 8 <= cnt; q += 8) {
        float x[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) x[u] = __builtin_nontemporal_load(p.C + size_t(base + q + u) * p.n + c);
#pragma unroll
        for (int u = 0; u < 8; ++u) acc = fma(sr[q + u], double(x[u]), acc);
      }
      for (; q < cnt; ++q) acc = fma(sr[q], double(p.C[size_t(base + q) * p.n + c]), acc);
    }
  }
  if (c < p.n) p.scorepart[size_t(blockIdx.y) * p.n + c] = acc;
}

// Step l's pick: panel sums in panel order, the smallest score over the
// unselected tokens (smaller index on ties), and the residual mass.
__global__ __launch_bounds__(kSelectBlock) void lit_select_kernel(LitDev p, int l) {
  __shared__ double sv[kSelectBlock];
  __shared__ int si[kSelectBlock];
  __shared__ double sm[kSelectBlock];
  double best = DBL_MAX, mass = 0.0;
  int bi = INT_MAX;
  for (int c = threadIdx.x; c < p.n; c += kSelectBlock) {
    mass += p.r[c];
    if (p.chosen[c]) continue;
    double s = 0.0;
    for (int q = 0; q < p.panels; ++q) s += p.scorepart[size_t(q) * p.n + c];
    if (s < best) {
      best = s;
      bi = c;
    }
  }
  sv[threadIdx.x] = best;
  si[threadIdx.x] = bi;
  sm[threadIdx.x] = mass;
  __syncthreads();
  for (int h = kSelectBlock / 2; h > 0; h >>= 1) {
    if (threadIdx.x < h) {
      const double ov = sv[threadIdx.x + h];
      const int oi = si[threadIdx.x + h];
      if (ov < sv[threadIdx.x] || (ov == sv[threadIdx.x] && oi < si[threadIdx.x])) {
        sv[threadIdx.x] = ov;
        si[threadIdx.x] = oi;
      }
      sm[threadIdx.x] += sm[threadIdx.x + h];
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    int pick = si[0];
    double score = sv[0];
    if (p.follow) {
      pick = min(max(int(p.follow[l]), 0), p.n - 1);
      score = 0.0;
      for (int q = 0; q < p.panels; ++q) score += p.scorepart[size_t(q) * p.n + pick];
    }
    p.selected[l] = pick;
    if (p.step_score) p.step_score[l] = score;
    if (p.step_residual) p.step_residual[l] = sm[0];
  }
}

// The picks of a trajectory to follow, when no per-step output is wanted.
__global__ void lit_follow_kernel(LitDev p) {
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < p.k; i += gridDim.x * blockDim.x)
    p.selected[i] = min(max(int(p.follow[i]), 0), p.n - 1);
}

// Transport cost of the final plan: block partials of
// sum_j sum_i a_i E_ji b_j C(s_i, j).
__global__ __launch_bounds__(kLitBlock) void lit_objective_kernel(LitDev p) {
  __shared__ double sa[kLitMaxK];
  __shared__ int ss[kLitMaxK];
  __shared__ double sw[kLitWaves];
  const int lane = threadIdx.x & (kWave - 1), w = threadIdx.x >> 6;
  for (int i = threadIdx.x; i < p.k; i += kLitBlock) {
    sa[i] = p.a[i];
    ss[i] = min(max(int(p.selected[i]), 0), p.n - 1);
  }
  __syncthreads();
  const int j0 = blockIdx.x * kLitRows;
  const int rows = min(kLitRows, p.n - j0);
  double acc = 0.0;
  for (int q = w; q < rows; q += kLitWaves) {
    const int j = j0 + q;
    const double* e = p.E + size_t(j) * p.kp;
    const float* c = p.C + size_t(j) * p.n;
    double s = 0.0;
    for (int i = lane; i < p.k; i += kWave) s = fma(sa[i] * e[i], double(c[ss[i]]), s);
    acc += wave_sum(s) * p.b[j];
  }
  if (lane == 0) sw[w] = acc;
  __syncthreads();
  if (threadIdx.x == 0) {
    double s = 0.0;
    for (int q = 0; q < kLitWaves; ++q) s += sw[q];
    p.objpart[blockIdx.x] = s;
  }
}

__global__ void lit_objective_sum_kernel(LitDev p) {
  if (threadIdx.x == 0 && blockIdx.x == 0) {
    double s = 0.0;
    for (int rb = 0; rb < p.nrb; ++rb) s += p.objpart[rb];
    *p.objective = s;
  }
}

size_t a256(size_t x) { return (x + 255) / 256 * 256; }

struct LitLayout {
  size_t E, a, b, r, colpart, scorepart, objpart, chosen, total;
  int kp, nrb, panels, strips;
};

LitLayout lit_layout(int64_t n, int64_t k) {
  LitLayout L;
  L.kp = int((k + 3) / 4 * 4);
  L.nrb = int((n + kLitRows - 1) / kLitRows);
  L.strips = int((n + kLitBlock - 1) / kLitBlock);
  L.panels = std::max(1, std::min(64, (512 + L.strips - 1) / L.strips));
  size_t o = 0;
  L.E = o;
  o = a256(o + size_t(n) * L.kp * 8);
  L.a = o;
  o = a256(o + size_t(L.kp) * 8);
  L.b = o;
  o = a256(o + size_t(n) * 8);
  L.r = o;
  o = a256(o + size_t(n) * 8);
  L.colpart = o;
  o = a256(o + size_t(L.nrb) * L.kp * 8);
  L.scorepart = o;
  o = a256(o + size_t(L.panels) * n * 8);
  L.objpart = o;
  o = a256(o + size_t(L.nrb) * 8);
  L.chosen = o;
  o = a256(o + size_t(n));
  L.total = o;
  return L;
}

// One solve over the first l retained tokens: `rounds` scaling rounds, the
// last one leaving b and the residual.
hipError_t solve(const LitDev& p, int l, int rounds, hipStream_t stream) {
  const int a_blocks = (l + kLitWaves - 1) / kLitWaves;
  lit_rows_kernel<<<p.nrb, kLitBlock, 0, stream>>>(p, l, 0);
  for (int it = 0; it < rounds; ++it) {
    lit_a_kernel<<<a_blocks, kLitBlock, 0, stream>>>(p, l);
    lit_rows_kernel<<<p.nrb, kLitBlock, 0, stream>>>(p, l, it + 1 < rounds ? 1 : 2);
  }
  return hipGetLastError();
}

}  // namespace

size_t sgs_literal_workspace_bytes(int64_t n, int64_t k) { return lit_layout(n, k).total; }

hipError_t launch_sgs_literal(const LiteralParams& q, hipStream_t stream) {
  if (q.n < 1 || q.k < 1 || q.k > q.n || q.k > kLitMaxK || q.rounds < 1) return hipErrorInvalidValue;
  const LitLayout L = lit_layout(q.n, q.k);
  char* w = static_cast<char*>(q.workspace);
  LitDev p;
  p.C = q.cost;
  p.v = q.capacity;
  p.n = q.n;
  p.k = q.k;
  p.kp = L.kp;
  p.eps = double(q.epsilon);
  p.u = 1.0 / double(q.k);
  p.E = reinterpret_cast<double*>(w + L.E);
  p.a = reinterpret_cast<double*>(w + L.a);
  p.b = reinterpret_cast<double*>(w + L.b);
  p.r = reinterpret_cast<double*>(w + L.r);
  p.colpart = reinterpret_cast<double*>(w + L.colpart);
  p.scorepart = reinterpret_cast<double*>(w + L.scorepart);
  p.objpart = reinterpret_cast<double*>(w + L.objpart);
  p.chosen = reinterpret_cast<unsigned char*>(w + L.chosen);
  p.selected = q.selected;
  p.follow = q.follow;
  p.step_score = q.step_score;
  p.step_residual = q.step_residual;
  p.objective = q.objective;
  p.nrb = L.nrb;
  p.panels = L.panels;
  p.strips = L.strips;

  hipError_t e;
  const int grid_n = std::min(1024, (q.n + 255) / 256);
  lit_init_kernel<<<grid_n, 256, 0, stream>>>(p);
  if (q.follow && !q.step_score && !q.step_residual) {
    // A trajectory to follow and no per-step output: only the final plan.
    lit_follow_kernel<<<(q.k + 255) / 256, 256, 0, stream>>>(p);
    for (int l = 1; l <= q.k; ++l) lit_append_kernel<<<grid_n, 256, 0, stream>>>(p, l);
  } else {
    for (int l = 0; l < q.k; ++l) {
      if (l > 0) {
        lit_append_kernel<<<grid_n, 256, 0, stream>>>(p, l);
        if ((e = solve(p, l, q.rounds, stream)) != hipSuccess) return e;
      }
      lit_score_kernel<<<dim3(L.strips, L.panels), kLitBlock, 0, stream>>>(p);
      lit_select_kernel<<<1, kSelectBlock, 0, stream>>>(p, l);
      if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    lit_append_kernel<<<grid_n, 256, 0, stream>>>(p, q.k);
  }
  if ((e = solve(p, q.k, q.rounds, stream)) != hipSuccess) return e;
  if (q.objective) {
    lit_objective_kernel<<<L.nrb, kLitBlock, 0, stream>>>(p);
    lit_objective_sum_kernel<<<1, 64, 0, stream>>>(p);
  }
  return hipGetLastError();
}

}  // namespace cp
