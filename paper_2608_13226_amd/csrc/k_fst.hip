// FST transport cost, everything except the feature Gram (Sec. 3.3, Eq. 7-8).
//
//   prep      inverse feature norms, frame-index range (M_tau) and the exact
//             maximum pairwise distance (M_x, over all N^2 pairs)
//   epilogue  turns the Gram's raw d_f (upper tiles only) into the final
//             target-major cost C_tm[t][s] = C(s, t), writing both triangles
#include <hip/hip_runtime.h>

#include <algorithm>
#include <climits>

#include "common.h"
#include "fixed_point.h"
#include "launch.h"

namespace cp {
namespace {

__global__ void fst_init_kernel(FstScratch s) {
  *s.mf_bits = 0u;
  *s.mx2_bits = 0ull;
  *s.tau_min = INT_MAX;
  *s.tau_max = INT_MIN;
}

constexpr int kPrepThreads = 256;
constexpr int kPrepWaves = kPrepThreads / 64;

// Inverse feature norms, as block blk of nblk: each wave walks rows
// blk * 4 + w, + 4 * nblk, ..., with a row's 16-byte loads (up to 8 per lane)
// in flight together.  Frame indices fold into a per-block range first, so
// the grid issues only two atomics per block.
template <bool BF16>
__device__ void row_norms(const void* feats, int n, int d, const int32_t* frame, FstScratch s, int blk,
                          int nblk) {
  const int lane = threadIdx.x & 63, wib = threadIdx.x >> 6;
  int fmin = INT_MAX, fmax = INT_MIN;
  const int m = BF16 ? d / 8 : d / 4;   // 16-byte chunks per row
  for (int row = blk * kPrepWaves + wib; row < n; row += nblk * kPrepWaves) {
    const uint4* p = reinterpret_cast<const uint4*>(static_cast<const char*>(feats) +
                                                    size_t(row) * d * (BF16 ? 2 : 4));
    float acc = 0.f;
    for (int i0 = 0; i0 < m; i0 += 8 * 64) {
      uint4 q[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int i = i0 + u * 64 + lane;
        q[u] = i < m ? p[i] : make_uint4(0u, 0u, 0u, 0u);
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const uint32_t w4[4] = {q[u].x, q[u].y, q[u].z, q[u].w};
#pragma unroll
        for (int h = 0; h < 4; ++h) {
          if (BF16) {
            const float lo = bf16_bits_to_float(w4[h] & 0xffffu), hi = bf16_bits_to_float(w4[h] >> 16);
            acc = fmaf(lo, lo, acc);
            acc = fmaf(hi, hi, acc);
          } else {
            const float x = __uint_as_float(w4[h]);
            acc = fmaf(x, x, acc);
          }
        }
      }
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) acc += __shfl_xor(acc, o);
    if (lane == 0) {
      s.inv_norm[row] = acc > 0.f ? 1.0f / sqrtf(acc) : 0.f;
      const int f = frame[row];
      fmin = min(fmin, f);
      fmax = max(fmax, f);
    }
  }
  __shared__ int smin[kPrepWaves], smax[kPrepWaves];
  if (lane == 0) {
    smin[wib] = fmin;
    smax[wib] = fmax;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    int lo = smin[0], hi = smax[0];
    for (int w = 1; w < kPrepWaves; ++w) {
      lo = min(lo, smin[w]);
      hi = max(hi, smax[w]);
    }
    if (lo != INT_MAX) {
      atomicMin(s.tau_min, lo);
      atomicMax(s.tau_max, hi);
    }
  }
}

// Upper-triangular tile index b -> (ti <= tj).
__device__ __forceinline__ void upper_tile(int b, int& ti, int& tj) {
  int j = int((sqrt(8.0 * double(b) + 1.0) - 1.0) * 0.5);
  while (j * (j + 1) / 2 > b) --j;
  while ((j + 1) * (j + 2) / 2 <= b) ++j;
  tj = j;
  ti = b - j * (j + 1) / 2;
}

// Squared distance in float64 with a fixed operation order and no fused
// multiply-add, so the maximum is bitwise reproducible.
__device__ __forceinline__ double sq_dist(double ax, double ay, double az, double bx, double by,
                                          double bz) {
#pragma clang fp contract(off)
  const double dx = ax - bx, dy = ay - by, dz = az - bz;
  return (dx * dx + dy * dy) + dz * dz;
}

constexpr int kPosTile = 256;

// Exact maximum squared distance over all pairs: one block per upper
// 256 x 256 tile (enough waves in flight to hide the float64 latency; this
// is block b of the tiles), a thread takes one row of the tile against the
// tile's columns staged in LDS, and a block whose maximum is larger than the
// running one raises it.
__device__ void pos_pairmax(const float* pos, int n, int b, FstScratch s) {
  static_assert(kPosTile == kPrepThreads, "one tile row per thread");
  __shared__ double sx[kPosTile], sy[kPosTile], sz[kPosTile];
  __shared__ double sm[kPrepWaves];
  double best = 0.0;
  {
    int ti, tj;
    upper_tile(b, ti, tj);
    const int j = tj * kPosTile + threadIdx.x;
    const int jn = min(kPosTile, n - tj * kPosTile);
    __syncthreads();
    if (threadIdx.x < jn) {
      sx[threadIdx.x] = pos[3 * j];
      sy[threadIdx.x] = pos[3 * j + 1];
      sz[threadIdx.x] = pos[3 * j + 2];
    }
    __syncthreads();
    const int i = ti * kPosTile + threadIdx.x;
    if (i < n) {
      const double x = pos[3 * i], y = pos[3 * i + 1], z = pos[3 * i + 2];
      for (int jj = 0; jj < jn; ++jj) best = fmax(best, sq_dist(x, y, z, sx[jj], sy[jj], sz[jj]));
    }
  }
  best = wave_max(best);
  if ((threadIdx.x & 63) == 0) sm[threadIdx.x >> 6] = best;
  __syncthreads();
  // Read first: the maximum only grows, and atomics from many blocks on one
  // address serialize.
  const double m = fmax(fmax(sm[0], sm[1]), fmax(sm[2], sm[3]));
  if (threadIdx.x == 0 && m > __longlong_as_double((long long)get(s.mx2_bits))) atomic_max_nonneg(s.mx2_bits, m);
}

// The prep in one launch: the compute-bound pair maxima (blocks [0, tiles))
// run beside the memory-bound row norms (the nr blocks after them).
template <bool BF16>
__global__ __launch_bounds__(kPrepThreads) void fst_prep_kernel(const void* feats, int n, int d,
                                                                const int32_t* frame, const float* pos,
                                                                int tiles, int nr, FstScratch s) {
  if (int(blockIdx.x) < tiles) pos_pairmax(pos, n, blockIdx.x, s);
  else row_norms<BF16>(feats, n, d, frame, s, blockIdx.x - tiles, nr);
}

// ---------------------------------------------------------------------------
constexpr int kEpiTile = 64;

// log1p from the hardware base-2 logarithm with Goldberg's correction
// (D. Goldberg, "What every computer scientist should know about
// floating-point arithmetic", 1991, Thm. 4): with u = fl(1 + x), log1p(x) =
// log(u) x / (u - 1) to within a few ulps, and x itself when u rounds to 1.
// The library's log1pf made the epilogue bound by instruction issue.
__device__ __forceinline__ float log1p_hw(float x) {
  const float u = 1.f + x;
  const float d = u - 1.f;
  return d == 0.f ? x : __builtin_amdgcn_logf(u) * 0.69314718055994531f * (x * __builtin_amdgcn_rcpf(d));
}

__device__ __forceinline__ float phi_kappa(float z, float kappa, float inv_log1p_kappa) {
  return kappa > 0.f ? log1p_hw(kappa * z) * inv_log1p_kappa : z;
}

// Block = one upper tile pair (ti <= tj) of 64 x 64.  The upper tile holds
// d_f(i, j) from the Gram (rows i in ti, columns j in tj).  It becomes
// C_tm[i][j] = C(s = j, t = i) in place, and its mirror C_tm[j][i] = C(s = i, t = j)
// is staged through LDS and written transposed.  With VEC (n % 4 == 0) a
// thread moves 4 consecutive columns per 16-byte load and store: 16 threads
// cover a tile row of 256 bytes.
template <bool VEC>
__global__ __launch_bounds__(256) void fst_epilogue_kernel(FstParams p, FstScratch s) {
  int ti, tj;
  upper_tile(blockIdx.x, ti, tj);
  const int n = p.n;
  __shared__ float rx[kEpiTile], ry[kEpiTile], rz[kEpiTile], cx[kEpiTile], cy[kEpiTile], cz[kEpiTile];
  __shared__ int rf[kEpiTile], cf[kEpiTile];
  __shared__ float tr[kEpiTile][kEpiTile + 1];

  const int t = threadIdx.x;
  if (t < kEpiTile) {
    const int i = ti * kEpiTile + t;
    if (i < n) {
      rx[t] = p.pos[3 * i];
      ry[t] = p.pos[3 * i + 1];
      rz[t] = p.pos[3 * i + 2];
      rf[t] = p.frame[i];
    }
  } else if (t < 2 * kEpiTile) {
    const int c = t - kEpiTile, j = tj * kEpiTile + c;
    if (j < n) {
      cx[c] = p.pos[3 * j];
      cy[c] = p.pos[3 * j + 1];
      cz[c] = p.pos[3 * j + 2];
      cf[c] = p.frame[j];
    }
  }

  const float m_f = __uint_as_float(*s.mf_bits);
  const float m_x = float(sqrt(__longlong_as_double((long long)*s.mx2_bits)));
  const int m_t = *s.tau_max - *s.tau_min;
  if (blockIdx.x == 0 && t == 0 && p.maxima) {
    p.maxima[0] = m_f;
    p.maxima[1] = m_x;
    p.maxima[2] = float(m_t);
  }
  const float wf = m_f > 0.f ? p.lambda_f / m_f : 0.f;
  const float inv_mx = m_x > 0.f ? 1.f / m_x : 0.f;
  const float wt = m_t > 0 ? p.lambda_tau / float(m_t) : 0.f;
  __syncthreads();

  const bool mirror = ti != tj;
  // Both terms of an entry from its raw d_f; writes the mirror value to LDS.
  auto cost_at = [&](int r, int c, float df) {
    const float dx = rx[r] - cx[c], dy = ry[r] - cy[c], dz = rz[r] - cz[c];
    const float dist = __builtin_amdgcn_sqrtf(dx * dx + dy * dy + dz * dz);   // v_sqrt_f32, 1 ulp
    const float base = wf * df + p.lambda_x * phi_kappa(dist * inv_mx, p.kappa, p.inv_log1p_kappa);
    if (mirror) tr[c][r] = base + wt * float(max(0, rf[r] - cf[c]));
    return base + wt * float(max(0, cf[c] - rf[r]));
  };
  const bool full = (ti + 1) * kEpiTile <= n && (tj + 1) * kEpiTile <= n;
  if (VEC && full) {
    const int c4 = (t & 15) * 4;
#pragma unroll 4
    for (int r = t >> 4; r < kEpiTile; r += 16) {
      float4* at = reinterpret_cast<float4*>(p.cost + size_t(ti * kEpiTile + r) * n + tj * kEpiTile + c4);
      const float4 df = *at;
      float4 out;
      out.x = cost_at(r, c4, df.x);
      out.y = cost_at(r, c4 + 1, df.y);
      out.z = cost_at(r, c4 + 2, df.z);
      out.w = cost_at(r, c4 + 3, df.w);
      *at = out;
    }
    if (!mirror) return;
    __syncthreads();
#pragma unroll 2
    for (int r = t >> 4; r < kEpiTile; r += 16) {
      float4 v;
      v.x = tr[r][c4];
      v.y = tr[r][c4 + 1];
      v.z = tr[r][c4 + 2];
      v.w = tr[r][c4 + 3];
      *reinterpret_cast<float4*>(p.cost + size_t(tj * kEpiTile + r) * n + ti * kEpiTile + c4) = v;
    }
    return;
  }
  const int c = t & 63;
  const int j = tj * kEpiTile + c;
#pragma unroll 4
  for (int r = t >> 6; r < kEpiTile; r += 4) {
    const int i = ti * kEpiTile + r;
    if (i < n && j < n) {
      const size_t at = size_t(i) * n + j;
      p.cost[at] = cost_at(r, c, p.cost[at]);
    }
  }
  if (!mirror) return;
  __syncthreads();
  const int i = ti * kEpiTile + c;
#pragma unroll 4
  for (int r = t >> 6; r < kEpiTile; r += 4) {
    const int jr = tj * kEpiTile + r;
    if (jr < n && i < n) p.cost[size_t(jr) * n + i] = tr[r][c];
  }
}

// The epilogue of coverprune_prune (n a multiple of 64): the cost as above,
// and for the greedy that follows it the source-major copy T and the step-0
// gains, so that the greedy needs no pass of its own over the cost.  For the
// upper tile pair (ti, tj), with X[r][c] = C(s = j_c, t = i_r) (the tile's
// own entries) and Y[r][c] = C(s = i_r, t = j_c) (its mirror's, transposed):
//   C_tm tile (ti, tj) = X and, off the diagonal, C_tm tile (tj, ti) = Y^T;
//   T tile (tj, ti) = X^T and, off the diagonal, T tile (ti, tj) = Y;
//   part[ti][j_c] = sum_r fx(v_{i_r} max(0, c0 - X[r][c])) and, off the
//   diagonal, part[tj][i_r] = sum_c fx(v_{j_c} max(0, c0 - Y[r][c])).
// Every (64-target block, column) partial is written exactly once, and the
// greedy adds the n / 64 partials of a column in 64-bit integers, so the
// gains do not depend on the split.  A thread holds 4 rows x 4 columns of
// both X and Y; the two transposed tiles go through LDS one after the other.
__global__ __launch_bounds__(256) void fst_epilogue_sgs_kernel(FstParams p, FstScratch s, EpiSgs g) {
  int ti, tj;
  upper_tile(blockIdx.x, ti, tj);
  const int n = p.n;
  __shared__ float rx[kEpiTile], ry[kEpiTile], rz[kEpiTile], cx[kEpiTile], cy[kEpiTile], cz[kEpiTile];
  __shared__ int rf[kEpiTile], cf[kEpiTile];
  __shared__ double rvs[kEpiTile], cvs[kEpiTile];
  __shared__ float tr[kEpiTile][kEpiTile + 1];
  __shared__ long long red[4][kEpiTile];

  const int t = threadIdx.x, lane = t & 63, w = t >> 6;
  const int S = *g.scale;
  if (t < kEpiTile) {
    const int i = ti * kEpiTile + t;
    rx[t] = p.pos[3 * i];
    ry[t] = p.pos[3 * i + 1];
    rz[t] = p.pos[3 * i + 2];
    rf[t] = p.frame[i];
    rvs[t] = fx_scale(double(g.v[i]), S);
  } else if (t < 2 * kEpiTile) {
    const int c = t - kEpiTile, j = tj * kEpiTile + c;
    cx[c] = p.pos[3 * j];
    cy[c] = p.pos[3 * j + 1];
    cz[c] = p.pos[3 * j + 2];
    cf[c] = p.frame[j];
    cvs[c] = fx_scale(double(g.v[j]), S);
  }
  const float m_f = __uint_as_float(*s.mf_bits);
  const float m_x = float(sqrt(__longlong_as_double((long long)*s.mx2_bits)));
  const int m_t = *s.tau_max - *s.tau_min;
  if (blockIdx.x == 0 && t == 0 && p.maxima) {
    p.maxima[0] = m_f;
    p.maxima[1] = m_x;
    p.maxima[2] = float(m_t);
  }
  const float wf = m_f > 0.f ? p.lambda_f / m_f : 0.f;
  const float inv_mx = m_x > 0.f ? 1.f / m_x : 0.f;
  const float wt = m_t > 0 ? p.lambda_tau / float(m_t) : 0.f;
  __syncthreads();

  const bool mirror = ti != tj;
  const int c4 = (t & 15) * 4, r0 = t >> 4;
  float X[4][4], Y[4][4];
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int r = r0 + 16 * k;
    float4* at = reinterpret_cast<float4*>(p.cost + size_t(ti * kEpiTile + r) * n + tj * kEpiTile + c4);
    const float4 df4 = *at;
    const float df[4] = {df4.x, df4.y, df4.z, df4.w};
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int c = c4 + u;
      const float dx = rx[r] - cx[c], dy = ry[r] - cy[c], dz = rz[r] - cz[c];
      const float dist = __builtin_amdgcn_sqrtf(dx * dx + dy * dy + dz * dz);
      const float base = wf * df[u] + p.lambda_x * phi_kappa(dist * inv_mx, p.kappa, p.inv_log1p_kappa);
      X[k][u] = base + wt * float(max(0, cf[c] - rf[r]));
      Y[k][u] = base + wt * float(max(0, rf[r] - cf[c]));
    }
    *at = make_float4(X[k][0], X[k][1], X[k][2], X[k][3]);
    if (mirror)
      *reinterpret_cast<float4*>(g.T + size_t(ti * kEpiTile + r) * g.ldt + tj * kEpiTile + c4) =
          make_float4(Y[k][0], Y[k][1], Y[k][2], Y[k][3]);
  }

  // Step-0 partial gains.  Column sums of X: a thread's four rows, then the
  // lanes 16 and 32 apart (same columns, other rows), then the four waves.
  unsigned long long xs[4];
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    long long a = 0;
#pragma unroll
    for (int k = 0; k < 4; ++k) a += fx_term(rvs[r0 + 16 * k], fmaxf(g.c0 - X[k][u], 0.f));
    xs[u] = (unsigned long long)a;
#pragma unroll
    for (int o = 16; o < 64; o <<= 1) xs[u] += __shfl_xor(xs[u], o);
  }
  if (lane < 16) {
#pragma unroll
    for (int u = 0; u < 4; ++u) red[w][c4 + u] = (long long)xs[u];
  }
  // Row sums of Y (mirror tiles): a thread's four columns, then the 16 lanes
  // of its row (a DPP row).
  if (mirror) {
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      long long a = 0;
#pragma unroll
      for (int u = 0; u < 4; ++u) a += fx_term(cvs[c4 + u], fmaxf(g.c0 - Y[k][u], 0.f));
      unsigned long long y = (unsigned long long)a;
      y += dpp_u64<0xB1>(y);    // quad_perm [1,0,3,2]
      y += dpp_u64<0x4E>(y);    // quad_perm [2,3,0,1]
      y += dpp_u64<0x141>(y);   // row_half_mirror
      y += dpp_u64<0x140>(y);   // row_mirror
      if ((t & 15) == 0) g.part[size_t(tj) * n + ti * kEpiTile + r0 + 16 * k] = (long long)y;
    }
  }
  __syncthreads();
  if (t < kEpiTile)
    g.part[size_t(ti) * n + tj * kEpiTile + t] = red[0][t] + red[1][t] + red[2][t] + red[3][t];

  // Off the diagonal, C_tm tile (tj, ti) = Y^T; then T tile (tj, ti) = X^T
  // (on the diagonal too: there the Gram's two triangles can differ in the
  // last bit, so T is the cost's own transpose rather than Y), through LDS.
  if (mirror) {
#pragma unroll
    for (int k = 0; k < 4; ++k)
#pragma unroll
      for (int u = 0; u < 4; ++u) tr[c4 + u][r0 + 16 * k] = Y[k][u];
    __syncthreads();
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int r = r0 + 16 * k;
      *reinterpret_cast<float4*>(p.cost + size_t(tj * kEpiTile + r) * n + ti * kEpiTile + c4) =
          make_float4(tr[r][c4], tr[r][c4 + 1], tr[r][c4 + 2], tr[r][c4 + 3]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int k = 0; k < 4; ++k)
#pragma unroll
    for (int u = 0; u < 4; ++u) tr[c4 + u][r0 + 16 * k] = X[k][u];
  __syncthreads();
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int r = r0 + 16 * k;
    *reinterpret_cast<float4*>(g.T + size_t(tj * kEpiTile + r) * g.ldt + ti * kEpiTile + c4) =
        make_float4(tr[r][c4], tr[r][c4 + 1], tr[r][c4 + 2], tr[r][c4 + 3]);
  }
}

int tiles_of(int n, int tile) { return (n + tile - 1) / tile; }

}  // namespace

hipError_t launch_fst_prep(const FstParams& p, const FstScratch& s, hipStream_t stream) {
  fst_init_kernel<<<1, 1, 0, stream>>>(s);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int nr = std::min((p.n + kPrepWaves - 1) / kPrepWaves, 1024);
  const int t = tiles_of(p.n, kPosTile);
  const int tiles = t * (t + 1) / 2;
  if (p.bf16)
    fst_prep_kernel<true><<<tiles + nr, kPrepThreads, 0, stream>>>(p.feats, p.n, p.d, p.frame, p.pos, tiles, nr, s);
  else
    fst_prep_kernel<false><<<tiles + nr, kPrepThreads, 0, stream>>>(p.feats, p.n, p.d, p.frame, p.pos, tiles, nr, s);
  return hipGetLastError();
}

hipError_t launch_fst_epilogue_sgs(const FstParams& p, const FstScratch& s, const EpiSgs& g, hipStream_t stream) {
  if (p.n % kEpiTile != 0) return hipErrorInvalidValue;
  const int t = p.n / kEpiTile;
  fst_epilogue_sgs_kernel<<<t * (t + 1) / 2, 256, 0, stream>>>(p, s, g);
  return hipGetLastError();
}

hipError_t launch_fst_epilogue(const FstParams& p, const FstScratch& s, hipStream_t stream) {
  const int t = tiles_of(p.n, kEpiTile);
  if (p.n % 4 == 0)
    fst_epilogue_kernel<true><<<t * (t + 1) / 2, 256, 0, stream>>>(p, s);
  else
    fst_epilogue_kernel<false><<<t * (t + 1) / 2, 256, 0, stream>>>(p, s);
  return hipGetLastError();
}

}  // namespace cp
