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
#include "launch.h"

namespace cp {
namespace {

__global__ void fst_init_kernel(FstScratch s) {
  *s.mf_bits = 0u;
  *s.mx2_bits = 0ull;
  *s.tau_min = INT_MAX;
  *s.tau_max = INT_MIN;
}

// Inverse feature norms: each wave walks rows blockIdx.x * 8 + w, + 8 *
// gridDim.x, ..., with a row's 16-byte loads (up to 8 per lane) in flight
// together.  Frame indices fold into a per-block range first, so the grid
// issues only two atomics per block.
template <bool BF16>
__global__ __launch_bounds__(512) void row_norm_kernel(const void* feats, int n, int d,
                                                       const int32_t* frame, FstScratch s) {
  const int lane = threadIdx.x & 63, wib = threadIdx.x >> 6;
  int fmin = INT_MAX, fmax = INT_MIN;
  const int m = BF16 ? d / 8 : d / 4;   // 16-byte chunks per row
  for (int row = blockIdx.x * 8 + wib; row < n; row += gridDim.x * 8) {
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
  __shared__ int smin[8], smax[8];
  if (lane == 0) {
    smin[wib] = fmin;
    smax[wib] = fmax;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    int lo = smin[0], hi = smax[0];
    for (int w = 1; w < 8; ++w) {
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
// 256 x 256 tile (enough waves in flight to hide the float64 latency), a
// thread takes one row of the tile against the tile's columns staged in LDS,
// and a block whose maximum is larger than the running one raises it.
__global__ __launch_bounds__(256) void pos_pairmax_kernel(const float* pos, int n, int ntiles, FstScratch s) {
  __shared__ double sx[kPosTile], sy[kPosTile], sz[kPosTile];
  __shared__ double sm[4];
  double best = 0.0;
  for (int b = blockIdx.x; b < ntiles; b += gridDim.x) {
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

int tiles_of(int n, int tile) { return (n + tile - 1) / tile; }

}  // namespace

hipError_t launch_fst_prep(const FstParams& p, const FstScratch& s, hipStream_t stream) {
  fst_init_kernel<<<1, 1, 0, stream>>>(s);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int nb = std::min((p.n + 7) / 8, 512);
  if (p.bf16)
    row_norm_kernel<true><<<nb, 512, 0, stream>>>(p.feats, p.n, p.d, p.frame, s);
  else
    row_norm_kernel<false><<<nb, 512, 0, stream>>>(p.feats, p.n, p.d, p.frame, s);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  const int t = tiles_of(p.n, kPosTile);
  const int tiles = t * (t + 1) / 2;
  pos_pairmax_kernel<<<tiles, 256, 0, stream>>>(p.pos, p.n, tiles, s);
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
