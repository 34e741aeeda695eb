// FST capacity (Sec. 3.4, Eq. 9-10).
//
// r_j = (1/n) sum_{k in N_n(j)} (a_f d_f(j,k)/M_f + a_x d_x(j,k)/M_x + a_tau d_tau(j,k)/M_tau),
// v_j = r_j / sum_l r_l (uniform when every r is 0).  N_n(j) is the n tokens
// nearest to j other than j, by (squared distance, index): the first n
// entries of j's (n+1)-nearest table with j left out.  d_f = 1 - cos clamped
// to [0, 2] (cos = 0 for a zero-norm row), d_x the Euclidean distance,
// d_tau(j, k) = ReLU(tau_j - tau_k); each M is the maximum of its term over
// the n * N scored pairs (a term whose maximum is 0 contributes 0).
//
// Kernels, in stream order:
//   knn tables with g = n + 1 (k_knn.hip)
//   cap_pairs_kernel     one wave per token: gathers each neighbour's feature
//                        row, dot product and norms in float64 (bf16 and f32
//                        products are exact there), writes the three
//                        discrepancies and raises the maxima
//   cap_score_kernel     r_j and per-block partial sums of r in fixed order
//   cap_normalise_kernel v_j = r_j / sum r, the sum taken from the partials
//                        in the same fixed order by every block
#include <hip/hip_runtime.h>

#include <algorithm>

#include "common.h"
#include "launch.h"

namespace cp {
namespace {

constexpr int kCapBlock = 256;
constexpr int kCapWaves = kCapBlock / kWave;

struct CapDev {
  const void* feats;
  int n, d, g, nn;                 // tokens, feature width, table width (nn + 1), neighbours
  const float* pos;
  const int32_t* frame;
  const int32_t* table;            // [n, g]
  double* pairs;                   // [n, nn, 3]
  unsigned long long* maxbits;     // [3] float64 bits of M_f, M_x, M_tau
  double a_f, a_x, a_t;
  double* r;                       // [n]
  double* partial;                 // [ceil(n / kCapBlock)]
  float* v;                        // [n]
};

__global__ void cap_init_kernel(unsigned long long* maxbits) {
  if (threadIdx.x < 3) maxbits[threadIdx.x] = 0ull;
}

// Sum over the wave's lanes of f_a . f_b and |f_b|^2 (and |f_a|^2 when
// want_aa), float64.  Rows are read as 16-byte chunks: 8 bf16 or 4 float.
template <bool BF16>
__device__ __forceinline__ void row_dots(const void* feats, int d, int a, int b, double& ab, double& bb) {
  const int lane = threadIdx.x & (kWave - 1);
  const int chunks = BF16 ? d / 8 : d / 4;
  const uint4* ra = reinterpret_cast<const uint4*>(feats) + size_t(a) * chunks;
  const uint4* rb = reinterpret_cast<const uint4*>(feats) + size_t(b) * chunks;
  double s_ab = 0.0, s_bb = 0.0;
  for (int c = lane; c < chunks; c += kWave) {
    const uint4 x = ra[c], y = rb[c];
    const unsigned int xw[4] = {x.x, x.y, x.z, x.w}, yw[4] = {y.x, y.y, y.z, y.w};
#pragma unroll
    for (int h = 0; h < 4; ++h) {
      if (BF16) {
        const double x0 = bf16_bits_to_float(xw[h] & 0xffffu), x1 = bf16_bits_to_float(xw[h] >> 16);
        const double y0 = bf16_bits_to_float(yw[h] & 0xffffu), y1 = bf16_bits_to_float(yw[h] >> 16);
        s_ab = fma(x0, y0, s_ab);
        s_ab = fma(x1, y1, s_ab);
        s_bb = fma(y0, y0, s_bb);
        s_bb = fma(y1, y1, s_bb);
      } else {
        const double x0 = __uint_as_float(xw[h]), y0 = __uint_as_float(yw[h]);
        s_ab = fma(x0, y0, s_ab);
        s_bb = fma(y0, y0, s_bb);
      }
    }
  }
  ab = wave_sum(s_ab);
  bb = wave_sum(s_bb);
}

template <bool BF16>
__global__ __launch_bounds__(kCapBlock) void cap_pairs_kernel(CapDev p) {
  __shared__ double smax[kCapWaves][3];
  const int lane = threadIdx.x & (kWave - 1), w = threadIdx.x >> 6;
  const int j = blockIdx.x * kCapWaves + w;
  double mf = 0.0, mx = 0.0, mt = 0.0;
  if (j < p.n) {
    double jj, unused;
    row_dots<BF16>(p.feats, p.d, j, j, unused, jj);
    const double nj = sqrt(jj);
    const float xj = p.pos[3 * j], yj = p.pos[3 * j + 1], zj = p.pos[3 * j + 2];
    const int tj = p.frame[j];
    int q = 0;
    for (int e = 0; e < p.g && q < p.nn; ++e) {
      const int k = __builtin_amdgcn_readfirstlane(p.table[size_t(j) * p.g + e]);
      if (k == j) continue;
      double jk, kk;
      row_dots<BF16>(p.feats, p.d, j, k, jk, kk);
      const double den = nj * sqrt(kk);
      const double cosv = den > 0.0 ? jk / den : 0.0;
      const double df = fmin(fmax(1.0 - cosv, 0.0), 2.0);
      double dx;
      {
#pragma clang fp contract(off)
        const double ex = double(xj) - double(p.pos[3 * k]), ey = double(yj) - double(p.pos[3 * k + 1]),
                     ez = double(zj) - double(p.pos[3 * k + 2]);
        dx = sqrt((ex * ex + ey * ey) + ez * ez);
      }
      const double dt = fmax(double(tj) - double(p.frame[k]), 0.0);
      if (lane == 0) {
        double* o = p.pairs + (size_t(j) * p.nn + q) * 3;
        o[0] = df;
        o[1] = dx;
        o[2] = dt;
      }
      mf = fmax(mf, df);
      mx = fmax(mx, dx);
      mt = fmax(mt, dt);
      ++q;
    }
  }
  if (lane == 0) {
    smax[w][0] = mf;
    smax[w][1] = mx;
    smax[w][2] = mt;
  }
  __syncthreads();
  if (threadIdx.x < 3) {
    double m = 0.0;
#pragma unroll
    for (int u = 0; u < kCapWaves; ++u) m = fmax(m, smax[u][threadIdx.x]);
    atomic_max_nonneg(p.maxbits + threadIdx.x, m);
  }
}

__global__ __launch_bounds__(kCapBlock) void cap_score_kernel(CapDev p) {
  __shared__ double red[kCapBlock];
  const int j = blockIdx.x * kCapBlock + threadIdx.x;
  const double M_f = __longlong_as_double((long long)p.maxbits[0]);
  const double M_x = __longlong_as_double((long long)p.maxbits[1]);
  const double M_t = __longlong_as_double((long long)p.maxbits[2]);
  double r = 0.0;
  if (j < p.n) {
    double s = 0.0;
    const double* o = p.pairs + size_t(j) * p.nn * 3;
    for (int q = 0; q < p.nn; ++q) {
      const double tf = M_f > 0.0 ? o[3 * q] / M_f : 0.0;
      const double tx = M_x > 0.0 ? o[3 * q + 1] / M_x : 0.0;
      const double tt = M_t > 0.0 ? o[3 * q + 2] / M_t : 0.0;
      s += (p.a_f * tf + p.a_x * tx) + p.a_t * tt;
    }
    r = s / double(p.nn);
    p.r[j] = r;
  }
  red[threadIdx.x] = r;
  __syncthreads();
  for (int h = kCapBlock / 2; h > 0; h >>= 1) {
    if (threadIdx.x < h) red[threadIdx.x] += red[threadIdx.x + h];
    __syncthreads();
  }
  if (threadIdx.x == 0) p.partial[blockIdx.x] = red[0];
}

__global__ __launch_bounds__(kCapBlock) void cap_normalise_kernel(CapDev p, int nparts) {
  __shared__ double stotal;
  if (threadIdx.x == 0) {
    double t = 0.0;
    for (int b = 0; b < nparts; ++b) t += p.partial[b];
    stotal = t;
  }
  __syncthreads();
  const double total = stotal;
  const int j = blockIdx.x * kCapBlock + threadIdx.x;
  if (j < p.n) p.v[j] = total > 0.0 ? float(p.r[j] / total) : float(1.0 / double(p.n));
}

size_t align256(size_t x) { return (x + 255) / 256 * 256; }

struct CapLayout {
  size_t table, pairs, maxbits, r, partial, total;
};

CapLayout cap_layout(int64_t n, int64_t nn) {
  CapLayout L;
  size_t o = 0;
  L.table = o;
  o = align256(o + size_t(n) * size_t(nn + 1) * 4);
  L.pairs = o;
  o = align256(o + size_t(n) * size_t(nn) * 24);
  L.maxbits = o;
  o = align256(o + 3 * 8);
  L.r = o;
  o = align256(o + size_t(n) * 8);
  L.partial = o;
  o = align256(o + size_t((n + kCapBlock - 1) / kCapBlock) * 8);
  L.total = o;
  return L;
}

}  // namespace

size_t capacity_workspace_bytes(int64_t n, int64_t nn) { return cap_layout(n, nn).total; }

hipError_t launch_capacity(const CapacityParams& c, hipStream_t stream) {
  const CapLayout L = cap_layout(c.n, c.nn);
  char* w = static_cast<char*>(c.workspace);
  CapDev p{};
  p.feats = c.feats;
  p.n = c.n;
  p.d = c.d;
  p.g = c.nn + 1;
  p.nn = c.nn;
  p.pos = c.pos;
  p.frame = c.frame;
  p.table = reinterpret_cast<int32_t*>(w + L.table);
  p.pairs = reinterpret_cast<double*>(w + L.pairs);
  p.maxbits = reinterpret_cast<unsigned long long*>(w + L.maxbits);
  p.a_f = c.alpha_f;
  p.a_x = c.alpha_x;
  p.a_t = c.alpha_tau;
  p.r = c.score ? c.score : reinterpret_cast<double*>(w + L.r);
  p.partial = reinterpret_cast<double*>(w + L.partial);
  p.v = c.capacity;

  hipError_t e;
  cap_init_kernel<<<1, 64, 0, stream>>>(p.maxbits);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if ((e = launch_knn(c.pos, c.n, p.g, reinterpret_cast<int32_t*>(w + L.table), stream)) != hipSuccess) return e;
  const int pair_blocks = (c.n + kCapWaves - 1) / kCapWaves;
  if (c.bf16)
    cap_pairs_kernel<true><<<pair_blocks, kCapBlock, 0, stream>>>(p);
  else
    cap_pairs_kernel<false><<<pair_blocks, kCapBlock, 0, stream>>>(p);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  const int blocks = (c.n + kCapBlock - 1) / kCapBlock;
  cap_score_kernel<<<blocks, kCapBlock, 0, stream>>>(p);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  cap_normalise_kernel<<<blocks, kCapBlock, 0, stream>>>(p, blocks);
  return hipGetLastError();
}

}  // namespace cp
