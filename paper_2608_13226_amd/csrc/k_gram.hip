// Feature Gram on the matrix cores -> raw feature discrepancy d_f (Eq. 7).
//
// d_f(i, j) = clamp(1 - <f_i, f_j> / (|f_i| |f_j|), 0, 2), d_f(i, i) = 0.  The
// Gram is symmetric, so only tiles with row-tile <= column-tile are computed
// (N(N+1)D multiply-adds instead of 2 N^2 D); each writes its d_f values at
// [i][j] and folds them into the global maximum M_f.  The epilogue kernel
// mirrors the lower triangle.
//
// bf16: v_mfma_f32_32x32x16_bf16, fp32 accumulation.  f32: v_mfma_f32_32x32x2f32.
// Block tile 128 x 128, four waves in a 2 x 2 arrangement of 64 x 64 wave
// tiles (2 x 2 MFMA 32 x 32 tiles each); K staged through LDS.
#include <hip/hip_runtime.h>

#include "common.h"
#include "launch.h"

namespace cp {
namespace {

constexpr int kTile = 128;

__device__ __forceinline__ void upper_tile(int b, int& ti, int& tj) {
  int j = int((sqrt(8.0 * double(b) + 1.0) - 1.0) * 0.5);
  while (j * (j + 1) / 2 > b) --j;
  while ((j + 1) * (j + 2) / 2 <= b) ++j;
  tj = j;
  ti = b - j * (j + 1) / 2;
}

// Accumulator element (mi, ni, r) of lane `lane` in a 32x32 MFMA output sits at
// row 8*(r/4) + 4*(lane/32) + r%4 and column lane%32 of that 32x32 tile.
__device__ __forceinline__ void store_df(const f32x16 (&acc)[2][2], int row0, int col0, int wm, int wn,
                                         int lane, int n, const float* inv_norm, float* out,
                                         unsigned int* mf_bits) {
  float lmax = 0.f;
#pragma unroll
  for (int ni = 0; ni < 2; ++ni) {
    const int col = col0 + wn * 64 + ni * 32 + (lane & 31);
    const float rc = col < n ? inv_norm[col] : 0.f;
#pragma unroll
    for (int mi = 0; mi < 2; ++mi) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = row0 + wm * 64 + mi * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
        if (row < n && col < n) {
          const float cosv = acc[mi][ni][r] * inv_norm[row] * rc;
          float df = fminf(fmaxf(1.f - cosv, 0.f), 2.f);
          if (row == col) df = 0.f;
          out[size_t(row) * n + col] = df;
          lmax = fmaxf(lmax, df);
        }
      }
    }
  }
  lmax = wave_max(lmax);
  if (lane == 0) atomic_max_nonneg(mf_bits, lmax);
}

// ---------------------------------------------------------------------------
constexpr int kBkB = 64;           // K per LDS stage (bf16 elements)
constexpr int kLdB = kBkB + 8;     // padded LDS row (bf16 elements): conflict-free 16 B reads

__global__ __launch_bounds__(256) void gram_bf16_kernel(const uint16_t* __restrict__ F, int n, int d,
                                                        const float* __restrict__ inv_norm,
                                                        float* __restrict__ out, unsigned int* mf_bits) {
  int ti, tj;
  upper_tile(blockIdx.x, ti, tj);
  const int row0 = ti * kTile, col0 = tj * kTile;
  const bool diag = ti == tj;
  __shared__ __attribute__((aligned(16))) uint16_t As[kTile * kLdB];
  __shared__ __attribute__((aligned(16))) uint16_t Bs[kTile * kLdB];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  f32x16 acc[2][2];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[a][b][r] = 0.f;

  // Global -> register staging: 128 rows x 64 bf16 = 1024 chunks of 16 B per
  // operand; thread t moves chunks t + 256 i (8 threads cover one 128 B row slice).
  uint4 ra0, ra1, ra2, ra3, rb0, rb1, rb2, rb3;
  const int lr = tid >> 3, lk = (tid & 7) * 8;   // chunk row (+32 i) and K offset
  const uint4 zero = {0u, 0u, 0u, 0u};
#define CP_GLOAD_B(R, ROW0, I, K0)                                                     \
  {                                                                                    \
    const int gr = ROW0 + lr + 32 * I, kc = K0 + lk;                                   \
    R = (gr < n && kc < d) ? *reinterpret_cast<const uint4*>(F + size_t(gr) * d + kc) : zero; \
  }
#define CP_GLOAD_ALL_B(K0)                                                             \
  CP_GLOAD_B(ra0, row0, 0, K0) CP_GLOAD_B(ra1, row0, 1, K0)                            \
  CP_GLOAD_B(ra2, row0, 2, K0) CP_GLOAD_B(ra3, row0, 3, K0)                            \
  if (!diag) {                                                                         \
    CP_GLOAD_B(rb0, col0, 0, K0) CP_GLOAD_B(rb1, col0, 1, K0)                          \
    CP_GLOAD_B(rb2, col0, 2, K0) CP_GLOAD_B(rb3, col0, 3, K0)                          \
  }

  const uint16_t* Bsrc = diag ? As : Bs;
  CP_GLOAD_ALL_B(0)
  for (int k0 = 0; k0 < d; k0 += kBkB) {
    __syncthreads();
    *reinterpret_cast<uint4*>(&As[(lr + 0) * kLdB + lk]) = ra0;
    *reinterpret_cast<uint4*>(&As[(lr + 32) * kLdB + lk]) = ra1;
    *reinterpret_cast<uint4*>(&As[(lr + 64) * kLdB + lk]) = ra2;
    *reinterpret_cast<uint4*>(&As[(lr + 96) * kLdB + lk]) = ra3;
    if (!diag) {
      *reinterpret_cast<uint4*>(&Bs[(lr + 0) * kLdB + lk]) = rb0;
      *reinterpret_cast<uint4*>(&Bs[(lr + 32) * kLdB + lk]) = rb1;
      *reinterpret_cast<uint4*>(&Bs[(lr + 64) * kLdB + lk]) = rb2;
      *reinterpret_cast<uint4*>(&Bs[(lr + 96) * kLdB + lk]) = rb3;
    }
    __syncthreads();
    if (k0 + kBkB < d) { CP_GLOAD_ALL_B(k0 + kBkB) }
#pragma unroll
    for (int kk = 0; kk < kBkB / 16; ++kk) {
      bf16x8 a[2], b[2];
      const int koff = kk * 16 + (lane >> 5) * 8;
#pragma unroll
      for (int mi = 0; mi < 2; ++mi)
        a[mi] = *reinterpret_cast<const bf16x8*>(&As[(wm * 64 + mi * 32 + (lane & 31)) * kLdB + koff]);
#pragma unroll
      for (int ni = 0; ni < 2; ++ni)
        b[ni] = *reinterpret_cast<const bf16x8*>(&Bsrc[(wn * 64 + ni * 32 + (lane & 31)) * kLdB + koff]);
#pragma unroll
      for (int mi = 0; mi < 2; ++mi)
#pragma unroll
        for (int ni = 0; ni < 2; ++ni)
          acc[mi][ni] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[mi], b[ni], acc[mi][ni], 0, 0, 0);
    }
  }
#undef CP_GLOAD_ALL_B
#undef CP_GLOAD_B
  store_df(acc, row0, col0, wm, wn, lane, n, inv_norm, out, mf_bits);
}

// ---------------------------------------------------------------------------
constexpr int kBkF = 32;           // K per LDS stage (floats)
constexpr int kLdF = kBkF + 4;

__global__ __launch_bounds__(256) void gram_f32_kernel(const float* __restrict__ F, int n, int d,
                                                       const float* __restrict__ inv_norm,
                                                       float* __restrict__ out, unsigned int* mf_bits) {
  int ti, tj;
  upper_tile(blockIdx.x, ti, tj);
  const int row0 = ti * kTile, col0 = tj * kTile;
  const bool diag = ti == tj;
  __shared__ __attribute__((aligned(16))) float As[kTile * kLdF];
  __shared__ __attribute__((aligned(16))) float Bs[kTile * kLdF];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  f32x16 acc[2][2];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[a][b][r] = 0.f;

  // 128 rows x 32 floats = 1024 chunks of 16 B per operand.
  f32x4 ra0, ra1, ra2, ra3, rb0, rb1, rb2, rb3;
  const int lr = tid >> 3, lk = (tid & 7) * 4;
#define CP_GLOAD_F(R, ROW0, I, K0)                                                      \
  {                                                                                     \
    const int gr = ROW0 + lr + 32 * I, kc = K0 + lk;                                    \
    if (gr < n && kc < d) R = *reinterpret_cast<const f32x4*>(F + size_t(gr) * d + kc); \
    else R = f32x4{0.f, 0.f, 0.f, 0.f};                                                 \
  }
#define CP_GLOAD_ALL_F(K0)                                                              \
  CP_GLOAD_F(ra0, row0, 0, K0) CP_GLOAD_F(ra1, row0, 1, K0)                             \
  CP_GLOAD_F(ra2, row0, 2, K0) CP_GLOAD_F(ra3, row0, 3, K0)                             \
  if (!diag) {                                                                          \
    CP_GLOAD_F(rb0, col0, 0, K0) CP_GLOAD_F(rb1, col0, 1, K0)                           \
    CP_GLOAD_F(rb2, col0, 2, K0) CP_GLOAD_F(rb3, col0, 3, K0)                           \
  }

  const float* Bsrc = diag ? As : Bs;
  CP_GLOAD_ALL_F(0)
  for (int k0 = 0; k0 < d; k0 += kBkF) {
    __syncthreads();
    *reinterpret_cast<f32x4*>(&As[(lr + 0) * kLdF + lk]) = ra0;
    *reinterpret_cast<f32x4*>(&As[(lr + 32) * kLdF + lk]) = ra1;
    *reinterpret_cast<f32x4*>(&As[(lr + 64) * kLdF + lk]) = ra2;
    *reinterpret_cast<f32x4*>(&As[(lr + 96) * kLdF + lk]) = ra3;
    if (!diag) {
      *reinterpret_cast<f32x4*>(&Bs[(lr + 0) * kLdF + lk]) = rb0;
      *reinterpret_cast<f32x4*>(&Bs[(lr + 32) * kLdF + lk]) = rb1;
      *reinterpret_cast<f32x4*>(&Bs[(lr + 64) * kLdF + lk]) = rb2;
      *reinterpret_cast<f32x4*>(&Bs[(lr + 96) * kLdF + lk]) = rb3;
    }
    __syncthreads();
    if (k0 + kBkF < d) { CP_GLOAD_ALL_F(k0 + kBkF) }
    // Each lane reads 4 consecutive k of its row; MFMA u consumes element u, so
    // the two lane halves x four MFMAs cover 8 distinct k per step.
#pragma unroll
    for (int kk = 0; kk < kBkF / 8; ++kk) {
      const int koff = kk * 8 + (lane >> 5) * 4;
      const f32x4 a0 = *reinterpret_cast<const f32x4*>(&As[(wm * 64 + (lane & 31)) * kLdF + koff]);
      const f32x4 a1 = *reinterpret_cast<const f32x4*>(&As[(wm * 64 + 32 + (lane & 31)) * kLdF + koff]);
      const f32x4 b0 = *reinterpret_cast<const f32x4*>(&Bsrc[(wn * 64 + (lane & 31)) * kLdF + koff]);
      const f32x4 b1 = *reinterpret_cast<const f32x4*>(&Bsrc[(wn * 64 + 32 + (lane & 31)) * kLdF + koff]);
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        acc[0][0] = __builtin_amdgcn_mfma_f32_32x32x2f32(a0[u], b0[u], acc[0][0], 0, 0, 0);
        acc[0][1] = __builtin_amdgcn_mfma_f32_32x32x2f32(a0[u], b1[u], acc[0][1], 0, 0, 0);
        acc[1][0] = __builtin_amdgcn_mfma_f32_32x32x2f32(a1[u], b0[u], acc[1][0], 0, 0, 0);
        acc[1][1] = __builtin_amdgcn_mfma_f32_32x32x2f32(a1[u], b1[u], acc[1][1], 0, 0, 0);
      }
    }
  }
#undef CP_GLOAD_ALL_F
#undef CP_GLOAD_F
  store_df(acc, row0, col0, wm, wn, lane, n, inv_norm, out, mf_bits);
}

}  // namespace

hipError_t launch_gram(const FstParams& p, const FstScratch& s, hipStream_t stream) {
  const int t = (p.n + kTile - 1) / kTile;
  const int blocks = t * (t + 1) / 2;
  if (p.bf16)
    gram_bf16_kernel<<<blocks, 256, 0, stream>>>(static_cast<const uint16_t*>(p.feats), p.n, p.d,
                                                 s.inv_norm, p.cost, s.mf_bits);
  else
    gram_f32_kernel<<<blocks, 256, 0, stream>>>(static_cast<const float*>(p.feats), p.n, p.d,
                                                s.inv_norm, p.cost, s.mf_bits);
  return hipGetLastError();
}

}  // namespace cp
