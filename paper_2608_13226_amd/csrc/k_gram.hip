// Feature Gram on the matrix cores -> raw feature discrepancy d_f (Eq. 7).
//
// d_f(i, j) = clamp(1 - <f_i, f_j> / (|f_i| |f_j|), 0, 2), d_f(i, i) = 0.  The
// Gram is symmetric, so only tiles with row-tile <= column-tile are computed
// (N(N+1)D multiply-adds instead of 2 N^2 D); each writes its d_f values at
// [i][j] and folds them into the global maximum M_f.  The epilogue kernel
// mirrors the lower triangle.
//
// bf16: v_mfma_f32_32x32x16_bf16, fp32 accumulation.  f32: v_mfma_f32_32x32x2f32.
// Large bf16 problems use 256 x 256 block tiles (gram_bf16_big_kernel); the
// rest use 128 x 128 block tiles, four waves in a 2 x 2 arrangement of 64 x 64
// wave tiles (2 x 2 MFMA 32 x 32 tiles each), K staged through LDS.
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
// (row0, col0) is the wave's corner.  The inverse norms of a 32-row group are
// fetched before its first store.  A wave block that lies inside the matrix
// and off the diagonal (the common case) stores through a buffer resource
// based at its corner: per-lane 32-bit offsets, row steps in the scalar
// offset, no per-element checks.
template <int MT, int NT>
__device__ __forceinline__ void store_df(const f32x16 (&acc)[MT][NT], int row0, int col0, int lane, int n,
                                         const float* inv_norm, float* out, unsigned int* mf_bits) {
  float rc[NT];
#pragma unroll
  for (int ni = 0; ni < NT; ++ni) rc[ni] = inv_norm[min(col0 + ni * 32 + (lane & 31), n - 1)];
  float lmax = 0.f;
  const bool fast = row0 + MT * 32 <= n && col0 + NT * 32 <= n && (row0 >= col0 + NT * 32 || col0 >= row0 + MT * 32);
  if (fast) {
    float* base = out + size_t(row0) * n + col0;
    const size_t left = (size_t(n) * n - (size_t(row0) * n + col0)) * 4;
    const __amdgpu_buffer_rsrc_t rsrc =
        __builtin_amdgcn_make_buffer_rsrc(base, 0, int(left < 0x7fffffffu ? left : 0x7fffffffu), 0x00020000);
    const int voff = ((4 * (lane >> 5)) * n + (lane & 31)) * 4;
#pragma unroll
    for (int mi = 0; mi < MT; ++mi) {
      float rn[16];
#pragma unroll
      for (int r = 0; r < 16; ++r) rn[r] = inv_norm[row0 + mi * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3)];
#pragma unroll
      for (int ni = 0; ni < NT; ++ni)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float df = fminf(fmaxf(1.f - acc[mi][ni][r] * rn[r] * rc[ni], 0.f), 2.f);
          lmax = fmaxf(lmax, df);
          __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(df), rsrc, voff + ni * 128,
                                                (mi * 32 + 8 * (r >> 2) + (r & 3)) * n * 4, 0);
        }
    }
  } else {
#pragma unroll
    for (int mi = 0; mi < MT; ++mi) {
      float rn[16];
#pragma unroll
      for (int r = 0; r < 16; ++r)
        rn[r] = inv_norm[min(row0 + mi * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3), n - 1)];
#pragma unroll
      for (int ni = 0; ni < NT; ++ni) {
        const int col = col0 + ni * 32 + (lane & 31);
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int row = row0 + mi * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
          float df = fminf(fmaxf(1.f - acc[mi][ni][r] * rn[r] * rc[ni], 0.f), 2.f);
          if (row == col) df = 0.f;
          if (row < n && col < n) {
            out[size_t(row) * n + col] = df;
            lmax = fmaxf(lmax, df);
          }
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

  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
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
  store_df(acc, row0 + wm * 64, col0 + wn * 64, lane, n, inv_norm, out, mf_bits);
}

// ---------------------------------------------------------------------------
// Large-tile bf16 Gram for D % 128 == 0 and n d < 2^30: 256 x 256 block
// tiles, eight waves (two per SIMD) of 128 x 64, K in slabs of 64 (128-byte
// row segments, one cache line per row) with two LDS stages of 64 KB.  Slabs
// go from global memory straight into LDS (buffer_load_dwordx4 ... lds: lane
// l's 16 bytes land at base + 16 l), so the next slab streams in while the
// current one is multiplied.
constexpr int kBig = 256;
constexpr int kBigK = 64;

// LDS serves a 16-byte read for 16 lanes per cycle from 64 four-byte banks,
// so one 256-byte bank row holds two 128-byte slab rows.  The 16-byte chunk
// index is XOR-ed with (row / 2) mod 8: the 16 consecutive rows that one
// operand read touches per cycle then cover all 16 (row mod 2, chunk) bank
// groups.
__device__ __forceinline__ int swz(int row, int chunk) { return row * 8 + (chunk ^ ((row >> 1) & 7)); }

// The upper tile at position `lin` of the band order: the triangle is walked
// in bands of kBand tile rows, column by column.  Each band starts with a
// triangle (column r0 + j holds j + 1 tiles, j < rows - 1) followed by full
// columns of `rows` tiles.
constexpr int kBand = 8;
__device__ __forceinline__ bool band_tile(int lin, int T, int& ti, int& tj) {
  for (int r0 = 0; r0 < T; r0 += kBand) {
    const int rows = min(kBand, T - r0);
    const int tri = rows * (rows - 1) / 2;
    const int size = tri + rows * (T - r0 - rows + 1);
    if (lin < size) {
      if (lin < tri) {
        int j = 0;
        while ((j + 1) * (j + 2) / 2 <= lin) ++j;
        ti = r0 + lin - j * (j + 1) / 2;
        tj = r0 + j;
      } else {
        const int q = lin - tri;
        ti = r0 + q % rows;
        tj = r0 + rows - 1 + q / rows;
      }
      return true;
    }
    lin -= size;
  }
  return false;
}

// Map block b of the `nb` full-tile blocks to an upper tile.  Blocks are
// dealt to the 8 XCDs round-robin, so each XCD gets a contiguous range of
// the band order: the ~32 tiles resident on one XCD span about 4 row and 8
// column panels and share their K slabs through the XCD's L2.  Returns false
// for padding blocks.
__device__ __forceinline__ bool big_tile(int b, int nb, int T, int& ti, int& tj) {
  const int per = (nb + 7) / 8;
  const int lin = (b % 8) * per + b / 8;
  if (lin >= nb) return false;
  return band_tile(lin, T, ti, tj);
}

// Slab loader for R-row operands: instruction i < R / 64 of wave w (eight
// waves) fills LDS slots (R / 64 w + i) * 64 + lane of one operand (slot =
// row * 8 + physical chunk), i.e. row R / 8 w + 8 i + lane / 8 at physical
// chunk lane % 8, holding logical chunk (lane % 8) ^ (lane / 16) ^ (4 (i %
// 2)).  `voff_even` / `voff_odd` are the lane's byte offsets for i = 0 / 1 at
// k = 0; rows past the feature matrix read as zero (buffer range check).
template <int R>
__device__ __forceinline__ void load_slab(uint4* dst, __amdgpu_buffer_rsrc_t rsrc, int voff_even, int voff_odd,
                                          int row_step, int k0, int wave) {
#pragma unroll
  for (int i = 0; i < R / 64; ++i)
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc, dst + (wave * (R / 64) + i) * 64, 16,
                                             ((i & 1) ? voff_odd : voff_even) + (i >> 1) * row_step, k0 * 2, 0, 0);
}

// Operand fragments of one 16-wide K step: MT tiles of A and NT tiles of B
// (32 rows each, 256 slots apart) from slot offsets `ia` / `ib` of the first.
template <int MT, int NT>
__device__ __forceinline__ void load_frags(bf16x8 (&a)[MT], bf16x8 (&b)[NT], const uint4* sa, const uint4* sb,
                                           int ia, int ib) {
#pragma unroll
  for (int m = 0; m < MT; ++m) {
    const uint4 v = sa[ia + m * 256];
    __builtin_memcpy(&a[m], &v, 16);
  }
#pragma unroll
  for (int m = 0; m < NT; ++m) {
    const uint4 v = sb[ib + m * 256];
    __builtin_memcpy(&b[m], &v, 16);
  }
}

template <int MT, int NT>
__device__ __forceinline__ void mma_step(f32x16 (&acc)[MT][NT], const bf16x8 (&a)[MT], const bf16x8 (&b)[NT]) {
#pragma unroll
  for (int mi = 0; mi < MT; ++mi)
#pragma unroll
    for (int ni = 0; ni < NT; ++ni)
      acc[mi][ni] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[mi], b[ni], acc[mi][ni], 0, 0, 0);
}

// Workgroup barrier for the slab pipeline.  Unlike __syncthreads() it does not
// wait for all of this wave's loads: the caller has already waited for the
// slab it is about to read, and the LDS reads of the previous slab have been
// consumed by MFMAs.  The signal fences only keep the compiler from moving
// memory operations across it.
__device__ __forceinline__ void slab_barrier() {
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
  __builtin_amdgcn_s_barrier();
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

// Issue order of K step 0 (8 MFMAs, the 6 fragment reads of step 1, all 8
// loads of the next slab) and of steps 1-2 (8 MFMAs, the 6 reads of the next
// step): memory instructions ride between MFMAs instead of arriving in bursts
// that leave the matrix core idle, and the loads go out early in the slab so
// they have most of it to land.
__device__ __forceinline__ void interleave_first() {
#pragma unroll
  for (int i = 0; i < 6; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // MFMA
    __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);   // DS read
    __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);   // VMEM read
  }
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // MFMA
    __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);   // VMEM read
  }
}
__device__ __forceinline__ void interleave_step() {
#pragma unroll
  for (int i = 0; i < 3; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // MFMA
    __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);   // DS read
  }
  __builtin_amdgcn_sched_group_barrier(0x008, 5, 0);
}

// One slab of the K loop in LDS stage ST: wait for this wave's loads of it,
// barrier so every wave's part has landed and every wave is done with the
// other stage, then run the four K steps, the reads of step kk + 1 issued
// ahead of the MFMAs of step kk and the loads that refill the other stage
// (NX) with slab LOAD (when LOAD >= 0) issued during step 0.  The steps carry
// no branches, which keeps the compiler's per-object tracking of in-flight
// LDS loads intact.
#define CP_BIG_SLAB(ST, NX, LOAD)                                                        \
  {                                                                                      \
    __builtin_amdgcn_s_waitcnt(0xF70); /* vmcnt(0) */                                    \
    slab_barrier();                                                                      \
    load_frags(fa[0], fb[0], ST, ST + R * 8, offa[0], offb[0]);                          \
    __builtin_amdgcn_sched_barrier(0);                                                   \
    _Pragma("unroll") for (int kk = 0; kk < 4; ++kk) {                                   \
      if (kk < 3) load_frags(fa[(kk + 1) & 1], fb[(kk + 1) & 1], ST, ST + R * 8,         \
                             offa[kk + 1], offb[kk + 1]);                                \
      if (kk == 0 && LOAD >= 0) {                                                        \
        load_slab<R>(NX, rsrc, voff_a0, voff_a1, row_step, (LOAD) * kBigK, wave);        \
        load_slab<R>(NX + R * 8, rsrc, voff_b0, voff_b1, row_step, (LOAD) * kBigK, wave); \
      }                                                                                  \
      mma_step(acc, fa[kk & 1], fb[kk & 1]);                                             \
      if (R == kBig && kk == 0) interleave_first();                                      \
      else if (R == kBig && kk < 3) interleave_step();                                   \
      __builtin_amdgcn_sched_barrier(0);                                                 \
    }                                                                                    \
  }

// Eight waves in a 2 x 4 arrangement of (R / 2) x (R / 4) wave tiles (R / 64
// x R / 128 MFMA 32 x 32 tiles; at R = 256, 128 accumulators per lane), two
// waves per SIMD: while one waits on LDS or a barrier the other keeps the
// matrix core busy.  Loads into one stage stay in flight while the other is
// read.  Requires d % (2 * kBigK) == 0.
template <int R>
__device__ __forceinline__ void gram_big_tile(const uint16_t* __restrict__ F, int n, int d,
                                              const float* __restrict__ inv_norm, float* __restrict__ out,
                                              unsigned int* mf_bits, int row0, int col0, uint4* st0, uint4* st1) {
  constexpr int MT = R / 64, NT = R / 128;
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave >> 2, wn = wave & 3;

  f32x16 acc[MT][NT];
#pragma unroll
  for (int a = 0; a < MT; ++a)
#pragma unroll
    for (int b = 0; b < NT; ++b)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[a][b][r] = 0.f;

  // Raw buffer over the whole feature matrix (bytes); 0x00020000 selects
  // plain 32-bit data for the descriptor's format field.
  const __amdgpu_buffer_rsrc_t rsrc =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(F), 0, n * d * 2, 0x00020000);
  const int lrow = lane >> 3, lc_even = (lane & 7) ^ (lane >> 4), lc_odd = lc_even ^ 4;
  const int ra = row0 + wave * (R / 8) + lrow, rb = col0 + wave * (R / 8) + lrow;
  const int voff_a0 = (ra * d + lc_even * 8) * 2, voff_a1 = ((ra + 8) * d + lc_odd * 8) * 2;
  const int voff_b0 = (rb * d + lc_even * 8) * 2, voff_b1 = ((rb + 8) * d + lc_odd * 8) * 2;
  const int row_step = 32 * d;    // 16 rows, in bytes
  // MFMA operand reads: lane l reads row l % 32 of each 32-row tile at logical
  // chunk 2 kk + l / 32; every tile starts at a multiple of 32 rows, so the
  // swizzle term depends on l only.
  int offa[4], offb[4];
#pragma unroll
  for (int kk = 0; kk < 4; ++kk) {
    offa[kk] = swz(wm * (R / 2) + (lane & 31), kk * 2 + (lane >> 5));
    offb[kk] = swz(wn * (R / 4) + (lane & 31), kk * 2 + (lane >> 5));
  }

  bf16x8 fa[2][MT], fb[2][NT];
  const int nslabs = d / kBigK;   // even, at least 2
  load_slab<R>(st0, rsrc, voff_a0, voff_a1, row_step, 0, wave);
  load_slab<R>(st0 + R * 8, rsrc, voff_b0, voff_b1, row_step, 0, wave);
  int s = 0;
  for (; s + 2 < nslabs; s += 2) {
    CP_BIG_SLAB(st0, st1, s + 1)
    CP_BIG_SLAB(st1, st0, s + 2)
  }
  CP_BIG_SLAB(st0, st1, s + 1)
  CP_BIG_SLAB(st1, st0, -1)
  store_df(acc, row0 + wm * (R / 2), col0 + wn * (R / 4), lane, n, inv_norm, out, mf_bits);
}
#undef CP_BIG_SLAB

// Blocks [0, nfull) take full 256 x 256 tiles (band order, XCD-aware); the
// tiles after them, which would fill only part of a last round of the
// device's compute units, are split into four 128 x 128 quarters, block
// nfull + 4 t + q taking quarter q (row half q / 2, column half q % 2) of
// tile nfull + t in band order.  A diagonal tile's lower-left quarter lies
// below the diagonal and is left out.
__global__ __launch_bounds__(512) void gram_bf16_big_kernel(const uint16_t* __restrict__ F, int n, int d,
                                                            const float* __restrict__ inv_norm,
                                                            float* __restrict__ out, unsigned int* mf_bits,
                                                            int nfull, int ntiles, int T) {
  // One LDS object per stage (A rows, then B rows), so the compiler can tell
  // which stage each in-flight load targets.
  __shared__ uint4 st0[2 * kBig * 8], st1[2 * kBig * 8];
  int ti, tj;
  const int b = blockIdx.x;
  if (b < nfull) {
    if (!big_tile(b, nfull, T, ti, tj)) return;
    gram_big_tile<kBig>(F, n, d, inv_norm, out, mf_bits, ti * kBig, tj * kBig, st0, st1);
    return;
  }
  const int lin = nfull + (b - nfull) / 4, q = (b - nfull) % 4;
  if (lin >= ntiles || !band_tile(lin, T, ti, tj)) return;
  if (ti == tj && q == 2) return;
  gram_big_tile<kBig / 2>(F, n, d, inv_norm, out, mf_bits, ti * kBig + (q >> 1) * (kBig / 2),
                          tj * kBig + (q & 1) * (kBig / 2), st0, st1);
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

  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
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
  store_df(acc, row0 + wm * 64, col0 + wn * 64, lane, n, inv_norm, out, mf_bits);
}

}  // namespace

hipError_t launch_gram(const FstParams& p, const FstScratch& s, hipStream_t stream) {
  if (p.bf16 && p.d % (2 * kBigK) == 0 && p.n >= 4096 && int64_t(p.n) * p.d < (int64_t(1) << 30)) {
    const int t = (p.n + kBig - 1) / kBig;
    const int tiles = t * (t + 1) / 2;
    int dev = 0, cus = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess) return e;
    // Whole rounds of full tiles (a multiple of 8 blocks, for the XCD
    // dealing), the rest as quarter tiles.
    const int nfull = cus > 0 ? tiles / cus * cus / 8 * 8 : tiles / 8 * 8;
    const int blocks = nfull + 4 * (tiles - nfull);
    gram_bf16_big_kernel<<<blocks, 512, 0, stream>>>(static_cast<const uint16_t*>(p.feats), p.n, p.d,
                                                       s.inv_norm, p.cost, s.mf_bits, nfull, tiles, t);
    return hipGetLastError();
  }
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
