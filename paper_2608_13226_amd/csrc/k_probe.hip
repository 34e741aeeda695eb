// The latency floor of one greedy step (Sec. 3.5) on this device.
//
// A step of the rows schedule (k_sgs_inc.hip) cannot avoid two dependent
// operations: the exchange that makes every block agree on the winner (each
// block publishes its best candidate in its own slot and reads every block's
// slot), and the read of the winner's 64 KB row of the source-major cost,
// which every block needs before it knows which targets the pick improves.
// This kernel runs exactly those two, round after round, with the greedy's
// launch shape (one block of eight waves per compute unit) and its own slot
// layout, waits and loads, and nothing else: a round publishes a key that
// depends on the previous round's row, takes the exchange's winner, and reads
// the row the winner names.  Its time per round is therefore a floor for a
// step of the greedy; with `read_rows` = 0 only the exchange runs.
#include <hip/hip_runtime.h>

#include "sgs_exchange.h"

namespace cp {
namespace {

constexpr int kProbeChunk = 256;   // floats a wave loads per instruction (16 bytes a lane)

struct ProbeDev {
  const float* rows;          // [n_rows][ldt]
  int n_rows, ldt, rounds;
  unsigned long long* cand;   // exchange slots, as in the greedy
  unsigned int* abort;
  unsigned int poll_limit;
};

template <int RL, bool kRead>
__global__ __launch_bounds__(kBlock) void step_floor_kernel(ProbeDev a) {
  const int blk = blockIdx.x, nb = gridDim.x;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  __shared__ unsigned long long su[kWaves];
  __shared__ unsigned int sx[kWaves];
  __shared__ int sflag;
  const int nch = a.ldt / kProbeChunk;
  unsigned int x = unsigned(blk) * 2654435761u + 1u;
  for (int r = 0; r < a.rounds; ++r) {
    if (tid == 0) {
      const unsigned long long key = ((unsigned long long)(x & 0x3fffffffu) << kIndexBits) |
                                     (kIndexMask - (unsigned long long)blk);
      put(cand_slot(a.cand, r & 1, blk), key | epoch_of(r));
    }
    const int tw = read_winner(cand_slot(a.cand, r & 1, 0), epoch_of(r), nb, a.abort, a.poll_limit, su, &sflag);
    if (tw < 0) break;
    if (kRead) {
      // The winner's row, every chunk of the wave in flight together, folded
      // into the next key so that the next publish waits for the data.
      const f32x4* row = reinterpret_cast<const f32x4*>(a.rows + size_t((tw + r) % a.n_rows) * a.ldt);
      f32x4 v[RL];
#pragma unroll
      for (int i = 0; i < RL; ++i)
        if (w + i * kWaves < nch) v[i] = row[(w + i * kWaves) * (kProbeChunk / 4) + lane];
      unsigned int m = 0;
#pragma unroll
      for (int i = 0; i < RL; ++i)
        if (w + i * kWaves < nch)
          m ^= __float_as_uint(v[i][0]) ^ __float_as_uint(v[i][1]) ^ __float_as_uint(v[i][2]) ^
               __float_as_uint(v[i][3]);
#pragma unroll
      for (int o = 32; o > 0; o >>= 1) m ^= unsigned(__shfl_xor(int(m), o));
      if (lane == 0) sx[w] = m;
      __syncthreads();
#pragma unroll
      for (int q = 0; q < kWaves; ++q) m ^= sx[q];
      x = x * 1664525u + m;
    } else {
      x = x * 1664525u + 1013904223u + unsigned(tw);
    }
  }
}

__global__ void step_floor_init_kernel(unsigned long long* cand, unsigned int* abort, unsigned int preset) {
  for (int s = blockIdx.x * blockDim.x + threadIdx.x; s < 2 * kMaxBlocks * kSlotStride; s += gridDim.x * blockDim.x)
    cand[s] = 0ull;
  if (blockIdx.x == 0 && threadIdx.x == 0) *abort = preset;
}

constexpr size_t kProbeSlotBytes = size_t(2) * kMaxBlocks * kSlotStride * 8;

}  // namespace

size_t step_floor_workspace_bytes() { return kProbeSlotBytes + 256; }

hipError_t launch_step_floor(const float* rows, int n_rows, int row_len, int rounds, bool read_rows, void* workspace,
                             hipStream_t stream) {
  int dev = 0, cus = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if ((e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev)) != hipSuccess) return e;
  // The greedy's grid for a scene of n_rows tokens.
  const int nb = blocks_for(n_rows, cus);
  ProbeDev a{};
  a.rows = rows;
  a.n_rows = n_rows;
  a.ldt = row_len;
  a.rounds = rounds;
  a.cand = static_cast<unsigned long long*>(workspace);
  a.abort = reinterpret_cast<unsigned int*>(static_cast<char*>(workspace) + kProbeSlotBytes);
  const WaitPolicy wp = wait_policy();
  a.poll_limit = wp.limit;
  step_floor_init_kernel<<<64, 256, 0, stream>>>(a.cand, a.abort, wp.preset);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  const int nch = row_len / kProbeChunk;
  const void* kernel;
  if (!read_rows)
    kernel = reinterpret_cast<const void*>(step_floor_kernel<1, false>);
  else if (nch <= 8 * kWaves)
    kernel = reinterpret_cast<const void*>(step_floor_kernel<8, true>);
  else
    kernel = reinterpret_cast<const void*>(step_floor_kernel<16, true>);
  void* args[] = {&a};
  return hipLaunchCooperativeKernel(kernel, dim3(nb), dim3(kBlock), args, 0, stream);
}

}  // namespace cp
