// Host-side launchers: the only interface between the C-ABI layer (api.hip)
// and the kernel translation units.  Every launcher enqueues on `stream`,
// never synchronises, and returns the HIP status of its launches.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace cp {

// Workspace of coverprune_fst_cost.
struct FstScratch {
  float* inv_norm;                // [n] 1 / |f_i| (0 for a zero row)
  unsigned int* mf_bits;          // max d_f as float bits
  unsigned long long* mx2_bits;   // max squared distance as double bits
  int* tau_min;                   // min frame index
  int* tau_max;                   // max frame index
};

struct FstParams {
  const void* feats;
  bool bf16;
  int n;
  int d;
  const float* pos;
  const int32_t* frame;
  float lambda_f, lambda_x, lambda_tau, kappa;
  float inv_log1p_kappa;          // 1 / log1p(kappa), unused when kappa == 0
  float* cost;                    // [n, n] target-major
  float* maxima;                  // [3] or nullptr
};

hipError_t launch_fst_prep(const FstParams& p, const FstScratch& s, hipStream_t stream);
hipError_t launch_gram(const FstParams& p, const FstScratch& s, hipStream_t stream);
hipError_t launch_fst_epilogue(const FstParams& p, const FstScratch& s, hipStream_t stream);

// The epilogue of coverprune_prune (n a multiple of 64): the cost, and for
// the incremental greedy that follows, its source-major copy T and the
// step-0 gains as partial sums over 64-target blocks.
struct EpiSgs {
  float* T;                       // [n][ldt] T[s][t] = C(s, t)
  int ldt;
  long long* part;                // [n / 64][n] fixed-point partial gains
  const float* v;                 // [n] capacities
  float c0;
  const int* scale;               // the greedy's fixed-point exponent, set before the launch
};
hipError_t launch_fst_epilogue_sgs(const FstParams& p, const FstScratch& s, const EpiSgs& g, hipStream_t stream);

// Greedy selection.
struct SgsParams {
  const float* cost;              // [n, n] target-major
  int n;
  const float* capacity;          // [n]
  int k;
  float c0;
  int32_t* selected;              // [k]
  double* step_gain;              // [k] or nullptr
  double* step_objective;         // [k] or nullptr
  int32_t* assign;                // [n] or nullptr
  void* workspace;
  size_t workspace_bytes;
};

size_t sgs_workspace_bytes(int64_t n, int64_t k);
hipError_t launch_sgs_dense(const SgsParams& p, hipStream_t stream);
// Incremental form: the rows schedule (workspace about 4 n bytes per token)
// unless `compact` or the scene is too large for it, else the exchange
// schedule (about 16 bytes per token).
size_t sgs_inc_workspace_bytes(int64_t n, int64_t k, bool compact);
hipError_t launch_sgs_incremental(const SgsParams& p, bool compact, hipStream_t stream);
// The incremental greedy after launch_fst_epilogue_sgs (coverprune_prune):
// the rows schedule, whose T and step-0 partial gains that epilogue writes.
// sgs_fused_fits: n a multiple of 64 that the rows schedule serves on this
// device.  sgs_fused_prepare points f into p.workspace (sized by
// sgs_fused_workspace_bytes) and enqueues the scale the epilogue needs;
// launch_sgs_fused runs the greedy itself.
struct SgsFused {
  float* T;
  int ldt;
  long long* part;
  int P;
  int* scale;
};
bool sgs_fused_fits(int64_t n);
size_t sgs_fused_workspace_bytes(int64_t n, int64_t k);
hipError_t sgs_fused_prepare(const SgsParams& p, SgsFused* f, hipStream_t stream);
hipError_t launch_sgs_fused(const SgsParams& p, const SgsFused& f, hipStream_t stream);
// Up to 16 scenes in one cooperative launch (incremental form); the scenes'
// workspaces lie one after another in `workspace` (each p[s].workspace is
// ignored).
size_t sgs_inc_batch_workspace_bytes(const int64_t* n, const int64_t* k, int count, bool compact);
hipError_t launch_sgs_incremental_batch(const SgsParams* p, int count, bool compact, void* workspace,
                                        hipStream_t stream);
// Local form: gains over the neighbour table nbr [n, g] (g <= 128, n <= 16384).
size_t sgs_local_workspace_bytes(int64_t n, int64_t k);
hipError_t launch_sgs_local(const SgsParams& p, const int32_t* nbr, int g, hipStream_t stream);

// Latency floor of a greedy step: rounds of the candidate exchange, each
// followed (read_rows) by the read of a row of `rows` [n_rows][row_len] that
// the exchange's winner names.  row_len is a multiple of 256, at most 32768.
size_t step_floor_workspace_bytes();
hipError_t launch_step_floor(const float* rows, int n_rows, int row_len, int rounds, bool read_rows, void* workspace,
                             hipStream_t stream);

// Nearest-neighbour tables: out [n, g], n <= 32768, g <= min(n, 1024).
hipError_t launch_knn(const float* pos, int n, int g, int32_t* out, hipStream_t stream);

// The greedy step solved as written: entropic semi-relaxed transport per step.
struct LiteralParams {
  const float* cost;              // [n, n] target-major
  int n;
  const float* capacity;          // [n]
  int k;                          // 1 <= k <= min(n, 4096)
  float epsilon;
  int rounds;
  const int32_t* follow;          // [k] or nullptr
  int32_t* selected;              // [k]
  double* step_score;             // [k] or nullptr
  double* step_residual;          // [k] or nullptr
  double* objective;              // [1] or nullptr
  void* workspace;
  size_t workspace_bytes;
};

size_t sgs_literal_workspace_bytes(int64_t n, int64_t k);
hipError_t launch_sgs_literal(const LiteralParams& p, hipStream_t stream);

// FST capacity.
struct CapacityParams {
  const void* feats;
  bool bf16;
  int n;
  int d;
  const float* pos;
  const int32_t* frame;
  int nn;                         // neighbours per token, 1 <= nn <= n - 1
  float alpha_f, alpha_x, alpha_tau;
  float* capacity;                // [n]
  double* score;                  // [n] or nullptr
  void* workspace;
  size_t workspace_bytes;
};

size_t capacity_workspace_bytes(int64_t n, int64_t nn);
hipError_t launch_capacity(const CapacityParams& p, hipStream_t stream);

// CoverPrune-Lite.
struct LiteParams {
  const void* feats;
  bool bf16;
  int n;
  int d;
  const float* pos;
  const int32_t* frame;
  const float* capacity;
  int k;
  float lambda_f, lambda_x, lambda_tau, kappa;
  double inv_log1p_kappa;
  double grid_scale;              // 256 / voxel_size, float64
  int32_t* selected;              // [k]
  int32_t* group;                 // [n] or nullptr
  double* objective;              // [1] or nullptr
  double* token_cost;             // [n] or nullptr
  void* workspace;
  size_t workspace_bytes;
};

size_t lite_workspace_bytes(int64_t n, int64_t k);
hipError_t launch_lite(const LiteParams& p, hipStream_t stream);

}  // namespace cp
