// C-ABI entry points of the CoverPrune library: host-side argument checks,
// workspace carving and kernel dispatch.  Nothing here touches device data.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <mutex>
#include <string>

#include "../../include/coverprune.h"
#include "launch.h"

namespace {

thread_local std::string g_last_error;

cp_status fail(cp_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return st;
}

cp_status ok() {
  g_last_error.clear();
  return CP_OK;
}

cp_status hip_fail(hipError_t e, const char* where) {
  return fail(CP_ERR_HIP, "%s: %s", where, hipGetErrorString(e));
}

constexpr int64_t kMaxDenseN = int64_t(1) << 18;   // cost matrix of 256 GiB
constexpr int64_t kMaxLiteN = int64_t(1) << 24;
constexpr int64_t kMaxD = int64_t(1) << 16;
constexpr size_t kAlign = 256;

size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

cp_status check_features(const void* feats, cp_dtype dtype, int64_t n, int64_t d, int64_t max_n) {
  if (n < 1 || n > max_n) return fail(CP_ERR_INVALID_ARG, "n = %lld outside [1, %lld]", (long long)n, (long long)max_n);
  if (d < 1 || d > kMaxD) return fail(CP_ERR_INVALID_ARG, "d = %lld outside [1, %lld]", (long long)d, (long long)kMaxD);
  if (dtype != CP_F32 && dtype != CP_BF16) return fail(CP_ERR_UNSUPPORTED, "unknown feature dtype %d", (int)dtype);
  if (dtype == CP_BF16 && d % 8 != 0) return fail(CP_ERR_UNSUPPORTED, "bf16 features need d %% 8 == 0 (d = %lld)", (long long)d);
  if (dtype == CP_F32 && d % 4 != 0) return fail(CP_ERR_UNSUPPORTED, "f32 features need d %% 4 == 0 (d = %lld)", (long long)d);
  if (!feats) return fail(CP_ERR_INVALID_ARG, "feats is NULL");
  if (!aligned16(feats)) return fail(CP_ERR_INVALID_ARG, "feats is not 16-byte aligned");
  return CP_OK;
}

cp_status check_weights(const cp_fst_weights& w) {
  const float v[4] = {w.lambda_f, w.lambda_x, w.lambda_tau, w.kappa};
  for (float x : v)
    if (!std::isfinite(x) || x < 0.f) return fail(CP_ERR_INVALID_ARG, "weights and kappa must be finite and >= 0");
  return CP_OK;
}

cp_status check_workspace(void* ws, size_t have, size_t need) {
  if (need == 0) return CP_OK;
  if (!ws) return fail(CP_ERR_WORKSPACE, "workspace is NULL (%zu bytes needed)", need);
  if (!aligned16(ws)) return fail(CP_ERR_WORKSPACE, "workspace is not 16-byte aligned");
  if (have < need) return fail(CP_ERR_WORKSPACE, "workspace has %zu bytes, %zu needed", have, need);
  return CP_OK;
}

float inv_log1p(float kappa) { return kappa > 0.f ? float(1.0 / std::log1p(double(kappa))) : 0.f; }

}  // namespace

extern "C" {

const char* coverprune_status_string(cp_status s) {
  switch (s) {
    case CP_OK: return "ok";
    case CP_ERR_INVALID_ARG: return "invalid argument";
    case CP_ERR_UNSUPPORTED: return "unsupported";
    case CP_ERR_WORKSPACE: return "workspace too small";
    case CP_ERR_HIP: return "HIP runtime error";
  }
  return "unknown status";
}

const char* coverprune_last_error(void) { return g_last_error.c_str(); }

int coverprune_abi_version(void) { return 2; }

float coverprune_uncovered_cost(cp_fst_weights w) { return (w.lambda_f + w.lambda_x) + w.lambda_tau; }

// ---------------------------------------------------------------------------
size_t coverprune_fst_cost_workspace(int64_t n, int64_t d, cp_dtype dtype) {
  (void)d;
  (void)dtype;
  if (n < 1) return 0;
  return align_up(size_t(n) * sizeof(float)) + kAlign;
}

cp_status coverprune_fst_cost(const void* feats, cp_dtype dtype, int64_t n, int64_t d,
                              const float* pos, const int32_t* frame, cp_fst_weights w,
                              float* cost, float* maxima, void* workspace,
                              size_t workspace_bytes, void* stream) {
  cp_status st = check_features(feats, dtype, n, d, kMaxDenseN);
  if (st != CP_OK) return st;
  if (!pos || !frame || !cost) return fail(CP_ERR_INVALID_ARG, "pos, frame and cost must be non-NULL");
  if (!aligned16(cost)) return fail(CP_ERR_INVALID_ARG, "cost is not 16-byte aligned");
  if ((st = check_weights(w)) != CP_OK) return st;
  const size_t need = coverprune_fst_cost_workspace(n, d, dtype);
  if ((st = check_workspace(workspace, workspace_bytes, need)) != CP_OK) return st;

  char* base = static_cast<char*>(workspace);
  cp::FstScratch s;
  s.inv_norm = reinterpret_cast<float*>(base);
  char* tail = base + align_up(size_t(n) * sizeof(float));
  s.mf_bits = reinterpret_cast<unsigned int*>(tail);
  s.tau_min = reinterpret_cast<int*>(tail + 4);
  s.tau_max = reinterpret_cast<int*>(tail + 8);
  s.mx2_bits = reinterpret_cast<unsigned long long*>(tail + 16);

  cp::FstParams p;
  p.feats = feats;
  p.bf16 = dtype == CP_BF16;
  p.n = int(n);
  p.d = int(d);
  p.pos = pos;
  p.frame = frame;
  p.lambda_f = w.lambda_f;
  p.lambda_x = w.lambda_x;
  p.lambda_tau = w.lambda_tau;
  p.kappa = w.kappa;
  p.inv_log1p_kappa = inv_log1p(w.kappa);
  p.cost = cost;
  p.maxima = maxima;

  hipStream_t s_ = static_cast<hipStream_t>(stream);
  hipError_t e;
  if ((e = cp::launch_fst_prep(p, s, s_)) != hipSuccess) return hip_fail(e, "fst prep");
  if ((e = cp::launch_gram(p, s, s_)) != hipSuccess) return hip_fail(e, "gram");
  if ((e = cp::launch_fst_epilogue(p, s, s_)) != hipSuccess) return hip_fail(e, "fst epilogue");
  return ok();
}

// ---------------------------------------------------------------------------
size_t coverprune_sgs_workspace(int64_t n, int64_t k, uint32_t flags) {
  if (n < 1 || k < 1) return 0;
  if (flags == CP_SGS_INCREMENTAL) return cp::sgs_inc_workspace_bytes(n, k, false);
  if (flags == (CP_SGS_INCREMENTAL | CP_SGS_COMPACT)) return cp::sgs_inc_workspace_bytes(n, k, true);
  if (flags == CP_SGS_DENSE) return cp::sgs_workspace_bytes(n, k);
  return 0;
}

cp_status coverprune_sgs_select(const float* cost, int64_t n, const float* capacity, int64_t k,
                                float c0, uint32_t flags, int32_t* selected, double* step_gain,
                                double* step_objective, int32_t* assign, void* workspace,
                                size_t workspace_bytes, void* stream) {
  if (n < 1 || n > kMaxDenseN) return fail(CP_ERR_INVALID_ARG, "n = %lld outside [1, %lld]", (long long)n, (long long)kMaxDenseN);
  if (k < 1 || k > n) return fail(CP_ERR_INVALID_ARG, "k = %lld outside [1, n = %lld]", (long long)k, (long long)n);
  if (!std::isfinite(c0)) return fail(CP_ERR_INVALID_ARG, "c0 must be finite");
  if (flags != CP_SGS_DENSE && flags != CP_SGS_INCREMENTAL && flags != (CP_SGS_INCREMENTAL | CP_SGS_COMPACT))
    return fail(CP_ERR_UNSUPPORTED, "unknown flags 0x%x", flags);
  if (!cost || !capacity || !selected) return fail(CP_ERR_INVALID_ARG, "cost, capacity and selected must be non-NULL");
  if (!aligned16(cost)) return fail(CP_ERR_INVALID_ARG, "cost is not 16-byte aligned");
  cp_status st = check_workspace(workspace, workspace_bytes, coverprune_sgs_workspace(n, k, flags));
  if (st != CP_OK) return st;

  cp::SgsParams p;
  p.cost = cost;
  p.n = int(n);
  p.capacity = capacity;
  p.k = int(k);
  p.c0 = c0;
  p.selected = selected;
  p.step_gain = step_gain;
  p.step_objective = step_objective;
  p.assign = assign;
  p.workspace = workspace;
  p.workspace_bytes = workspace_bytes;
  hipError_t e = flags == CP_SGS_DENSE
                     ? cp::launch_sgs_dense(p, static_cast<hipStream_t>(stream))
                     : cp::launch_sgs_incremental(p, (flags & CP_SGS_COMPACT) != 0, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "sgs");
  return ok();
}

// ---------------------------------------------------------------------------
// The greedy's part of the prune workspace: the fused form's (the rows
// schedule and the epilogue's partial gains) for n a multiple of 64, the
// incremental form's otherwise.
static size_t prune_sgs_bytes(int64_t n, int64_t k) {
  return n % 64 == 0 ? cp::sgs_fused_workspace_bytes(n, k) : cp::sgs_inc_workspace_bytes(n, k, false);
}

size_t coverprune_prune_workspace(int64_t n, int64_t d, int64_t k, cp_dtype dtype) {
  if (n < 1 || k < 1 || k > n) return 0;
  return align_up(coverprune_fst_cost_workspace(n, d, dtype)) + prune_sgs_bytes(n, k);
}

cp_status coverprune_prune(const void* feats, cp_dtype dtype, int64_t n, int64_t d, const float* pos,
                           const int32_t* frame, cp_fst_weights w, const float* capacity, int64_t k, float c0,
                           float* cost, float* maxima, int32_t* selected, double* step_gain,
                           double* step_objective, int32_t* assign, void* workspace, size_t workspace_bytes,
                           void* stream) {
  cp_status st = check_features(feats, dtype, n, d, kMaxDenseN);
  if (st != CP_OK) return st;
  if (k < 1 || k > n) return fail(CP_ERR_INVALID_ARG, "k = %lld outside [1, n = %lld]", (long long)k, (long long)n);
  if (!std::isfinite(c0)) return fail(CP_ERR_INVALID_ARG, "c0 must be finite");
  if (!pos || !frame || !cost || !capacity || !selected)
    return fail(CP_ERR_INVALID_ARG, "pos, frame, cost, capacity and selected must be non-NULL");
  if (!aligned16(cost)) return fail(CP_ERR_INVALID_ARG, "cost is not 16-byte aligned");
  if ((st = check_weights(w)) != CP_OK) return st;
  if ((st = check_workspace(workspace, workspace_bytes, coverprune_prune_workspace(n, d, k, dtype))) != CP_OK)
    return st;

  const size_t fst_bytes = align_up(coverprune_fst_cost_workspace(n, d, dtype));
  char* base = static_cast<char*>(workspace);
  cp::FstScratch s;
  s.inv_norm = reinterpret_cast<float*>(base);
  char* tail = base + align_up(size_t(n) * sizeof(float));
  s.mf_bits = reinterpret_cast<unsigned int*>(tail);
  s.tau_min = reinterpret_cast<int*>(tail + 4);
  s.tau_max = reinterpret_cast<int*>(tail + 8);
  s.mx2_bits = reinterpret_cast<unsigned long long*>(tail + 16);

  cp::FstParams p;
  p.feats = feats;
  p.bf16 = dtype == CP_BF16;
  p.n = int(n);
  p.d = int(d);
  p.pos = pos;
  p.frame = frame;
  p.lambda_f = w.lambda_f;
  p.lambda_x = w.lambda_x;
  p.lambda_tau = w.lambda_tau;
  p.kappa = w.kappa;
  p.inv_log1p_kappa = inv_log1p(w.kappa);
  p.cost = cost;
  p.maxima = maxima;

  cp::SgsParams q;
  q.cost = cost;
  q.n = int(n);
  q.capacity = capacity;
  q.k = int(k);
  q.c0 = c0;
  q.selected = selected;
  q.step_gain = step_gain;
  q.step_objective = step_objective;
  q.assign = assign;
  q.workspace = base + fst_bytes;
  q.workspace_bytes = workspace_bytes - fst_bytes;

  hipStream_t s_ = static_cast<hipStream_t>(stream);
  hipError_t e;
  if ((e = cp::launch_fst_prep(p, s, s_)) != hipSuccess) return hip_fail(e, "fst prep");
  if ((e = cp::launch_gram(p, s, s_)) != hipSuccess) return hip_fail(e, "gram");
  if (!cp::sgs_fused_fits(n)) {
    // The two calls' kernels one after the other.
    if ((e = cp::launch_fst_epilogue(p, s, s_)) != hipSuccess) return hip_fail(e, "fst epilogue");
    if ((e = cp::launch_sgs_incremental(q, false, s_)) != hipSuccess) return hip_fail(e, "sgs");
    return ok();
  }
  cp::SgsFused f;
  if ((e = cp::sgs_fused_prepare(q, &f, s_)) != hipSuccess) return hip_fail(e, "sgs scale");
  cp::EpiSgs g;
  g.T = f.T;
  g.ldt = f.ldt;
  g.part = f.part;
  g.v = capacity;
  g.c0 = c0;
  g.scale = f.scale;
  if ((e = cp::launch_fst_epilogue_sgs(p, s, g, s_)) != hipSuccess) return hip_fail(e, "fst epilogue");
  if ((e = cp::launch_sgs_fused(q, f, s_)) != hipSuccess) return hip_fail(e, "sgs");
  return ok();
}

// ---------------------------------------------------------------------------
static bool batch_flags_ok(uint32_t flags) {
  return flags == CP_SGS_INCREMENTAL || flags == (CP_SGS_INCREMENTAL | CP_SGS_COMPACT);
}

size_t coverprune_sgs_batch_workspace(const cp_sgs_scene* scenes, int32_t count, uint32_t flags) {
  if (!scenes || count < 1 || count > CP_SGS_MAX_BATCH || !batch_flags_ok(flags)) return 0;
  int64_t n[CP_SGS_MAX_BATCH], k[CP_SGS_MAX_BATCH];
  for (int32_t s = 0; s < count; ++s) {
    if (scenes[s].n < 1 || scenes[s].k < 1) return 0;
    n[s] = scenes[s].n;
    k[s] = scenes[s].k;
  }
  return cp::sgs_inc_batch_workspace_bytes(n, k, int(count), (flags & CP_SGS_COMPACT) != 0);
}

cp_status coverprune_sgs_select_batch(const cp_sgs_scene* scenes, int32_t count, uint32_t flags,
                                      void* workspace, size_t workspace_bytes, void* stream) {
  if (!scenes) return fail(CP_ERR_INVALID_ARG, "scenes is NULL");
  if (!batch_flags_ok(flags)) return fail(CP_ERR_UNSUPPORTED, "unknown flags 0x%x", flags);
  if (count < 1 || count > CP_SGS_MAX_BATCH)
    return fail(CP_ERR_INVALID_ARG, "count = %d outside [1, %d]", (int)count, CP_SGS_MAX_BATCH);
  cp::SgsParams p[CP_SGS_MAX_BATCH];
  for (int32_t s = 0; s < count; ++s) {
    const cp_sgs_scene& c = scenes[s];
    if (c.n < 1 || c.n > kMaxDenseN)
      return fail(CP_ERR_INVALID_ARG, "scene %d: n = %lld outside [1, %lld]", (int)s, (long long)c.n, (long long)kMaxDenseN);
    if (c.k < 1 || c.k > c.n)
      return fail(CP_ERR_INVALID_ARG, "scene %d: k = %lld outside [1, n = %lld]", (int)s, (long long)c.k, (long long)c.n);
    if (!std::isfinite(c.c0)) return fail(CP_ERR_INVALID_ARG, "scene %d: c0 must be finite", (int)s);
    if (!c.cost || !c.capacity || !c.selected)
      return fail(CP_ERR_INVALID_ARG, "scene %d: cost, capacity and selected must be non-NULL", (int)s);
    if (!aligned16(c.cost)) return fail(CP_ERR_INVALID_ARG, "scene %d: cost is not 16-byte aligned", (int)s);
    p[s].cost = c.cost;
    p[s].n = int(c.n);
    p[s].capacity = c.capacity;
    p[s].k = int(c.k);
    p[s].c0 = c.c0;
    p[s].selected = c.selected;
    p[s].step_gain = c.step_gain;
    p[s].step_objective = c.step_objective;
    p[s].assign = c.assign;
    p[s].workspace = nullptr;
    p[s].workspace_bytes = 0;
  }
  cp_status st = check_workspace(workspace, workspace_bytes, coverprune_sgs_batch_workspace(scenes, count, flags));
  if (st != CP_OK) return st;
  hipError_t e = cp::launch_sgs_incremental_batch(p, int(count), (flags & CP_SGS_COMPACT) != 0, workspace,
                                                  static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "sgs batch");
  return ok();
}

// ---------------------------------------------------------------------------
// The greedy without a workspace argument, for callers that cannot allocate.
// Its scratch space is one file-scope device array: each GPU the library runs
// on holds its own copy until the process ends.  In host code the array's
// name is not a device address, so the address is looked up once per device
// (hipGetSymbolAddress, with that device current) and only that address is
// ever handed to kernels.

}  // extern "C"

namespace {

// The compact schedule's workspace at CP_SGS_NOALLOC_MAX_N tokens is about
// 1.35 MiB (change list, exchange slots, step-0 partial gains); the array is
// a little larger and every call checks the exact need against it.
constexpr size_t kNoallocBytes = size_t(3) << 19;   // 1.5 MiB
__device__ __align__(256) unsigned char scratch[kNoallocBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// The current device's copy of `scratch`, looked up on its first use.
cp_status scratch_of_current_device(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (dev < 0 || dev >= kMaxDevices)
    return fail(CP_ERR_UNSUPPORTED, "device %d outside the %d devices the scratch table covers", dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
    if (!p) return fail(CP_ERR_HIP, "hipGetSymbolAddress(scratch) returned NULL");
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return CP_OK;
}

}  // namespace

extern "C" {

cp_status coverprune_sgs_select_noalloc(const float* cost, int64_t n, const float* capacity, int64_t k, float c0,
                                        int32_t* selected, double* step_gain, double* step_objective,
                                        int32_t* assign, void* stream) {
  if (n < 1 || n > CP_SGS_NOALLOC_MAX_N)
    return fail(CP_ERR_INVALID_ARG, "n = %lld outside [1, %d] (the no-allocation greedy's scratch limit)",
                (long long)n, CP_SGS_NOALLOC_MAX_N);
  if (k < 1 || k > n) return fail(CP_ERR_INVALID_ARG, "k = %lld outside [1, n = %lld]", (long long)k, (long long)n);
  if (!std::isfinite(c0)) return fail(CP_ERR_INVALID_ARG, "c0 must be finite");
  if (!cost || !capacity || !selected) return fail(CP_ERR_INVALID_ARG, "cost, capacity and selected must be non-NULL");
  if (!aligned16(cost)) return fail(CP_ERR_INVALID_ARG, "cost is not 16-byte aligned");
  const size_t need = cp::sgs_inc_workspace_bytes(n, k, true);
  if (need > kNoallocBytes)
    return fail(CP_ERR_UNSUPPORTED, "scene needs %zu bytes of scratch, %zu available", need, kNoallocBytes);
  void* ws = nullptr;
  cp_status st = scratch_of_current_device(&ws);
  if (st != CP_OK) return st;

  cp::SgsParams p;
  p.cost = cost;
  p.n = int(n);
  p.capacity = capacity;
  p.k = int(k);
  p.c0 = c0;
  p.selected = selected;
  p.step_gain = step_gain;
  p.step_objective = step_objective;
  p.assign = assign;
  p.workspace = ws;
  p.workspace_bytes = kNoallocBytes;
  hipError_t e = cp::launch_sgs_incremental(p, true, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "sgs noalloc");
  return ok();
}

// ---------------------------------------------------------------------------
size_t coverprune_step_floor_workspace(void) { return cp::step_floor_workspace_bytes(); }

cp_status coverprune_step_floor(const float* rows, int64_t n_rows, int64_t row_len, int32_t rounds,
                                int32_t read_rows, void* workspace, size_t workspace_bytes, void* stream) {
  if (n_rows < 1 || n_rows > kMaxDenseN)
    return fail(CP_ERR_INVALID_ARG, "n_rows = %lld outside [1, %lld]", (long long)n_rows, (long long)kMaxDenseN);
  if (row_len < 256 || row_len > 32768 || row_len % 256 != 0)
    return fail(CP_ERR_INVALID_ARG, "row_len = %lld must be a multiple of 256 in [256, 32768]", (long long)row_len);
  if (rounds < 1) return fail(CP_ERR_INVALID_ARG, "rounds = %d must be >= 1", (int)rounds);
  if (!rows) return fail(CP_ERR_INVALID_ARG, "rows is NULL");
  if (!aligned16(rows)) return fail(CP_ERR_INVALID_ARG, "rows is not 16-byte aligned");
  cp_status st = check_workspace(workspace, workspace_bytes, coverprune_step_floor_workspace());
  if (st != CP_OK) return st;
  hipError_t e = cp::launch_step_floor(rows, int(n_rows), int(row_len), int(rounds), read_rows != 0, workspace,
                                       static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "step floor");
  return ok();
}

// ---------------------------------------------------------------------------
size_t coverprune_sgs_literal_workspace(int64_t n, int64_t k) {
  if (n < 1 || k < 1 || k > n) return 0;
  return cp::sgs_literal_workspace_bytes(n, k);
}

cp_status coverprune_sgs_literal_select(const float* cost, int64_t n, const float* capacity, int64_t k,
                                        float epsilon, int32_t rounds, const int32_t* follow, int32_t* selected,
                                        double* step_score, double* step_residual, double* objective,
                                        void* workspace, size_t workspace_bytes, void* stream) {
  if (n < 1 || n > kMaxDenseN) return fail(CP_ERR_INVALID_ARG, "n = %lld outside [1, %lld]", (long long)n, (long long)kMaxDenseN);
  if (k < 1 || k > std::min<int64_t>(n, CP_SGS_LITERAL_MAX_K))
    return fail(CP_ERR_INVALID_ARG, "k = %lld outside [1, min(n, %d)]", (long long)k, CP_SGS_LITERAL_MAX_K);
  if (!std::isfinite(epsilon) || !(epsilon > 0.f)) return fail(CP_ERR_INVALID_ARG, "epsilon must be finite and > 0");
  if (rounds < 1 || rounds > CP_SGS_LITERAL_MAX_ROUNDS)
    return fail(CP_ERR_INVALID_ARG, "rounds = %d outside [1, %d]", (int)rounds, CP_SGS_LITERAL_MAX_ROUNDS);
  if (!cost || !capacity || !selected) return fail(CP_ERR_INVALID_ARG, "cost, capacity and selected must be non-NULL");
  if (!aligned16(cost)) return fail(CP_ERR_INVALID_ARG, "cost is not 16-byte aligned");
  cp_status st = check_workspace(workspace, workspace_bytes, coverprune_sgs_literal_workspace(n, k));
  if (st != CP_OK) return st;

  cp::LiteralParams p;
  p.cost = cost;
  p.n = int(n);
  p.capacity = capacity;
  p.k = int(k);
  p.epsilon = epsilon;
  p.rounds = int(rounds);
  p.follow = follow;
  p.selected = selected;
  p.step_score = step_score;
  p.step_residual = step_residual;
  p.objective = objective;
  p.workspace = workspace;
  p.workspace_bytes = workspace_bytes;
  hipError_t e = cp::launch_sgs_literal(p, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "sgs literal");
  return ok();
}

// ---------------------------------------------------------------------------
cp_status coverprune_knn(const float* pos, int64_t n, int64_t g, int32_t* neighbours, void* stream) {
  if (n < 1 || n > CP_KNN_MAX_N) return fail(CP_ERR_INVALID_ARG, "n = %lld outside [1, %d]", (long long)n, CP_KNN_MAX_N);
  if (g < 1 || g > std::min<int64_t>(n, CP_KNN_MAX_G))
    return fail(CP_ERR_INVALID_ARG, "g = %lld outside [1, min(n, %d)]", (long long)g, CP_KNN_MAX_G);
  if (!pos || !neighbours) return fail(CP_ERR_INVALID_ARG, "pos and neighbours must be non-NULL");
  hipError_t e = cp::launch_knn(pos, int(n), int(g), neighbours, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "knn");
  return ok();
}

size_t coverprune_fst_capacity_workspace(int64_t n, int64_t n_nb) {
  if (n < 2 || n_nb < 1 || n_nb > n - 1) return 0;
  return cp::capacity_workspace_bytes(n, n_nb);
}

cp_status coverprune_fst_capacity(const void* feats, cp_dtype dtype, int64_t n, int64_t d, const float* pos,
                                  const int32_t* frame, int64_t n_nb, cp_capacity_weights alpha, float* capacity,
                                  double* score, void* workspace, size_t workspace_bytes, void* stream) {
  cp_status st = check_features(feats, dtype, n, d, CP_KNN_MAX_N);
  if (st != CP_OK) return st;
  if (n < 2) return fail(CP_ERR_INVALID_ARG, "n = %lld: the capacity needs at least 2 tokens", (long long)n);
  if (n_nb < 1 || n_nb > std::min<int64_t>(n - 1, CP_KNN_MAX_G - 1))
    return fail(CP_ERR_INVALID_ARG, "n_nb = %lld outside [1, min(n - 1, %d)]", (long long)n_nb, CP_KNN_MAX_G - 1);
  if (!pos || !frame || !capacity) return fail(CP_ERR_INVALID_ARG, "pos, frame and capacity must be non-NULL");
  const float a[3] = {alpha.alpha_f, alpha.alpha_x, alpha.alpha_tau};
  for (float x : a)
    if (!std::isfinite(x) || x < 0.f) return fail(CP_ERR_INVALID_ARG, "capacity weights must be finite and >= 0");
  if ((st = check_workspace(workspace, workspace_bytes, coverprune_fst_capacity_workspace(n, n_nb))) != CP_OK)
    return st;

  cp::CapacityParams p;
  p.feats = feats;
  p.bf16 = dtype == CP_BF16;
  p.n = int(n);
  p.d = int(d);
  p.pos = pos;
  p.frame = frame;
  p.nn = int(n_nb);
  p.alpha_f = alpha.alpha_f;
  p.alpha_x = alpha.alpha_x;
  p.alpha_tau = alpha.alpha_tau;
  p.capacity = capacity;
  p.score = score;
  p.workspace = workspace;
  p.workspace_bytes = workspace_bytes;
  hipError_t e = cp::launch_capacity(p, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "capacity");
  return ok();
}

size_t coverprune_sgs_local_workspace(int64_t n, int64_t k) {
  if (n < 1 || k < 1) return 0;
  return cp::sgs_local_workspace_bytes(n, k);
}

cp_status coverprune_sgs_local_select(const float* cost, int64_t n, const float* capacity,
                                      const int32_t* neighbours, int64_t g, int64_t k, float c0,
                                      int32_t* selected, double* step_gain, double* step_objective,
                                      int32_t* assign, void* workspace, size_t workspace_bytes,
                                      void* stream) {
  if (n < 1 || n > CP_SGS_LOCAL_MAX_N)
    return fail(CP_ERR_INVALID_ARG, "n = %lld outside [1, %d]", (long long)n, CP_SGS_LOCAL_MAX_N);
  if (g < 1 || g > std::min<int64_t>(n, CP_SGS_LOCAL_MAX_G))
    return fail(CP_ERR_INVALID_ARG, "g = %lld outside [1, min(n, %d)]", (long long)g, CP_SGS_LOCAL_MAX_G);
  if (k < 1 || k > n) return fail(CP_ERR_INVALID_ARG, "k = %lld outside [1, n = %lld]", (long long)k, (long long)n);
  if (!std::isfinite(c0)) return fail(CP_ERR_INVALID_ARG, "c0 must be finite");
  if (!cost || !capacity || !neighbours || !selected)
    return fail(CP_ERR_INVALID_ARG, "cost, capacity, neighbours and selected must be non-NULL");
  if (!aligned16(cost)) return fail(CP_ERR_INVALID_ARG, "cost is not 16-byte aligned");
  cp_status st = check_workspace(workspace, workspace_bytes, coverprune_sgs_local_workspace(n, k));
  if (st != CP_OK) return st;

  cp::SgsParams p;
  p.cost = cost;
  p.n = int(n);
  p.capacity = capacity;
  p.k = int(k);
  p.c0 = c0;
  p.selected = selected;
  p.step_gain = step_gain;
  p.step_objective = step_objective;
  p.assign = assign;
  p.workspace = workspace;
  p.workspace_bytes = workspace_bytes;
  hipError_t e = cp::launch_sgs_local(p, neighbours, int(g), static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "sgs local");
  return ok();
}

// ---------------------------------------------------------------------------
size_t coverprune_lite_workspace(int64_t n, int64_t d, int64_t k, cp_dtype dtype) {
  (void)d;
  (void)dtype;
  if (n < 1 || k < 1) return 0;
  return cp::lite_workspace_bytes(n, k);
}

cp_status coverprune_lite_select(const void* feats, cp_dtype dtype, int64_t n, int64_t d,
                                 const float* pos, const int32_t* frame, const float* capacity,
                                 int64_t k, cp_fst_weights w, float voxel_size, int32_t* selected,
                                 int32_t* group, double* objective, double* token_cost, void* workspace,
                                 size_t workspace_bytes, void* stream) {
  cp_status st = check_features(feats, dtype, n, d, kMaxLiteN);
  if (st != CP_OK) return st;
  if (k < 1 || k > n) return fail(CP_ERR_INVALID_ARG, "k = %lld outside [1, n = %lld]", (long long)k, (long long)n);
  if (k >= (int64_t(1) << 23)) return fail(CP_ERR_INVALID_ARG, "k = %lld must be below 2^23", (long long)k);
  if (!pos || !frame || !capacity || !selected) return fail(CP_ERR_INVALID_ARG, "pos, frame, capacity and selected must be non-NULL");
  if ((st = check_weights(w)) != CP_OK) return st;
  if (!std::isfinite(voxel_size) || !(voxel_size > 0.f)) return fail(CP_ERR_INVALID_ARG, "voxel_size must be finite and > 0");
  if ((st = check_workspace(workspace, workspace_bytes, coverprune_lite_workspace(n, d, k, dtype))) != CP_OK) return st;

  cp::LiteParams p;
  p.feats = feats;
  p.bf16 = dtype == CP_BF16;
  p.n = int(n);
  p.d = int(d);
  p.pos = pos;
  p.frame = frame;
  p.capacity = capacity;
  p.k = int(k);
  p.lambda_f = w.lambda_f;
  p.lambda_x = w.lambda_x;
  p.lambda_tau = w.lambda_tau;
  p.kappa = w.kappa;
  p.inv_log1p_kappa = w.kappa > 0.f ? 1.0 / std::log1p(double(w.kappa)) : 0.0;
  p.grid_scale = 256.0 / double(voxel_size);
  p.selected = selected;
  p.group = group;
  p.objective = objective;
  p.token_cost = token_cost;
  p.workspace = workspace;
  p.workspace_bytes = workspace_bytes;
  hipError_t e = cp::launch_lite(p, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "lite");
  return ok();
}

}  // extern "C"
