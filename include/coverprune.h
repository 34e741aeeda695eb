/*
 * coverprune.h -- C-ABI of the CoverPrune hot path for AMD Instinct MI355X (gfx950).
 *
 * CoverPrune (arXiv 2608.13226) prunes the N visual tokens of a video to K
 * tokens that best cover the scene in an optimal-transport sense.  This
 * library computes, on one GPU:
 *
 *   coverprune_fst_cost    the Feature-Spatial-Temporal transport cost between
 *                          every pair of tokens (Sec. 3.3, Eq. 7-8);
 *   coverprune_fst_capacity the target capacities v from each token's 3D
 *                          neighbours (Sec. 3.4, Eq. 9-10);
 *   coverprune_sgs_select  greedy selection of K tokens against that cost and
 *                          the target capacities (Sec. 3.5, Eq. 11-16);
 *   coverprune_sgs_select_batch  up to 16 scenes' greedies in one launch;
 *   coverprune_knn         the g nearest tokens of every token in 3D, and
 *   coverprune_sgs_local_select  the greedy with gains over those neighbours
 *                          only (Sec. 3.5, Eq. 13);
 *   coverprune_sgs_literal_select  the greedy with each step's transport
 *                          solved as written (Sec. 3.5, Eq. 11-15);
 *   coverprune_lite_select CoverPrune-Lite: Morton ordering, capacity-guided
 *                          grouping and per-group prototypes (Sec. 4, Eq. 17-20).
 *
 * Conventions shared by every entry point
 *   - Token j has a feature row f_j (D values), a 3D position x_j (metres) and
 *     the integer index tau_j of the frame it came from (problem setup, Sec. 3.2).
 *   - Every array argument is DEVICE memory owned by the caller, row-major and
 *     densely packed.  The library keeps no pointer after a call returns and
 *     allocates no memory: scratch space is the caller's workspace, sized by
 *     the matching *_workspace() query.  Workspace and array pointers must be
 *     16-byte aligned.
 *   - Calls are asynchronous: work is enqueued on `stream` (a hipStream_t; NULL
 *     is the default stream) and results are valid once the stream has
 *     completed it.  No call synchronises the host with the device.
 *   - Arguments are validated on the host before anything is enqueued; a
 *     failed check returns an error status and enqueues nothing.  Data values
 *     are not checked (finite inputs, capacities >= 0 with a positive sum are
 *     the caller's duty).  coverprune_last_error() describes the last failure
 *     of the calling thread.
 *   - Results are bitwise reproducible run to run on the same GPU.  Calls on
 *     distinct workspaces and streams may run concurrently.
 *   - Waits between the blocks of one launch are bounded.  The greedy
 *     selection calls (sgs_select, sgs_select_batch, sgs_local_select, and the
 *     greedy of prune) run persistent launches whose blocks wait for each
 *     other (lite_select has no such waits: ordinary launches only).  A wait
 *     that has polled for about a second (far beyond any legitimate wait: a launch
 *     starved of compute units, or a broken device) gives up, every block of
 *     the launch leaves, and every entry of `selected` is set to -1, which is
 *     never a token index.  The call itself has already returned CP_OK (the
 *     host is not synchronised), so a caller that must detect this checks
 *     selected[0] >= 0 once the stream has completed; the other outputs of
 *     that call are then undefined.  COVERPRUNE_TEST_ABORT=1 in the
 *     environment makes every such launch give up at its first unmet wait
 *     (a test of this path; every kernel still ends normally).
 */
#ifndef COVERPRUNE_H
#define COVERPRUNE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  CP_OK = 0,
  CP_ERR_INVALID_ARG = 1, /* a scalar out of range or a required pointer is NULL */
  CP_ERR_UNSUPPORTED = 2, /* a dtype, feature width or flag this build does not handle */
  CP_ERR_WORKSPACE = 3,   /* workspace missing or smaller than the query returned */
  CP_ERR_HIP = 4          /* the HIP runtime reported an error while enqueuing */
} cp_status;

typedef enum { CP_F32 = 0, CP_BF16 = 1 } cp_dtype;

/* Weights of Eq. 8.  lambda_* >= 0 weight the feature, spatial and temporal
 * terms; kappa >= 0 shapes phi_kappa(z) = log(1 + kappa z) / log(1 + kappa),
 * with kappa = 0 taken as the kappa -> 0 limit phi(z) = z.  The paper's
 * experiments use lambda = 1 (Sec. 5.1) and give no kappa. */
typedef struct {
  float lambda_f;
  float lambda_x;
  float lambda_tau;
  float kappa;
} cp_fst_weights;

/* SGS flags (the same greedy either way; see coverprune_sgs_select). */
#define CP_SGS_DENSE 0u       /* every step re-evaluates every candidate's gain over the whole cost matrix */
#define CP_SGS_INCREMENTAL 1u /* gains computed once, then updated from the rows whose best cost drops */
#define CP_SGS_COMPACT 2u     /* with CP_SGS_INCREMENTAL: the schedule with the small workspace */

/* The cost of leaving a target uncovered, c0 of the greedy (Sec. 3.5): the
 * largest value the cost of Eq. 8 can take, (lambda_f + lambda_x) +
 * lambda_tau in float arithmetic.  The selection calls take c0 as an argument;
 * this is the value to pass for a cost made with weights w.  Pure host
 * arithmetic, no device work. */
float coverprune_uncovered_cost(cp_fst_weights w);

/* ------------------------------------------------------------------------ */
/* FST transport cost (Sec. 3.3, Eq. 7-8).
 *
 * For source (retained) token s and target token t:
 *   d_f = 1 - cos(f_s, f_t),  d_x = |x_s - x_t|_2,  d_tau = max(0, tau_s - tau_t)
 *   C(s, t) = lambda_f d_f / M_f + lambda_x phi_kappa(d_x / M_x) + lambda_tau d_tau / M_tau
 * where each M is that discrepancy's maximum over all N^2 ordered pairs of the
 * scene ("min-max normalised within the sample"; the minimum is 0 because
 * d(t, t) = 0); a term whose M is 0 is 0.  cos with a zero-norm feature is 0,
 * d_f is clamped to [0, 2] and d_f(t, t) = 0.
 *
 *   feats   [n, d] features, dtype CP_F32 (float) or CP_BF16 (bfloat16);
 *           d % 8 == 0 for CP_BF16 and d % 4 == 0 for CP_F32
 *   pos     [n, 3] float positions in metres
 *   frame   [n] int32 frame indices
 *   cost    [n, n] float output, TARGET-MAJOR: cost[t * n + s] = C(s, t), so
 *           row t lists what every candidate s would pay to cover t
 *   maxima  [3] float output (may be NULL): M_f, M_x, M_tau
 *   Accumulation: features are multiplied in their storage type and summed in
 *   float32 (bfloat16 products on the matrix cores).
 */
size_t coverprune_fst_cost_workspace(int64_t n, int64_t d, cp_dtype dtype);
cp_status coverprune_fst_cost(const void* feats, cp_dtype dtype, int64_t n, int64_t d,
                              const float* pos, const int32_t* frame, cp_fst_weights w,
                              float* cost, float* maxima, void* workspace,
                              size_t workspace_bytes, void* stream);

/* Largest scene and neighbour count of the 3D nearest-neighbour tables
 * (coverprune_knn, coverprune_fst_capacity). */
#define CP_KNN_MAX_N 32768
#define CP_KNN_MAX_G 1024

/* ------------------------------------------------------------------------ */
/* FST capacity (Sec. 3.4, Eq. 9-10).
 *
 *   r_j = (1/n) sum_{k in N_n(j)} ( alpha_f d_f(j,k)/M_f + alpha_x d_x(j,k)/M_x
 *                                   + alpha_tau d_tau(j,k)/M_tau ),
 *   v_j = r_j / sum_l r_l          (uniform 1/N when every r_j is 0).
 *
 * N_n(j) is the n tokens nearest to j in 3D other than j itself, in the
 * (distance, index) order of coverprune_knn.  d_f = 1 - cos clamped to
 * [0, 2] (cos = 0 for a zero-norm row), d_x the Euclidean distance,
 * d_tau(j, k) = ReLU(tau_j - tau_k), as in the cost; each M is that term's
 * maximum over the N * n scored pairs (a term whose maximum is 0 adds 0).
 * phi of Eq. 10 is the identity.  Dot products, norms, scores and the sum are
 * float64; the capacity is rounded once to float32.  Deterministic.
 *
 *   feats, dtype, n, d, pos, frame: as for coverprune_fst_cost, 2 <= n <= CP_KNN_MAX_N
 *   n_nb      neighbours per token, 1 <= n_nb <= min(n - 1, CP_KNN_MAX_G - 1)
 *   alpha     term weights, finite and >= 0 (the experiments use 1, Sec. 5.1)
 *   capacity  [n] float output v, the input of the greedy and of Lite
 *   score     [n] double output r (may be NULL)
 *   workspace about (4 + 24 n_nb) bytes per token
 */
typedef struct {
  float alpha_f, alpha_x, alpha_tau;
} cp_capacity_weights;

size_t coverprune_fst_capacity_workspace(int64_t n, int64_t n_nb);
cp_status coverprune_fst_capacity(const void* feats, cp_dtype dtype, int64_t n, int64_t d, const float* pos,
                                  const int32_t* frame, int64_t n_nb, cp_capacity_weights alpha, float* capacity,
                                  double* score, void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------ */
/* Spatial-Guided Greedy Selection (Sec. 3.5, Eq. 11-16).
 *
 * Greedy over the coverage loss L(S) = sum_j v_j min(c0, min_{s in S} C(s, j)):
 * each step adds the unselected candidate c with the largest gain
 *   gain(c) = sum_j v_j max(0, b_j - C(c, j)),   b_j = min(c0, min_{s in S} C(s, j)),
 * i.e. the largest decrease of L (the free-source, epsilon -> 0 limit of the
 * semi-relaxed transport of Eq. 11-12, with every target as a neighbour,
 * g = N in Eq. 13).  Equal gains go to the smaller index; exactly k tokens
 * are selected even when gains reach 0.  Gains and L are summed in float64.
 *
 *   cost      [n, n] float, target-major as written by coverprune_fst_cost
 *   capacity  [n] float target capacities v (Sec. 3.4), v >= 0
 *   k         1 <= k <= n
 *   c0        cost of leaving a target uncovered; coverprune_uncovered_cost(w)
 *             (the largest value C can take) is the usual choice
 *   flags     CP_SGS_DENSE: every step sums every candidate's gain over the
 *             whole matrix (K full reads of the cost).
 *             CP_SGS_INCREMENTAL: the gains are summed once at b = c0 and then
 *             updated, step by step, from the rows of the targets whose best
 *             cost the pick lowers (their old and new b); the terms are the
 *             same float32 differences and float64 products, each rounded
 *             down onto a grid of 2^-S (c0 * sum v < 2^(62 - S) and
 *             c0 * max v < 2^(52 - S); costs are taken in [0, c0]) and summed
 *             exactly in 64-bit integers, so picks can differ from the dense
 *             sweep's float64 sums only between gains within rounding of
 *             each other.
 *             For n <= 32768 every compute unit keeps all n best costs and
 *             finds the targets a pick improves itself, from the pick's row
 *             of a source-major copy of the cost that the first pass writes
 *             into the workspace (4 n^2 bytes, 1 GiB at n = 16384).  For
 *             n <= 16384 the first steps, while a pick lowers at least 512
 *             best costs, split each step's improved targets between the
 *             compute units, which read those targets' whole rows and
 *             exchange per-column sums through the workspace (8 bytes per
 *             column and compute unit, up to 2 KB per token).  For
 *             n <= 16384 and k > 128 the steps after the 128th run from
 *             per-candidate lists of the targets each candidate can still
 *             improve (4 KB per token in the workspace), with the next
 *             winner predicted without an exchange when bounds that every
 *             compute unit computes identically prove it; the same
 *             integers, so the same picks.  Larger scenes, or
 *             CP_SGS_INCREMENTAL | CP_SGS_COMPACT, exchange the improved
 *             targets between the compute units instead (about 45 bytes
 *             per token, slower per step).  Both schedules sum the same
 *             integers and return the same result.
 *   selected        [k] int32 output: tokens in the order they were chosen
 *   step_gain       [k] double output (may be NULL): gain of each step
 *   step_objective  [k] double output (may be NULL): L(S) after each step
 *   assign          [n] int32 output (may be NULL): for each target the chosen
 *                   token that covers it most cheaply (the earliest chosen among
 *                   equals), or -1 if no chosen token costs less than c0
 */
/* Workspace for one form (flags as for coverprune_sgs_select; 0 for flags it
 * does not accept): the dense form needs about 9 MB at n = 16384 (private
 * best costs and float64 partial gains of up to 64 row panels), the
 * incremental form 4 n + 45 bytes per token up to n = 32768 (plus up to
 * 2 KB per token for the early steps' sums when n <= 16384, and 4 KB per
 * token for the candidate lists when n <= 16384 and k > 128) and about 45
 * bytes per token beyond that or with CP_SGS_COMPACT, each plus about
 * 100 KB of exchange slots. */
size_t coverprune_sgs_workspace(int64_t n, int64_t k, uint32_t flags);
cp_status coverprune_sgs_select(const float* cost, int64_t n, const float* capacity, int64_t k,
                                float c0, uint32_t flags, int32_t* selected, double* step_gain,
                                double* step_objective, int32_t* assign, void* workspace,
                                size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------ */
/* The whole prune of one scene (Sec. 3): the FST cost (Sec. 3.3, Eq. 7-8)
 * and the incremental greedy (Sec. 3.5, Eq. 11-16) in one call.
 *
 * The result is that of coverprune_fst_cost followed by coverprune_sgs_select
 * with CP_SGS_INCREMENTAL on the same arguments: the same cost in `cost`, the
 * same picks, gains, objective and assignment.  When n is a multiple of 64
 * and the greedy's rows schedule serves n (n <= 32768 on a device of 256
 * compute units), the cost's epilogue also writes the greedy's source-major
 * copy of the cost and its step-0 gains (as fixed-point partial sums over
 * blocks of 64 targets), so the greedy starts without a pass of its own over
 * the cost; otherwise the two calls' kernels run one after the other.
 *
 *   feats .. w       as for coverprune_fst_cost
 *   capacity .. c0   as for coverprune_sgs_select (c0 >= every cost value,
 *                    e.g. coverprune_uncovered_cost(w))
 *   cost             [n, n] float output, target-major (16-byte aligned)
 *   maxima           [3] float output (may be NULL), as for coverprune_fst_cost
 *   selected .. assign  outputs as for coverprune_sgs_select
 *   workspace        device memory of coverprune_prune_workspace bytes (0 for
 *                    bad sizes): the FST workspace, then the greedy's
 *                    incremental workspace, plus, when n is a multiple of 64,
 *                    the partial gains (8 bytes per column and block of 64
 *                    targets: 32 MB at n = 16384)
 * Errors: CP_ERR_INVALID_ARG / CP_ERR_UNSUPPORTED for bad arguments (checked
 * before anything is enqueued), CP_ERR_HIP when a launch fails.  A greedy
 * whose bounded waits give up writes -1 into every selected[] entry, as for
 * coverprune_sgs_select.
 */
size_t coverprune_prune_workspace(int64_t n, int64_t d, int64_t k, cp_dtype dtype);
cp_status coverprune_prune(const void* feats, cp_dtype dtype, int64_t n, int64_t d, const float* pos,
                           const int32_t* frame, cp_fst_weights w, const float* capacity, int64_t k, float c0,
                           float* cost, float* maxima, int32_t* selected, double* step_gain,
                           double* step_objective, int32_t* assign, void* workspace, size_t workspace_bytes,
                           void* stream);

/* ------------------------------------------------------------------------ */
/* Several scenes' greedies in one launch (the incremental form).
 *
 * Pruning runs once per request before the language model's prefill
 * (Sec. 5.1), and one scene's greedy occupies at most one compute unit per 64
 * tokens, so a few-thousand-token scene leaves most of the chip idle.  This
 * call runs up to CP_SGS_MAX_BATCH scenes of any sizes side by side in one
 * cooperative launch: scene s gets its own group of blocks (one block per
 * compute unit in all, groups balanced by tokens per block) and its own
 * exchanges, so each scene's result is what coverprune_sgs_select with
 * CP_SGS_INCREMENTAL computes for it alone (its block partition can differ,
 * which matters only for gains equal to 2^-31 relative in different blocks).
 * The call takes as long as its slowest scene.
 *
 *   scenes    host array of `count` scene descriptions (read during the call
 *             only); each field as for coverprune_sgs_select, all device memory
 *   count     1 <= count <= CP_SGS_MAX_BATCH (and at most the number of
 *             compute units)
 *   flags     CP_SGS_INCREMENTAL, or CP_SGS_INCREMENTAL | CP_SGS_COMPACT (as
 *             for coverprune_sgs_select; the small-workspace schedule also
 *             runs when any scene exceeds n = 32768)
 *   workspace the sum of the scenes' incremental workspaces for `flags`, laid
 *             out one after another; size from coverprune_sgs_batch_workspace
 *             (0 for bad scenes, count or flags)
 */
#define CP_SGS_MAX_BATCH 16
typedef struct {
  const float* cost;       /* [n, n] target-major */
  const float* capacity;   /* [n] */
  int64_t n;
  int64_t k;
  float c0;
  int32_t* selected;       /* [k] */
  double* step_gain;       /* [k] or NULL */
  double* step_objective;  /* [k] or NULL */
  int32_t* assign;         /* [n] or NULL */
} cp_sgs_scene;

size_t coverprune_sgs_batch_workspace(const cp_sgs_scene* scenes, int32_t count, uint32_t flags);
cp_status coverprune_sgs_select_batch(const cp_sgs_scene* scenes, int32_t count, uint32_t flags,
                                      void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------ */
/* The greedy without a workspace, for callers that cannot allocate memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc).
 *
 * coverprune_sgs_select with flags CP_SGS_INCREMENTAL | CP_SGS_COMPACT (the
 * same kernels, so the same result bit for bit), its scratch space taken
 * from a device array inside the library instead of a workspace argument:
 * about 1.5 MiB, one copy per GPU, held until the process ends.  The call
 * allocates nothing (no hipMalloc, hipFree or allocating library routine).
 * Its first call on a device looks up that device's copy of the array, with
 * the device current.
 *
 *   cost, n, capacity, k, c0, selected, step_gain, step_objective, assign:
 *             as for coverprune_sgs_select; n <= CP_SGS_NOALLOC_MAX_N (larger
 *             scenes return CP_ERR_INVALID_ARG before anything is enqueued)
 * Every call on one GPU uses that GPU's single scratch array, which keeps
 * the last call's contents (each call clears what must start at zero):
 * calls that overlap on one GPU, on different streams or from different
 * threads, race and give undefined results.  Serialise them.
 */
#define CP_SGS_NOALLOC_MAX_N 32768
cp_status coverprune_sgs_select_noalloc(const float* cost, int64_t n, const float* capacity, int64_t k, float c0,
                                        int32_t* selected, double* step_gain, double* step_objective,
                                        int32_t* assign, void* stream);

/* ------------------------------------------------------------------------ */
/* Spatially local greedy (Sec. 3.5, Eq. 13).
 *
 * The same greedy with each candidate's gain restricted to its neighbour set
 * M_g(c), the g targets nearest to it in 3D:
 *   gain(c) = sum_{j in M_g(c)} v_j max(0, b_j - C(c, j)),
 * while a pick still lowers b_j of every target it is cheaper for (the
 * residual of Eq. 14 is over all targets) and L(S) is summed over all of
 * them.  Each term takes the float64 difference of the two float32 costs and
 * a float64 product; every gain is summed afresh each step in exact 64-bit
 * fixed point at a scale of 2^-S with c0 * sum v < 2^(62 - S) (so only terms
 * below that resolution differ from a float64 sum).  Equal gains go to the
 * smaller index; exactly k tokens are selected.
 *
 * coverprune_knn writes the tables: row t lists the g tokens nearest to t,
 * ordered by (distance, index), t itself included.  Distances are compared as
 * float64 squared distances (dx^2 + dy^2) + dz^2 of the float32 positions,
 * formed without fused multiply-adds, so the tables are exact and
 * reproducible.
 *
 *   pos         [n, 3] float token positions (as for coverprune_fst_cost)
 *   g           1 <= g <= min(n, CP_KNN_MAX_G) for coverprune_knn,
 *               1 <= g <= min(n, CP_SGS_LOCAL_MAX_G) for the greedy
 *   neighbours  [n, g] int32, device memory: written by coverprune_knn, read
 *               by coverprune_sgs_local_select (row c = M_g(c); entries are
 *               clamped into [0, n); a target listed twice counts twice)
 *   cost, capacity, k, c0, selected, step_gain, step_objective, assign:
 *               as for coverprune_sgs_select (n <= CP_SGS_LOCAL_MAX_N)
 *
 * Both enqueue on `stream` and return before the work is done; bad sizes or
 * NULL pointers return CP_ERR_INVALID_ARG before anything is enqueued.  The
 * greedy keeps all n best costs on every compute unit and finds the targets
 * a pick improves from the pick's row of a source-major copy of the cost,
 * which it writes into the workspace first; the workspace is 4 n^2 bytes
 * for that copy (n rounded up to 256 per row; 1 GiB at n = 16384) plus 4 KB
 * per step of k for the objective's parts.
 */
#define CP_SGS_LOCAL_MAX_N 16384
#define CP_SGS_LOCAL_MAX_G 128
cp_status coverprune_knn(const float* pos, int64_t n, int64_t g, int32_t* neighbours, void* stream);
size_t coverprune_sgs_local_workspace(int64_t n, int64_t k);
cp_status coverprune_sgs_local_select(const float* cost, int64_t n, const float* capacity,
                                      const int32_t* neighbours, int64_t g, int64_t k, float c0,
                                      int32_t* selected, double* step_gain, double* step_objective,
                                      int32_t* assign, void* workspace, size_t workspace_bytes,
                                      void* stream);

/* ------------------------------------------------------------------------ */
/* The greedy step solved as written (Sec. 3.5, Eq. 11-15).
 *
 * Where coverprune_sgs_select reads each step's transport in its
 * epsilon -> 0, free-source limit, this call solves it: step l retains
 * S_l = {s_0 .. s_{l-1}} with source mass u = 1/k each and solves the
 * entropic semi-relaxed transport of Eq. 12 (P 1 = u, P^T 1 <= v) by
 * alternating scalings P = diag(a) E diag(b), E = exp(-C_S / epsilon):
 *   a <- u / (E b),   b <- min(1, v / (E^T a))   (b_j = 1 where E^T a is 0),
 * from b = 1, for `rounds` rounds.  The residual r = [v - P^T 1]_+ (Eq. 14)
 * weights the score sum_j r_j C(t, j) (Eq. 15, every target a neighbour; with
 * a restricted neighbourhood a covered one would score 0), and the unselected
 * token with the smallest score is retained (ties to the smaller index).
 * Step 0 has r = v, so the first pick is the capacity-weighted medoid.  After
 * k picks the same solve over the whole set gives the plan whose transport
 * cost <P, C_S> is reported as `objective`.  E and every sum are float64,
 * sums in a fixed order (deterministic); E underflows to 0 where
 * C / epsilon exceeds about 708, so epsilon should stay above max C / 700.
 * Each step costs `rounds` passes over an n x l matrix and one pass over the
 * cost.
 *
 *   cost, n, capacity: as for coverprune_sgs_select (every retained token must
 *             reach some target at finite E, e.g. C(s, s) = 0 as the FST cost has)
 *   k         1 <= k <= min(n, CP_SGS_LITERAL_MAX_K)
 *   epsilon   entropic regularisation, > 0, in the cost's units
 *   rounds    scaling rounds per solve, 1 <= rounds <= CP_SGS_LITERAL_MAX_ROUNDS
 *   follow    [k] int32 or NULL: picks to take instead of the argmin (a replay
 *             of another trajectory, e.g. to price the coverage-loss greedy's
 *             set); distinct indices in [0, n) are the caller's duty
 *   selected       [k] int32 output: the picks in order
 *   step_score     [k] double output (may be NULL): score of each pick
 *   step_residual  [k] double output (may be NULL): sum_j r_j before each pick
 *   objective      [1] double output (may be NULL): <P, C_S> of the final plan
 * With `follow` set and both step outputs NULL only the final plan is solved.
 * Workspace: about 8 k + 40 bytes per token plus 8 k per 64 tokens.
 */
#define CP_SGS_LITERAL_MAX_K 4096
#define CP_SGS_LITERAL_MAX_ROUNDS 1000000
size_t coverprune_sgs_literal_workspace(int64_t n, int64_t k);
cp_status coverprune_sgs_literal_select(const float* cost, int64_t n, const float* capacity, int64_t k,
                                        float epsilon, int32_t rounds, const int32_t* follow, int32_t* selected,
                                        double* step_score, double* step_residual, double* objective,
                                        void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------ */
/* CoverPrune-Lite (Sec. 4, Eq. 17-20).
 *
 *  1. Morton order: per axis q = floor((x - min_x) * (256 / voxel_size)) in
 *     float64, clamped to [0, 2^21 - 1]; key = bit interleave of (qx, qy, qz)
 *     with x in bit 0; tokens sorted by (key, index).  A token's voxel is
 *     q >> 8, so each voxel of edge voxel_size is a contiguous run.
 *  2. Groups (Eq. 17): V_j = floor(v_j * 2^40) in exact integers, W = sum V.
 *     Walking the order, the current group q closes before token p when
 *     K * (sum of V before p) >= (q + 1) * W, or when the tokens left equal
 *     the groups left; this yields exactly k non-empty contiguous groups of
 *     about 1/k capacity each.
 *  3. Costs: pairs in one group whose voxels are within one cell on every
 *     axis (27 neighbouring cells) cost C of Eq. 8 with M_f, M_x, M_tau taken
 *     over those pairs (diagonal included); other same-group pairs cost
 *     c0 = lambda_f + lambda_x + lambda_tau.
 *  4. Prototype of group q (Eq. 18): argmin over t in G_q of sum_{j in G_q}
 *     v_j C(t, j); ties to the smaller token index.
 *
 *   feats, dtype, n, d, pos, frame, w: as for coverprune_fst_cost
 *   capacity    [n] float target capacities, v >= 0, 0 < sum v < 2^20
 *   k           1 <= k <= n, k < 2^23
 *   voxel_size  voxel edge in metres, > 0
 *   selected    [k] int32 output: selected[q] is the prototype of group q
 *   group       [n] int32 output (may be NULL): group of every token
 *   objective   [1] double output (may be NULL): sum over groups of the
 *               prototype's cost, the block-plan transport cost of Eq. 20
 *   token_cost  [n] double output (may be NULL): every token t's cost to its
 *               group, sum_{j in G_q} v_j C(t, j), the quantity Eq. 18
 *               minimises (token order, not Morton order)
 * Every kernel of the call is an ordinary launch and no block waits for
 * another, so the call never gives up (COVERPRUNE_TEST_ABORT does not apply).
 */
size_t coverprune_lite_workspace(int64_t n, int64_t d, int64_t k, cp_dtype dtype);
cp_status coverprune_lite_select(const void* feats, cp_dtype dtype, int64_t n, int64_t d,
                                 const float* pos, const int32_t* frame, const float* capacity,
                                 int64_t k, cp_fst_weights w, float voxel_size, int32_t* selected,
                                 int32_t* group, double* objective, double* token_cost, void* workspace,
                                 size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------ */
/* Measurement: the latency floor of one greedy step on this device (Sec. 3.5).
 *
 * A step of coverprune_sgs_select's rows schedule cannot avoid two dependent
 * operations: the exchange in which every block publishes its best candidate
 * and reads every other block's, and the read of the winner's row of the
 * source-major cost (4 n bytes) that tells every block which targets the
 * pick improves.  This call runs `rounds` rounds of exactly those, with the
 * greedy's launch shape for a scene of n_rows tokens and its own slots,
 * waits and loads, and nothing else; each round's published key depends on
 * the previous round's row.  The call's duration divided by `rounds` is a
 * floor for a greedy step; with read_rows = 0 only the exchange runs.
 *
 *   rows      [n_rows, row_len] float device buffer, any contents (a cost
 *             matrix serves); row_len % 256 == 0, 256 <= row_len <= 32768
 *   rounds    >= 1
 *   workspace coverprune_step_floor_workspace() bytes (exchange slots)
 * Waits are bounded as in the greedy.
 */
size_t coverprune_step_floor_workspace(void);
cp_status coverprune_step_floor(const float* rows, int64_t n_rows, int64_t row_len, int32_t rounds,
                                int32_t read_rows, void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------ */
const char* coverprune_status_string(cp_status status); /* static text, never NULL */
const char* coverprune_last_error(void);                /* thread-local; "" if none */
int coverprune_abi_version(void);                       /* 2 */

#ifdef __cplusplus
}
#endif
#endif /* COVERPRUNE_H */
