/*
 * gba.h -- C ABI of the GBA (Global Batch gradients Aggregation) push-step on
 * one parameter-server shard, implemented with HIP kernels for gfx950 (MI355X).
 *
 * Paper: Wang et al., "Global Batch gradients Aggregation (GBA) for training
 * recommendation models", arXiv 2205.11048.  Sec. 3.1 defines the token
 * mechanism and the tolerance function (Eq. 1); Alg. 2 (PS workflow, push
 * responder) pops the K buffered gradients of one global batch, decays them,
 * takes the weighted sums (dense: divided by N_a; embeddings: divided by how
 * many workers sent the ID) and applies them.  K here is the
 * paper's M = N_a, the number of local-batch gradients aggregated per step.
 *
 * Conventions shared by every call:
 *  - Every array argument is a DEVICE pointer owned by the caller, except where
 *    a comment says otherwise.  The library never allocates, frees or keeps
 *    caller memory; scratch memory is passed in (size from a query).
 *  - Every call only enqueues work on `stream` (0 = the null stream) and
 *    returns without synchronising.
 *  - Misuse the host can see (null pointer, bad size, unsupported width,
 *    workspace too small) returns a non-zero gba_status and enqueues nothing.
 *  - Errors that depend on device data are OR-ed into the caller's `*err`
 *    word as GBA_DERR_* bits; the library never clears it.  When `*err` is
 *    non-zero after the stream has drained, the outputs of that call are
 *    undefined (but every access stayed inside the arrays described here).
 *  - No global state is mutated; calls on different streams may overlap when
 *    their arrays do not.
 */
#ifndef GBA_H
#define GBA_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum gba_status {
  GBA_OK = 0,
  GBA_ERR_NULL = 1,          /* a required pointer is NULL                   */
  GBA_ERR_INVALID_ARG = 2,   /* a size or mode is out of range               */
  GBA_ERR_UNSUPPORTED = 3,   /* valid but not supported (e.g. width D)       */
  GBA_ERR_WORKSPACE = 4,     /* workspace smaller than the size query asked  */
  GBA_ERR_HIP = 5,           /* a HIP launch failed                          */
  GBA_ERR_SCRATCH_LIMIT = 6  /* sizes beyond the no-allocation call's array   */
} gba_status;

/* Bits OR-ed into *err by device code. */
enum {
  GBA_DERR_ID_RANGE = 1,      /* an embedding ID outside [0, R)                    */
  GBA_DERR_FUTURE_TOKEN = 2,  /* a token newer than the step being applied         */
  GBA_DERR_OFFSETS = 4,       /* contribution offsets not 0 .. N and non-decreasing */
  GBA_DERR_ROW_RANGE = 8,     /* a row index passed to a sparse apply outside [0, R) */
  GBA_DERR_TABLE_FULL = 16    /* the ID index or the row pool has no room left      */
};

/* How embedding gradients are decayed (Alg. 2). */
typedef enum gba_decay {
  GBA_DECAY_TOKEN = 0,   /* every row of contribution m takes m's weight w_m          */
  GBA_DECAY_ID_TAG = 1   /* per-ID: s = max(0, tag[r] - tau_m + 1), weight [s <= iota] */
} gba_decay;

/* Divisor of the embedding weighted sum (Alg. 2). */
typedef enum gba_norm {
  GBA_NORM_PER_ID_COUNT = 0, /* c_r: contributions in the buffer that contain ID r */
  GBA_NORM_BY_K = 1          /* K: the synchronous global-batch mean               */
} gba_norm;

const char* gba_status_string(gba_status status);

/* Largest supported sizes. */
#define GBA_MAX_K 4096       /* contributions per call                        */
#define GBA_MAX_D 256        /* embedding width; D must be a multiple of 4    */

/*
 * Token weights -- Eq. 1 (Sec. 3.1).
 *   s_m = step - tokens[m];  w[m] = 1.0f if s_m <= iota, else 0.0f (excluded).
 * tokens     [K] int64, the global step at which contribution m's batch was issued.
 * w          [K] float out.
 * staleness  [K] int64 out, may be NULL.
 * num_excluded  one int32 out (count of w[m] == 0), may be NULL.
 * err        device error word; GBA_DERR_FUTURE_TOKEN when some s_m < 0 (that
 *            contribution then gets weight 0).
 * 1 <= K <= GBA_MAX_K.
 */
gba_status gba_token_weights(const int64_t* tokens, int32_t K, int64_t step, int64_t iota,
                             float* w, int64_t* staleness, int32_t* num_excluded,
                             int32_t* err, hipStream_t stream);

/*
 * Dense weighted sum divided by N_a -- Alg. 2 (push responder).
 *   out[i] = (sum over m with w[m] != 0 of w[m] * grads[m][i]) / K
 * accumulated in float64 in buffer order, rounded to float once.  A gradient
 * whose weight is 0 is never read (so it may hold anything, NaN included).
 * grads   DEVICE array of K device pointers, each to P floats.
 * w       [K] float (from gba_token_weights).
 * out     [P] float.
 * 1 <= K <= GBA_MAX_K, P >= 0.
 */
gba_status gba_aggregate_dense(const float* const* grads, const float* w, int32_t K, int64_t P,
                               float* out, hipStream_t stream);

/* Bytes of workspace gba_aggregate_sparse needs for these sizes. */
gba_status gba_aggregate_sparse_workspace_size(int64_t N, int32_t K, int32_t D, int64_t R,
                                               size_t* bytes /* host out */);

/*
 * Embedding gradients by ID -- Alg. 2 (push responder): dedup by ID, per-ID
 * decay, weighted sum divided by the number of contributions that hold the ID.
 * ids              [N] int64 embedding IDs in [0, R), contribution-major; ids, rows
 *                  and agg must be 16-byte aligned.
 * rows             [N][D] float, row j is the gradient of occurrence j.
 * contrib_offsets  [K+1] int64, occurrences of contribution m are
 *                  [offsets[m], offsets[m+1]); offsets[0] = 0, offsets[K] = N.
 * w, tokens        [K] token weights and tokens of the contributions.
 * tag              [R] int32, the last step each row was updated (-1: never).
 *                  Read and rewritten in GBA_DECAY_ID_TAG mode (every row with a
 *                  non-zero weight gets tag = step after all reads); ignored
 *                  (may be NULL) in GBA_DECAY_TOKEN mode.
 * Outputs, with U = number of distinct IDs (U <= N; size them for N):
 *   unique_ids     [U]   distinct IDs, ascending.
 *   seg_offsets    [U+1] exclusive prefix of the occurrence counts per ID.
 *   contrib_count  [U]   c_r, contributions that contain the ID.
 *   active_count   [U]   W_r, contributions with a non-zero weight for the ID.
 *   agg            [U][D] float, sum of the weighted rows of the ID (float64
 *                  accumulation) divided by c_r (or by K); 0 when W_r = 0.
 *   num_unique     one int64, U.
 * workspace        device scratch of at least the queried size.
 * Limits: 1 <= K <= GBA_MAX_K, 0 <= N < 2^28, 1 <= R <= 2^32,
 * D % 4 == 0 and 4 <= D <= GBA_MAX_D.
 */
gba_status gba_aggregate_sparse(const int64_t* ids, const float* rows,
                                const int64_t* contrib_offsets, int32_t K, int64_t N, int32_t D,
                                int64_t R, const float* w, const int64_t* tokens, int64_t step,
                                int64_t iota, int32_t* tag, gba_decay decay, gba_norm norm,
                                int64_t* unique_ids, int64_t* seg_offsets, int32_t* contrib_count,
                                int32_t* active_count, float* agg, int64_t* num_unique,
                                void* workspace, size_t workspace_bytes, int32_t* err,
                                hipStream_t stream);

/*
 * Optimiser apply (Table 1 names Adagrad and Adam; rules of Duchi et al. 2011
 * and Kingma and Ba 2015).  Arithmetic in float32 from the float32 state and
 * gradient (in every call that applies an optimiser), with the hardware
 * square root and reciprocal (each within 1 ulp) and the constants rounded
 * once from double, so each step is within a few float32 ulps and every
 * stored value takes one more rounding.
 *
 * Dense form (rows == NULL): elementwise over n elements of param/state/grad.
 * Row form (rows != NULL): for i < *num_rows (device int64, <= n), when
 * active == NULL or active[i] > 0, update table row r = rows[i] (param, state
 * are [R][D], grad is [n][D], row i of grad goes to row r).  Rows not listed
 * are untouched.  An r outside [0, R) sets GBA_DERR_ROW_RANGE and is skipped.
 * The row indices must be distinct (as gba_aggregate_sparse's unique_ids are).
 *
 * Adagrad: a' = a + g^2;  p' = p - lr * g / (sqrt(a') + eps).
 */
gba_status gba_apply_adagrad(float* param, float* accum, const float* grad, const int64_t* rows,
                             const int32_t* active, const int64_t* num_rows, int64_t n, int32_t D,
                             int64_t R, double lr, double eps, int32_t* err, hipStream_t stream);

/*
 * Adam with bias correction at step count t >= 1 (shared by the dense vector
 * and the rows; rows are updated only when listed, i.e. lazily):
 *   m' = b1 m + (1-b1) g;  v' = b2 v + (1-b2) g^2;
 *   p' = p - lr * (m' / (1 - b1^t)) / (sqrt(v' / (1 - b2^t)) + eps).
 */
gba_status gba_apply_adam(float* param, float* m, float* v, const float* grad, const int64_t* rows,
                          const int32_t* active, const int64_t* num_rows, int64_t n, int32_t D,
                          int64_t R, double lr, double beta1, double beta2, double eps, int64_t t,
                          int32_t* err, hipStream_t stream);

/*
 * gba_aggregate_sparse without a workspace argument, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc).  The call allocates nothing: its scratch
 * is a fixed device array of GBA_NOALLOC_SCRATCH_BYTES inside the library, one
 * per device, created when the library's code is first loaded on that device
 * and held until the process ends.  The first call on each device looks up the
 * array's address (make that first call outside graph capture).
 * Arguments, outputs, limits and errors as for gba_aggregate_sparse (agg is
 * required), plus GBA_ERR_SCRATCH_LIMIT, returned before any device work, when
 * gba_aggregate_sparse_workspace_size(N, K, D, R) exceeds the array (for
 * example N above 2^20 occurrences at D = 256, or about 2.5 * 2^20 at D = 32).
 * The outputs equal those of gba_aggregate_sparse bit for bit.
 * Every call on one device shares that device's array, and a call leaves its
 * contents behind (nothing in it must start at zero): calls that overlap in
 * time on one device, on different streams or from different host threads,
 * race on it and must be serialised by the caller.
 */
#define GBA_NOALLOC_SCRATCH_BYTES (64ull << 20)

gba_status gba_aggregate_sparse_noalloc(const int64_t* ids, const float* rows,
                                        const int64_t* contrib_offsets, int32_t K, int64_t N, int32_t D,
                                        int64_t R, const float* w, const int64_t* tokens, int64_t step,
                                        int64_t iota, int32_t* tag, gba_decay decay, gba_norm norm,
                                        int64_t* unique_ids, int64_t* seg_offsets, int32_t* contrib_count,
                                        int32_t* active_count, float* agg, int64_t* num_unique,
                                        int32_t* err, hipStream_t stream);

/*
 * gba_aggregate_sparse followed by the row form of gba_apply_adagrad /
 * gba_apply_adam over its active rows (Alg. 2: embeddings are updated by ID
 * with the per-ID mean; Table 1 names the optimisers), in one call.  Table,
 * state and every output come out bitwise equal to those of the two separate
 * calls (the same arithmetic and the same roundings).  With
 * Adagrad on rows of 20 to 32 floats (16 < D <= 32) the optimiser runs as each
 * ID's segment is finished, so the mean never makes a round trip through
 * memory; otherwise (other widths, Adam) the call aggregates and then applies.
 * ids ... num_unique   as for gba_aggregate_sparse, except that agg may be
 *                  NULL (the means are then not stored, or stored in the
 *                  workspace where they are needed).
 * table            [R][D] float, the embedding rows, updated in place (only
 *                  rows with W_r > 0 change).
 * accum / m, v     [R][D] float optimiser state, updated in place.
 * lr, eps, beta1, beta2, t   as for gba_apply_adagrad / gba_apply_adam.
 * workspace        at least gba_aggregate_apply_sparse_workspace_size bytes
 *                  for the optimiser (it includes room for the means where
 *                  they must go through memory and agg is NULL).
 * table and state must be 16-byte aligned.  Errors as for
 * gba_aggregate_sparse; also GBA_ERR_NULL for a missing table or state when
 * N > 0.
 */
enum { GBA_OPTIMIZER_ADAGRAD = 1, GBA_OPTIMIZER_ADAM = 2 };
gba_status gba_aggregate_apply_sparse_workspace_size(int64_t N, int32_t K, int32_t D, int64_t R,
                                                     int32_t optimizer /* GBA_OPTIMIZER_* */,
                                                     size_t* bytes /* host out */);

gba_status gba_aggregate_apply_sparse_adagrad(const int64_t* ids, const float* rows,
                                              const int64_t* contrib_offsets, int32_t K, int64_t N,
                                              int32_t D, int64_t R, const float* w, const int64_t* tokens,
                                              int64_t step, int64_t iota, int32_t* tag, gba_decay decay,
                                              gba_norm norm, int64_t* unique_ids, int64_t* seg_offsets,
                                              int32_t* contrib_count, int32_t* active_count, float* agg,
                                              int64_t* num_unique, float* table, float* accum, double lr,
                                              double eps, void* workspace, size_t workspace_bytes,
                                              int32_t* err, hipStream_t stream);

gba_status gba_aggregate_apply_sparse_adam(const int64_t* ids, const float* rows,
                                           const int64_t* contrib_offsets, int32_t K, int64_t N, int32_t D,
                                           int64_t R, const float* w, const int64_t* tokens, int64_t step,
                                           int64_t iota, int32_t* tag, gba_decay decay, gba_norm norm,
                                           int64_t* unique_ids, int64_t* seg_offsets, int32_t* contrib_count,
                                           int32_t* active_count, float* agg, int64_t* num_unique,
                                           float* table, float* m, float* v, double lr, double beta1,
                                           double beta2, double eps, int64_t t, void* workspace,
                                           size_t workspace_bytes, int32_t* err, hipStream_t stream);

/*
 * gba_aggregate_dense followed by the dense form of gba_apply_adagrad /
 * gba_apply_adam, in one pass over memory (Alg. 2: the weighted sum of the
 * dense gradients divided by K, then the Table 1 optimiser on the dense
 * parameters).  Each element's sum is rounded to float and applied exactly
 * as the two separate calls would, so param and state come out bitwise equal
 * to theirs; the sum itself never makes a round trip through memory.
 * grads, w, K, P   as for gba_aggregate_dense.
 * out              [P] float, receives the sum as gba_aggregate_dense would;
 *                  may be NULL.
 * param, accum / m, v   [P] float, updated in place.
 * lr, eps, beta1, beta2, t   as for gba_apply_adagrad / gba_apply_adam.
 * 16-byte-aligned buffers take the vector path; others work, more slowly.
 */
gba_status gba_aggregate_apply_dense_adagrad(const float* const* grads, const float* w, int32_t K,
                                             int64_t P, float* out, float* param, float* accum,
                                             double lr, double eps, hipStream_t stream);

/*
 * Host query, for profiling and for callers that count graph nodes: the
 * number of kernel launches one dense call over P elements with K
 * contributions makes on the current device (the weighted sum of Alg. 2 is
 * launched one round of resident blocks at a time when it spans more than two
 * rounds).  opt: 0 gba_aggregate_dense, 1 gba_aggregate_apply_dense_adagrad,
 * 2 gba_aggregate_apply_dense_adam, 3 gba_accumulate_dense (K = J).
 * launches   host out; 0 when P == 0.
 * Errors: GBA_ERR_NULL (launches), GBA_ERR_INVALID_ARG (K, P or opt out of range).
 */
gba_status gba_aggregate_dense_launches(int64_t P, int32_t K, int32_t opt, int64_t* launches);

gba_status gba_aggregate_apply_dense_adam(const float* const* grads, const float* w, int32_t K,
                                          int64_t P, float* out, float* param, float* m, float* v,
                                          double lr, double beta1, double beta2, double eps,
                                          int64_t t, hipStream_t stream);

/*
 * Early weighted sum of the dense gradients (App. B, with Alg. 2: the PS may
 * sum part of the buffer ahead of time, weighted by the tokens).  The
 * weight of a contribution depends only on its token and the step it will be
 * applied at, both known when it arrives, so it can be folded into a running
 * sum right away and the buffer holds P doubles instead of K gradients.
 *
 * gba_accumulate_dense: run[i] += w_j * g_j[i] for j = 0..J-1 in order, in
 * float64, skipping w_j == 0 (such gradients are never read).
 *   grads  device array of J gradient pointers, each [P] float.
 *   w      [J] float device weights (for example gba_token_weights of the J tokens).
 *   run    [P] double, device, caller-owned; all zero before the first
 *          contribution of a step (gba_finalize_* with reset != 0 leaves it so).
 *   1 <= J <= GBA_MAX_K.
 * gba_finalize_dense: out[i] = (float)(run[i] / K), K = the step's number of
 * contributions; run is cleared when reset != 0.
 * gba_finalize_apply_dense_*: the same sum, then the dense optimiser as in
 * gba_apply_adagrad / gba_apply_adam; out may be NULL.
 * Folding the contributions in buffer order, in any grouping into calls,
 * gives bitwise the results of gba_aggregate_dense / _apply_dense_* over the
 * whole buffer.  A 32-byte-aligned run and 16-byte-aligned arrays take the
 * vector path; others work, more slowly.
 */
gba_status gba_accumulate_dense(const float* const* grads, const float* w, int32_t J, int64_t P,
                                double* run, hipStream_t stream);

gba_status gba_finalize_dense(double* run, int32_t K, int64_t P, float* out, int32_t reset,
                              hipStream_t stream);

gba_status gba_finalize_apply_dense_adagrad(double* run, int32_t K, int64_t P, float* out,
                                            float* param, float* accum, double lr, double eps,
                                            int32_t reset, hipStream_t stream);

gba_status gba_finalize_apply_dense_adam(double* run, int32_t K, int64_t P, float* out, float* param,
                                         float* m, float* v, double lr, double beta1, double beta2,
                                         double eps, int64_t t, int32_t reset, hipStream_t stream);

/*
 * Grouping of embedding IDs by value -- the dedup step of gba_aggregate_sparse
 * (Alg. 2 handles embedding gradients per ID), on its own: a stable sort of
 * the IDs, keeping each one's occurrence index.
 *   ids        [n] int64 IDs in [0, R) (16-byte aligned).
 *   keys_out   [n] uint32 out, the IDs ascending.
 *   index_out  [n] uint32 out, the occurrence index of each sorted entry;
 *              equal IDs keep their input order.
 *   plan       GBA_SORT_AUTO, GBA_SORT_PLAIN or GBA_SORT_HOT: whether the
 *              frequent IDs found in a sample of the input are placed in the
 *              first pass so that only the others are sorted further (AUTO
 *              does so for large inputs).  The output does not depend on it.
 *   workspace  gba_sort_ids_workspace_size(n, R, plan) bytes.
 *   err        GBA_DERR_ID_RANGE for an ID outside [0, R) (sorted as 0).
 * Limits: 0 <= n < 2^28, 1 <= R <= 2^32.
 */
#define GBA_SORT_AUTO (-1)
#define GBA_SORT_PLAIN 0
#define GBA_SORT_HOT 1

gba_status gba_sort_ids_workspace_size(int64_t n, int64_t R, int32_t plan, size_t* bytes /* host out */);

gba_status gba_sort_ids(const int64_t* ids, int64_t n, int64_t R, int32_t plan, uint32_t* keys_out,
                        uint32_t* index_out, void* workspace, size_t workspace_bytes, int32_t* err,
                        hipStream_t stream);

/*
 * gba_aggregate_sparse with the sort plan chosen by the caller (GBA_SORT_AUTO,
 * GBA_SORT_PLAIN or GBA_SORT_HOT, as for gba_sort_ids); gba_aggregate_sparse
 * is this call with GBA_SORT_AUTO.  With the hot-key plan the frequent IDs
 * are also reduced apart from the others; every output is the same either way
 * (the sums to within their float64 rounding, taken in a fixed order).  The
 * workspace size depends on the plan.
 */
gba_status gba_aggregate_sparse_plan_workspace_size(int64_t N, int32_t K, int32_t D, int64_t R, int32_t plan,
                                                    size_t* bytes /* host out */);

gba_status gba_aggregate_sparse_plan(const int64_t* ids, const float* rows,
                                     const int64_t* contrib_offsets, int32_t K, int64_t N, int32_t D,
                                     int64_t R, const float* w, const int64_t* tokens, int64_t step,
                                     int64_t iota, int32_t* tag, gba_decay decay, gba_norm norm,
                                     int64_t* unique_ids, int64_t* seg_offsets, int32_t* contrib_count,
                                     int32_t* active_count, float* agg, int64_t* num_unique,
                                     void* workspace, size_t workspace_bytes, int32_t plan, int32_t* err,
                                     hipStream_t stream);

/*
 * Pull side (Sec. 3.1 token list; Alg. 2, pull responder).
 *
 * gba_token_of_batch (host function, no device work): the token handed out
 * with the i-th batch of the data list, t_i = floor(i / M) with M = K the
 * number of gradients aggregated per step: batches 0 .. M-1 get token 0, the
 * next M batches token 1, and so on.  (The formula printed in Sec. 3.1
 * divides by the number of updates K instead, which would contradict the
 * token count per value given beside it, M; the count is the one followed.)
 * Returns -1 if i < 0 or M < 1.
 *
 * gba_pull_rows: the embedding rows for a worker's request, looked up once per
 * distinct ID.
 *   ids         [n] int64 IDs in [0, R) of the request (16-byte aligned).
 *   table       [R][D] float embedding rows (16-byte aligned).
 *   unique_ids  [U] int64 out, the distinct IDs ascending (size it for n).
 *   inverse     [n] int32 out, ids[i] == unique_ids[inverse[i]].
 *   rows        [U][D] float out, rows[s] = table[unique_ids[s]] (16-byte aligned).
 *   num_unique  one int64 out, U.
 *   workspace   device scratch of gba_pull_workspace_size bytes.
 *   err         GBA_DERR_ID_RANGE for an ID outside [0, R) (outputs then undefined).
 * Limits: 0 <= n < 2^28, 1 <= R <= 2^32, D % 4 == 0 and 4 <= D <= GBA_MAX_D.
 */
int64_t gba_token_of_batch(int64_t i, int32_t M);

gba_status gba_pull_workspace_size(int64_t n, int64_t R, size_t* bytes /* host out */);

gba_status gba_pull_rows(const int64_t* ids, int64_t n, int64_t R, const float* table, int32_t D,
                         int64_t* unique_ids, int32_t* inverse, float* rows, int64_t* num_unique,
                         void* workspace, size_t workspace_bytes, int32_t* err, hipStream_t stream);

/*
 * Embedding storage keyed by 64-bit IDs (the paper's PS keeps embeddings in
 * expandable hash tables keyed by feature ID; Sec. 4.1 setting).  An
 * open-addressing index maps an ID to a row of a row pool; the push and pull
 * paths then run on row numbers (pass them as `ids`, with R = the pool size).
 *   slot_ids   [capacity] int64, the ID held by each slot (GBA_EMPTY_ID: free).
 *   slot_rows  [capacity] int32, the row of the ID in that slot.
 *   capacity   a power of two, <= 2^31; keep the load below about 0.7 and grow
 *              with gba_hash_rehash.
 * The ID value GBA_EMPTY_ID is reserved.  IDs are never removed.
 *
 * gba_hash_clear: every slot free (a fill kernel; no memset is recorded).
 *
 * gba_hash_find_or_insert: rows_out[i] = the row of ids[i]; an ID not yet in
 * the index gets a slot and the next free row of the pool.  The rows handed
 * out by one call are [old *num_rows, new *num_rows), in no particular order
 * of IDs; the caller initialises them (values and optimiser state) before the
 * step reads them.
 *   num_rows   one int64 on the device: rows in use (read and advanced).
 *   max_rows   size of the row pool (<= 2^31 - 1).
 *   row_ids    [max_rows] int64 out, row -> ID for the new rows; may be NULL.
 *   num_new    one int64 out on the device: IDs that asked for a row in this
 *              call (inserted now, or left without a row by an earlier call on
 *              a full pool); may be NULL.
 *   workspace  gba_hash_workspace_size(n) bytes.
 *   err        GBA_DERR_ID_RANGE for an ID equal to GBA_EMPTY_ID,
 *              GBA_DERR_TABLE_FULL when the index or the pool is full (those
 *              positions get row -1).  An ID that was given a slot but no
 *              row, because the pool was full, gets a row from a later call
 *              once the pool has room (a larger max_rows).
 * Which slot and which row an ID gets depends on the order in which threads
 * win their races; every other output is deterministic.
 *
 * gba_hash_rehash: build the index again at new_capacity (cleared here) from
 * the old one; rows do not move, so rows_out of later calls is unchanged.
 */
#define GBA_EMPTY_ID (-1)

gba_status gba_hash_clear(int64_t* slot_ids, int32_t* slot_rows, int64_t capacity, hipStream_t stream);

gba_status gba_hash_workspace_size(int64_t n, size_t* bytes /* host out */);

gba_status gba_hash_find_or_insert(int64_t* slot_ids, int32_t* slot_rows, int64_t capacity,
                                   const int64_t* ids, int64_t n, int64_t* rows_out, int64_t* num_rows,
                                   int64_t max_rows, int64_t* row_ids, int64_t* num_new, void* workspace,
                                   size_t workspace_bytes, int32_t* err, hipStream_t stream);

gba_status gba_hash_rehash(const int64_t* old_slot_ids, const int32_t* old_slot_rows, int64_t old_capacity,
                           int64_t* new_slot_ids, int32_t* new_slot_rows, int64_t new_capacity, int32_t* err,
                           hipStream_t stream);

#ifdef __cplusplus
}
#endif
#endif /* GBA_H */
