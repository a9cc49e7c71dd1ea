// C ABI of the GBA push-step (declared in include/gba.h): argument checks,
// workspace layout and launch order.  No allocation, no synchronisation.
#include <cmath>
#include <cstdint>
#include <mutex>

#include "gba_internal.hpp"

using namespace gba;

namespace {

constexpr int64_t kMaxN = (int64_t(1) << 28) - 1;

inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
inline size_t align_up(size_t x) { return (x + 255) & ~size_t(255); }

inline gba_status from_hip(hipError_t e) { return e == hipSuccess ? GBA_OK : GBA_ERR_HIP; }

bool width_ok(int32_t D) { return D >= 4 && D <= GBA_MAX_D && D % 4 == 0; }

size_t sparse_bytes(int64_t N, int32_t D, int64_t R, int32_t sort_plan, SortPlan* plan_out) {
  const SortPlan plan = plan_sort(N, R, sort_plan);
  if (plan_out) *plan_out = plan;
  return align_up(plan.bytes) + align_up(segments_workspace_bytes(N, D));
}

bool adam_args_ok(double beta1, double beta2, int64_t t) {
  return t >= 1 && beta1 >= 0.0 && beta1 < 1.0 && beta2 >= 0.0 && beta2 < 1.0;
}

AdamParams adam_params(double lr, double beta1, double beta2, double eps, int64_t t) {
  AdamParams hp;
  hp.lr = lr;
  hp.beta1 = beta1;
  hp.beta2 = beta2;
  hp.eps = eps;
  hp.bc1 = 1.0 - std::pow(beta1, (double)t);
  hp.bc2 = 1.0 - std::pow(beta2, (double)t);
  return hp;
}

}  // namespace

// ------------------------------------------------- the no-allocation variant
// Scratch of gba_aggregate_sparse_noalloc: one array per device, created when
// the code object is loaded there and held until the process ends.  Host code
// never passes `scratch` itself to a kernel (in host code the name is only a
// stand-in for the device symbol); it passes the device address looked up
// once per device below.
static __device__ __align__(256) unsigned char scratch[GBA_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};   // per device id; set once, under g_scratch_mu

// Device address of the current device's copy of `scratch`.
hipError_t current_device_scratch(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return hipSuccess;
}

}  // namespace

extern "C" {

const char* gba_status_string(gba_status s) {
  switch (s) {
    case GBA_OK: return "ok";
    case GBA_ERR_NULL: return "a required pointer is NULL";
    case GBA_ERR_INVALID_ARG: return "an argument is out of range";
    case GBA_ERR_UNSUPPORTED: return "unsupported size or width";
    case GBA_ERR_WORKSPACE: return "workspace too small";
    case GBA_ERR_HIP: return "a HIP launch failed";
    case GBA_ERR_SCRATCH_LIMIT:
      return "sizes need more scratch than the fixed device array of the no-allocation call holds";
  }
  return "unknown status";
}

gba_status gba_token_weights(const int64_t* tokens, int32_t K, int64_t step, int64_t iota, float* w,
                             int64_t* staleness, int32_t* num_excluded, int32_t* err,
                             hipStream_t stream) {
  if (!tokens || !w) return GBA_ERR_NULL;
  if (K < 1 || K > GBA_MAX_K) return GBA_ERR_INVALID_ARG;
  return from_hip(launch_token_weights(tokens, K, step, iota, w, staleness, num_excluded, err, stream));
}

gba_status gba_aggregate_dense(const float* const* grads, const float* w, int32_t K, int64_t P,
                               float* out, hipStream_t stream) {
  if (K < 1 || K > GBA_MAX_K || P < 0) return GBA_ERR_INVALID_ARG;
  if (P == 0) return GBA_OK;
  if (!grads || !w || !out) return GBA_ERR_NULL;
  return from_hip(launch_aggregate_dense(grads, w, K, P, out, stream));
}

gba_status gba_aggregate_dense_launches(int64_t P, int32_t K, int32_t opt, int64_t* launches) {
  if (!launches) return GBA_ERR_NULL;
  if (K < 1 || K > GBA_MAX_K || P < 0 || opt < 0 || opt > 3) return GBA_ERR_INVALID_ARG;
  *launches = dense_launch_count(P, K, opt);
  return GBA_OK;
}

gba_status gba_aggregate_apply_dense_adagrad(const float* const* grads, const float* w, int32_t K,
                                             int64_t P, float* out, float* param, float* accum, double lr,
                                             double eps, hipStream_t stream) {
  if (K < 1 || K > GBA_MAX_K || P < 0) return GBA_ERR_INVALID_ARG;
  if (P == 0) return GBA_OK;
  if (!grads || !w || !param || !accum) return GBA_ERR_NULL;
  return from_hip(launch_aggregate_apply_dense_adagrad(grads, w, K, P, out, param, accum, lr, eps, stream));
}

gba_status gba_aggregate_apply_dense_adam(const float* const* grads, const float* w, int32_t K, int64_t P,
                                          float* out, float* param, float* m, float* v, double lr,
                                          double beta1, double beta2, double eps, int64_t t,
                                          hipStream_t stream) {
  if (K < 1 || K > GBA_MAX_K || P < 0 || !adam_args_ok(beta1, beta2, t)) return GBA_ERR_INVALID_ARG;
  if (P == 0) return GBA_OK;
  if (!grads || !w || !param || !m || !v) return GBA_ERR_NULL;
  return from_hip(launch_aggregate_apply_dense_adam(grads, w, K, P, out, param, m, v,
                                                    adam_params(lr, beta1, beta2, eps, t), stream));
}

gba_status gba_accumulate_dense(const float* const* grads, const float* w, int32_t J, int64_t P, double* run,
                                hipStream_t stream) {
  if (J < 1 || J > GBA_MAX_K || P < 0) return GBA_ERR_INVALID_ARG;
  if (P == 0) return GBA_OK;
  if (!grads || !w || !run) return GBA_ERR_NULL;
  return from_hip(launch_accumulate_dense(grads, w, J, P, run, stream));
}

gba_status gba_finalize_dense(double* run, int32_t K, int64_t P, float* out, int32_t reset, hipStream_t stream) {
  if (K < 1 || P < 0) return GBA_ERR_INVALID_ARG;
  if (P == 0) return GBA_OK;
  if (!run || !out) return GBA_ERR_NULL;
  return from_hip(launch_finalize_dense(run, K, P, out, reset != 0, stream));
}

gba_status gba_finalize_apply_dense_adagrad(double* run, int32_t K, int64_t P, float* out, float* param,
                                            float* accum, double lr, double eps, int32_t reset,
                                            hipStream_t stream) {
  if (K < 1 || P < 0) return GBA_ERR_INVALID_ARG;
  if (P == 0) return GBA_OK;
  if (!run || !param || !accum) return GBA_ERR_NULL;
  return from_hip(launch_finalize_apply_dense_adagrad(run, K, P, out, param, accum, lr, eps, reset != 0, stream));
}

gba_status gba_finalize_apply_dense_adam(double* run, int32_t K, int64_t P, float* out, float* param, float* m,
                                         float* v, double lr, double beta1, double beta2, double eps, int64_t t,
                                         int32_t reset, hipStream_t stream) {
  if (K < 1 || P < 0 || !adam_args_ok(beta1, beta2, t)) return GBA_ERR_INVALID_ARG;
  if (P == 0) return GBA_OK;
  if (!run || !param || !m || !v) return GBA_ERR_NULL;
  return from_hip(launch_finalize_apply_dense_adam(run, K, P, out, param, m, v,
                                                   adam_params(lr, beta1, beta2, eps, t), reset != 0, stream));
}

gba_status gba_aggregate_sparse_plan_workspace_size(int64_t N, int32_t K, int32_t D, int64_t R, int32_t plan,
                                                    size_t* bytes) {
  if (!bytes) return GBA_ERR_NULL;
  if (K < 1 || K > GBA_MAX_K || N < 0 || N > kMaxN || R < 1 || R > (int64_t(1) << 32) || plan < -1 || plan > 1)
    return GBA_ERR_INVALID_ARG;
  if (!width_ok(D)) return GBA_ERR_UNSUPPORTED;
  *bytes = sparse_bytes(N, D, R, plan, nullptr);
  return GBA_OK;
}

gba_status gba_aggregate_sparse_workspace_size(int64_t N, int32_t K, int32_t D, int64_t R,
                                               size_t* bytes) {
  return gba_aggregate_sparse_plan_workspace_size(N, K, D, R, GBA_SORT_AUTO, bytes);
}

gba_status gba_aggregate_sparse(const int64_t* ids, const float* rows, const int64_t* contrib_offsets,
                                int32_t K, int64_t N, int32_t D, int64_t R, const float* w,
                                const int64_t* tokens, int64_t step, int64_t iota, int32_t* tag,
                                gba_decay decay, gba_norm norm, int64_t* unique_ids,
                                int64_t* seg_offsets, int32_t* contrib_count, int32_t* active_count,
                                float* agg, int64_t* num_unique, void* workspace,
                                size_t workspace_bytes, int32_t* err, hipStream_t stream) {
  return gba_aggregate_sparse_plan(ids, rows, contrib_offsets, K, N, D, R, w, tokens, step, iota, tag, decay, norm,
                                   unique_ids, seg_offsets, contrib_count, active_count, agg, num_unique, workspace,
                                   workspace_bytes, GBA_SORT_AUTO, err, stream);
}

// The sparse call behind gba_aggregate_sparse(_plan) and the fused
// aggregate-and-apply calls: ap (may be null) applies the rows as their
// segments are finished (agg may then be null).
static gba_status sparse_call(const int64_t* ids, const float* rows, const int64_t* contrib_offsets, int32_t K,
                              int64_t N, int32_t D, int64_t R, const float* w, const int64_t* tokens, int64_t step,
                              int64_t iota, int32_t* tag, gba_decay decay, gba_norm norm, int64_t* unique_ids,
                              int64_t* seg_offsets, int32_t* contrib_count, int32_t* active_count, float* agg,
                              int64_t* num_unique, void* workspace, size_t workspace_bytes, int32_t sort_plan,
                              const RowApply* ap, int32_t* err, hipStream_t stream) {
  if (K < 1 || K > GBA_MAX_K || N < 0 || N > kMaxN || R < 1 || R > (int64_t(1) << 32))
    return GBA_ERR_INVALID_ARG;
  if (sort_plan < -1 || sort_plan > 1) return GBA_ERR_INVALID_ARG;
  if (decay != GBA_DECAY_TOKEN && decay != GBA_DECAY_ID_TAG) return GBA_ERR_INVALID_ARG;
  if (norm != GBA_NORM_PER_ID_COUNT && norm != GBA_NORM_BY_K) return GBA_ERR_INVALID_ARG;
  if (!width_ok(D)) return GBA_ERR_UNSUPPORTED;
  if (!contrib_offsets || !w || !tokens || !seg_offsets || !num_unique || !workspace)
    return GBA_ERR_NULL;
  if (N > 0 && (!ids || !rows || !unique_ids || !contrib_count || !active_count || (!agg && !ap)))
    return GBA_ERR_NULL;
  if (decay == GBA_DECAY_ID_TAG) {
    if (!tag) return GBA_ERR_NULL;
    if (step < INT32_MIN || step > INT32_MAX) return GBA_ERR_INVALID_ARG;
  }
  if ((ids && !aligned16(ids)) || (rows && !aligned16(rows)) || (agg && !aligned16(agg)) ||
      !aligned16(workspace))
    return GBA_ERR_INVALID_ARG;
  SortPlan plan;
  const size_t need = sparse_bytes(N, D, R, sort_plan, &plan);
  // a row apply at a width the row pass does not fuse goes through agg, in
  // the workspace when the caller gives none
  const bool separate = ap && !segments_fuse_apply(D, ap->mode);
  const size_t agg_ws = (separate && !agg) ? align_up((size_t)N * D * sizeof(float)) : 0;
  if (workspace_bytes < need + agg_ws) return GBA_ERR_WORKSPACE;

  char* ws = static_cast<char*>(workspace);
  float* g = agg ? agg : (agg_ws ? reinterpret_cast<float*>(ws + need) : nullptr);
  const uint32_t* keys = nullptr;
  const uint32_t* vals = nullptr;
  // with the hot-key plan the frequent IDs are reduced apart from the rest
  SortHot hot;
  hipError_t e = launch_sort_ids(ids, N, R, plan, ws, &keys, &vals, err, stream, plan.hot ? &hot : nullptr);
  if (e != hipSuccess) return GBA_ERR_HIP;

  SegmentArgs a;
  if (plan.hot) {
    a.n_dev = hot.n_cold;
    a.hot = hot;
  }
  a.keys = keys;
  a.vals = vals;
  a.rows = rows;
  a.offsets = contrib_offsets;
  a.w = w;
  a.tokens = tokens;
  a.tag = tag;
  a.N = N;
  a.R = R;
  a.step = step;
  a.iota = iota;
  a.K = K;
  a.D = D;
  a.decay = (int)decay;
  a.norm = (int)norm;
  a.unique_ids = unique_ids;
  a.seg_offsets = seg_offsets;
  a.contrib_count = contrib_count;
  a.active_count = active_count;
  a.agg = g;
  a.num_unique = num_unique;
  a.err = err;
  if (ap && !separate) a.ap = *ap;
  e = launch_segments(a, ws + align_up(plan.bytes), stream);
  if (e != hipSuccess || !separate || N == 0) return from_hip(e);
  // the rows apply after the aggregation, over the active distinct IDs
  if (ap->mode == 2)
    e = launch_rows_adam(ap->p, ap->s1, ap->s2, g, unique_ids, active_count, num_unique, N, D, R,
                         AdamParams{ap->lr, ap->beta1, ap->beta2, ap->eps, ap->bc1, ap->bc2}, err, stream);
  else
    e = launch_rows_adagrad(ap->p, ap->s1, g, unique_ids, active_count, num_unique, N, D, R, ap->lr, ap->eps, err,
                            stream);
  return from_hip(e);
}

gba_status gba_aggregate_sparse_plan(const int64_t* ids, const float* rows, const int64_t* contrib_offsets,
                                     int32_t K, int64_t N, int32_t D, int64_t R, const float* w,
                                     const int64_t* tokens, int64_t step, int64_t iota, int32_t* tag,
                                     gba_decay decay, gba_norm norm, int64_t* unique_ids,
                                     int64_t* seg_offsets, int32_t* contrib_count, int32_t* active_count,
                                     float* agg, int64_t* num_unique, void* workspace,
                                     size_t workspace_bytes, int32_t sort_plan, int32_t* err, hipStream_t stream) {
  return sparse_call(ids, rows, contrib_offsets, K, N, D, R, w, tokens, step, iota, tag, decay, norm, unique_ids,
                     seg_offsets, contrib_count, active_count, agg, num_unique, workspace, workspace_bytes, sort_plan,
                     nullptr, err, stream);
}

gba_status gba_aggregate_sparse_noalloc(const int64_t* ids, const float* rows, const int64_t* contrib_offsets,
                                        int32_t K, int64_t N, int32_t D, int64_t R, const float* w,
                                        const int64_t* tokens, int64_t step, int64_t iota, int32_t* tag,
                                        gba_decay decay, gba_norm norm, int64_t* unique_ids,
                                        int64_t* seg_offsets, int32_t* contrib_count, int32_t* active_count,
                                        float* agg, int64_t* num_unique, int32_t* err, hipStream_t stream) {
  // sizes first: a call the fixed array cannot hold is refused before any
  // device work (and before the first-call symbol lookup)
  if (K < 1 || K > GBA_MAX_K || N < 0 || N > kMaxN || R < 1 || R > (int64_t(1) << 32))
    return GBA_ERR_INVALID_ARG;
  if (!width_ok(D)) return GBA_ERR_UNSUPPORTED;
  if (sparse_bytes(N, D, R, GBA_SORT_AUTO, nullptr) > (size_t)GBA_NOALLOC_SCRATCH_BYTES)
    return GBA_ERR_SCRATCH_LIMIT;
  void* ws = nullptr;
  if (current_device_scratch(&ws) != hipSuccess) return GBA_ERR_HIP;
  return sparse_call(ids, rows, contrib_offsets, K, N, D, R, w, tokens, step, iota, tag, decay, norm, unique_ids,
                     seg_offsets, contrib_count, active_count, agg, num_unique, ws,
                     (size_t)GBA_NOALLOC_SCRATCH_BYTES, GBA_SORT_AUTO, nullptr, err, stream);
}

gba_status gba_aggregate_apply_sparse_workspace_size(int64_t N, int32_t K, int32_t D, int64_t R, int32_t optimizer,
                                                     size_t* bytes) {
  if (optimizer != GBA_OPTIMIZER_ADAGRAD && optimizer != GBA_OPTIMIZER_ADAM) return GBA_ERR_INVALID_ARG;
  const gba_status st = gba_aggregate_sparse_workspace_size(N, K, D, R, bytes);
  if (st == GBA_OK && !segments_fuse_apply(D, optimizer)) *bytes += align_up((size_t)N * D * sizeof(float));
  return st;
}

gba_status gba_aggregate_apply_sparse_adagrad(const int64_t* ids, const float* rows, const int64_t* contrib_offsets,
                                              int32_t K, int64_t N, int32_t D, int64_t R, const float* w,
                                              const int64_t* tokens, int64_t step, int64_t iota, int32_t* tag,
                                              gba_decay decay, gba_norm norm, int64_t* unique_ids,
                                              int64_t* seg_offsets, int32_t* contrib_count, int32_t* active_count,
                                              float* agg, int64_t* num_unique, float* table, float* accum,
                                              double lr, double eps, void* workspace, size_t workspace_bytes,
                                              int32_t* err, hipStream_t stream) {
  if (N > 0 && (!table || !accum)) return GBA_ERR_NULL;
  if ((table && !aligned16(table)) || (accum && !aligned16(accum))) return GBA_ERR_INVALID_ARG;
  RowApply ap;
  ap.mode = GBA_OPTIMIZER_ADAGRAD;
  ap.p = table;
  ap.s1 = accum;
  ap.lr = lr;
  ap.eps = eps;
  return sparse_call(ids, rows, contrib_offsets, K, N, D, R, w, tokens, step, iota, tag, decay, norm, unique_ids,
                     seg_offsets, contrib_count, active_count, agg, num_unique, workspace, workspace_bytes,
                     GBA_SORT_AUTO, &ap, err, stream);
}

gba_status gba_aggregate_apply_sparse_adam(const int64_t* ids, const float* rows, const int64_t* contrib_offsets,
                                           int32_t K, int64_t N, int32_t D, int64_t R, const float* w,
                                           const int64_t* tokens, int64_t step, int64_t iota, int32_t* tag,
                                           gba_decay decay, gba_norm norm, int64_t* unique_ids,
                                           int64_t* seg_offsets, int32_t* contrib_count, int32_t* active_count,
                                           float* agg, int64_t* num_unique, float* table, float* m, float* v,
                                           double lr, double beta1, double beta2, double eps, int64_t t,
                                           void* workspace, size_t workspace_bytes, int32_t* err, hipStream_t stream) {
  if (!adam_args_ok(beta1, beta2, t)) return GBA_ERR_INVALID_ARG;
  if (N > 0 && (!table || !m || !v)) return GBA_ERR_NULL;
  if ((table && !aligned16(table)) || (m && !aligned16(m)) || (v && !aligned16(v))) return GBA_ERR_INVALID_ARG;
  const AdamParams hp = adam_params(lr, beta1, beta2, eps, t);
  RowApply ap;
  ap.mode = GBA_OPTIMIZER_ADAM;
  ap.p = table;
  ap.s1 = m;
  ap.s2 = v;
  ap.lr = hp.lr;
  ap.eps = hp.eps;
  ap.beta1 = hp.beta1;
  ap.beta2 = hp.beta2;
  ap.bc1 = hp.bc1;
  ap.bc2 = hp.bc2;
  return sparse_call(ids, rows, contrib_offsets, K, N, D, R, w, tokens, step, iota, tag, decay, norm, unique_ids,
                     seg_offsets, contrib_count, active_count, agg, num_unique, workspace, workspace_bytes,
                     GBA_SORT_AUTO, &ap, err, stream);
}

gba_status gba_sort_ids_workspace_size(int64_t n, int64_t R, int32_t plan, size_t* bytes) {
  if (!bytes) return GBA_ERR_NULL;
  if (n < 0 || n > kMaxN || R < 1 || R > (int64_t(1) << 32) || plan < -1 || plan > 1) return GBA_ERR_INVALID_ARG;
  *bytes = align_up(plan_sort(n, R, plan).bytes);
  return GBA_OK;
}

gba_status gba_sort_ids(const int64_t* ids, int64_t n, int64_t R, int32_t plan, uint32_t* keys_out,
                        uint32_t* index_out, void* workspace, size_t workspace_bytes, int32_t* err,
                        hipStream_t stream) {
  if (n < 0 || n > kMaxN || R < 1 || R > (int64_t(1) << 32) || plan < -1 || plan > 1) return GBA_ERR_INVALID_ARG;
  if (!workspace) return GBA_ERR_NULL;
  if (n > 0 && (!ids || !keys_out || !index_out)) return GBA_ERR_NULL;
  if ((ids && !aligned16(ids)) || !aligned16(workspace)) return GBA_ERR_INVALID_ARG;
  const SortPlan p = plan_sort(n, R, plan);
  if (workspace_bytes < align_up(p.bytes)) return GBA_ERR_WORKSPACE;
  if (n == 0) return GBA_OK;
  const uint32_t* keys = nullptr;
  const uint32_t* vals = nullptr;
  hipError_t e = launch_sort_ids(ids, n, R, p, workspace, &keys, &vals, err, stream);
  if (e != hipSuccess) return GBA_ERR_HIP;
  e = hipMemcpyAsync(keys_out, keys, (size_t)n * 4, hipMemcpyDeviceToDevice, stream);
  if (e == hipSuccess) e = hipMemcpyAsync(index_out, vals, (size_t)n * 4, hipMemcpyDeviceToDevice, stream);
  return from_hip(e);
}

int64_t gba_token_of_batch(int64_t i, int32_t M) {
  if (i < 0 || M < 1) return -1;
  return i / M;
}

gba_status gba_pull_workspace_size(int64_t n, int64_t R, size_t* bytes) {
  if (!bytes) return GBA_ERR_NULL;
  if (n < 0 || n > kMaxN || R < 1 || R > (int64_t(1) << 32)) return GBA_ERR_INVALID_ARG;
  *bytes = align_up(plan_sort(n, R).bytes) + align_up(pull_workspace_bytes(n));
  return GBA_OK;
}

gba_status gba_pull_rows(const int64_t* ids, int64_t n, int64_t R, const float* table, int32_t D,
                         int64_t* unique_ids, int32_t* inverse, float* rows, int64_t* num_unique, void* workspace,
                         size_t workspace_bytes, int32_t* err, hipStream_t stream) {
  if (n < 0 || n > kMaxN || R < 1 || R > (int64_t(1) << 32)) return GBA_ERR_INVALID_ARG;
  if (!width_ok(D)) return GBA_ERR_UNSUPPORTED;
  if (!num_unique || !workspace) return GBA_ERR_NULL;
  if (n > 0 && (!ids || !table || !unique_ids || !inverse || !rows)) return GBA_ERR_NULL;
  if ((ids && !aligned16(ids)) || (table && !aligned16(table)) || (rows && !aligned16(rows)) ||
      !aligned16(workspace))
    return GBA_ERR_INVALID_ARG;
  const SortPlan plan = plan_sort(n, R);
  if (workspace_bytes < align_up(plan.bytes) + align_up(pull_workspace_bytes(n))) return GBA_ERR_WORKSPACE;
  char* ws = static_cast<char*>(workspace);
  const uint32_t* keys = nullptr;
  const uint32_t* vals = nullptr;
  hipError_t e = launch_sort_ids(ids, n, R, plan, ws, &keys, &vals, err, stream);
  if (e != hipSuccess) return GBA_ERR_HIP;
  PullArgs a;
  a.keys = keys;
  a.vals = vals;
  a.n = n;
  a.R = R;
  a.table = table;
  a.D = D;
  a.unique_ids = unique_ids;
  a.inverse = inverse;
  a.rows = rows;
  a.num_unique = num_unique;
  return from_hip(launch_pull(a, ws + align_up(plan.bytes), stream));
}

static bool pow2_capacity(int64_t c) { return c >= 1 && c <= (int64_t(1) << 31) && (c & (c - 1)) == 0; }

gba_status gba_hash_clear(int64_t* slot_ids, int32_t* slot_rows, int64_t capacity, hipStream_t stream) {
  if (!pow2_capacity(capacity)) return GBA_ERR_INVALID_ARG;
  if (!slot_ids || !slot_rows) return GBA_ERR_NULL;
  return from_hip(launch_hash_clear(slot_ids, slot_rows, capacity, stream));
}

gba_status gba_hash_workspace_size(int64_t n, size_t* bytes) {
  if (!bytes) return GBA_ERR_NULL;
  if (n < 0 || n > kMaxN) return GBA_ERR_INVALID_ARG;
  *bytes = hash_workspace_bytes(n);
  return GBA_OK;
}

gba_status gba_hash_find_or_insert(int64_t* slot_ids, int32_t* slot_rows, int64_t capacity, const int64_t* ids,
                                   int64_t n, int64_t* rows_out, int64_t* num_rows, int64_t max_rows,
                                   int64_t* row_ids, int64_t* num_new, void* workspace, size_t workspace_bytes,
                                   int32_t* err, hipStream_t stream) {
  if (!pow2_capacity(capacity) || n < 0 || n > kMaxN || max_rows < 1 || max_rows > INT32_MAX)
    return GBA_ERR_INVALID_ARG;
  if (!slot_ids || !slot_rows || !num_rows || !workspace) return GBA_ERR_NULL;
  if (n > 0 && (!ids || !rows_out)) return GBA_ERR_NULL;
  if (workspace_bytes < hash_workspace_bytes(n)) return GBA_ERR_WORKSPACE;
  return from_hip(launch_hash_find_or_insert(slot_ids, slot_rows, capacity, ids, n, rows_out, num_rows, max_rows,
                                             row_ids, num_new, workspace, err, stream));
}

gba_status gba_hash_rehash(const int64_t* old_slot_ids, const int32_t* old_slot_rows, int64_t old_capacity,
                           int64_t* new_slot_ids, int32_t* new_slot_rows, int64_t new_capacity, int32_t* err,
                           hipStream_t stream) {
  if (!pow2_capacity(old_capacity) || !pow2_capacity(new_capacity)) return GBA_ERR_INVALID_ARG;
  if (!old_slot_ids || !old_slot_rows || !new_slot_ids || !new_slot_rows) return GBA_ERR_NULL;
  return from_hip(launch_hash_rehash(old_slot_ids, old_slot_rows, old_capacity, new_slot_ids, new_slot_rows,
                                     new_capacity, err, stream));
}

gba_status gba_apply_adagrad(float* param, float* accum, const float* grad, const int64_t* rows,
                             const int32_t* active, const int64_t* num_rows, int64_t n, int32_t D,
                             int64_t R, double lr, double eps, int32_t* err, hipStream_t stream) {
  if (n < 0) return GBA_ERR_INVALID_ARG;
  if (n == 0) return GBA_OK;
  if (!param || !accum || !grad) return GBA_ERR_NULL;
  if (!rows) return from_hip(launch_dense_adagrad(param, accum, grad, n, lr, eps, stream));
  if (!num_rows) return GBA_ERR_NULL;
  if (!width_ok(D)) return GBA_ERR_UNSUPPORTED;
  if (R < 1) return GBA_ERR_INVALID_ARG;
  if (!aligned16(param) || !aligned16(accum) || !aligned16(grad)) return GBA_ERR_INVALID_ARG;
  return from_hip(
      launch_rows_adagrad(param, accum, grad, rows, active, num_rows, n, D, R, lr, eps, err, stream));
}

gba_status gba_apply_adam(float* param, float* m, float* v, const float* grad, const int64_t* rows,
                          const int32_t* active, const int64_t* num_rows, int64_t n, int32_t D,
                          int64_t R, double lr, double beta1, double beta2, double eps, int64_t t,
                          int32_t* err, hipStream_t stream) {
  if (n < 0 || !adam_args_ok(beta1, beta2, t)) return GBA_ERR_INVALID_ARG;
  if (n == 0) return GBA_OK;
  if (!param || !m || !v || !grad) return GBA_ERR_NULL;
  const AdamParams hp = adam_params(lr, beta1, beta2, eps, t);
  if (!rows) return from_hip(launch_dense_adam(param, m, v, grad, n, hp, stream));
  if (!num_rows) return GBA_ERR_NULL;
  if (!width_ok(D)) return GBA_ERR_UNSUPPORTED;
  if (R < 1) return GBA_ERR_INVALID_ARG;
  if (!aligned16(param) || !aligned16(m) || !aligned16(v) || !aligned16(grad))
    return GBA_ERR_INVALID_ARG;
  return from_hip(launch_rows_adam(param, m, v, grad, rows, active, num_rows, n, D, R, hp, err, stream));
}

}  // extern "C"
