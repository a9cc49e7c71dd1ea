// Host-side launchers of the GBA kernels, shared between the kernel sources
// and the C ABI layer.  Every launcher only enqueues on `stream` and returns
// the launch status; argument checks happen in the C ABI layer.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "gba.h"

namespace gba {

// ---- token weights (Eq. 1)
hipError_t launch_token_weights(const int64_t* tokens, int32_t K, int64_t step, int64_t iota,
                                float* w, int64_t* staleness, int32_t* num_excluded, int32_t* err,
                                hipStream_t stream);

// ---- dense weighted sum / N_a (Alg. 2)
// Kernel launches one dense call makes (opt: 0 sum only, 1 fused Adagrad,
// 2 fused Adam, 3 early accumulation), on the current device.
int64_t dense_launch_count(int64_t P, int32_t K, int opt);
hipError_t launch_aggregate_dense(const float* const* grads, const float* w, int32_t K, int64_t P,
                                  float* out, hipStream_t stream);

// ---- dense and row optimiser apply
struct AdamParams {
  double lr, beta1, beta2, eps, bc1, bc2;   // bc = 1 - beta^t
};
hipError_t launch_dense_adagrad(float* p, float* a, const float* g, int64_t n, double lr, double eps,
                                hipStream_t stream);
// the weighted sum and the optimiser in one pass; out (the sum) may be null
hipError_t launch_aggregate_apply_dense_adagrad(const float* const* grads, const float* w, int32_t K,
                                                int64_t P, float* out, float* p, float* a, double lr,
                                                double eps, hipStream_t stream);
hipError_t launch_dense_adam(float* p, float* m, float* v, const float* g, int64_t n,
                             const AdamParams& hp, hipStream_t stream);
hipError_t launch_aggregate_apply_dense_adam(const float* const* grads, const float* w, int32_t K,
                                             int64_t P, float* out, float* p, float* m, float* v,
                                             const AdamParams& hp, hipStream_t stream);
// early weighted sum: fold J gradients into the float64 running sum run[P];
// then finish (divide by K, optionally apply) and optionally clear run
hipError_t launch_accumulate_dense(const float* const* grads, const float* w, int32_t J, int64_t P, double* run,
                                   hipStream_t stream);
hipError_t launch_finalize_dense(double* run, int32_t K, int64_t P, float* out, int reset, hipStream_t stream);
hipError_t launch_finalize_apply_dense_adagrad(double* run, int32_t K, int64_t P, float* out, float* p, float* a,
                                               double lr, double eps, int reset, hipStream_t stream);
hipError_t launch_finalize_apply_dense_adam(double* run, int32_t K, int64_t P, float* out, float* p, float* m,
                                            float* v, const AdamParams& hp, int reset, hipStream_t stream);
hipError_t launch_rows_adagrad(float* p, float* a, const float* g, const int64_t* rows,
                               const int32_t* active, const int64_t* num_rows, int64_t n, int32_t D,
                               int64_t R, double lr, double eps, int32_t* err, hipStream_t stream);
hipError_t launch_rows_adam(float* p, float* m, float* v, const float* g, const int64_t* rows,
                            const int32_t* active, const int64_t* num_rows, int64_t n, int32_t D,
                            int64_t R, const AdamParams& hp, int32_t* err, hipStream_t stream);

// ---- device-wide exclusive scan of uint32 (in place allowed)
size_t scan_workspace_bytes(int64_t n);
hipError_t launch_exclusive_scan_u32(const uint32_t* in, uint32_t* out, int64_t n, uint32_t* total,
                                     void* ws, hipStream_t stream);

// ---- LSD radix sort of (u32 key, u32 occurrence index) pairs
struct SortPlan {
  int64_t n;
  int key_bits;          // significant key bits (>= 1)
  int passes;
  int first_bits;        // cold digit bits of the first pass (the later passes take 8)
  bool hot;              // hot-key plan: frequent IDs placed by the first pass
  int hot_cap;           // most hot IDs (hot plan)
  int64_t blocks;        // tiles of the first pass (the most of any pass)
  size_t bytes;          // workspace bytes
};
// hot_mode: -1 picks the hot-key plan for large inputs whose key width leaves
// room for it, 0 never, 1 whenever the key width allows.
SortPlan plan_sort(int64_t n, int64_t R, int hot_mode = -1);
// With the hot-key plan the sort can also hand over its two parts apart
// ("split"): the cold keys sorted in [0, *n_cold) of *keys_out / *vals_out,
// and the occurrence indices of the hot IDs grouped by hot ID (ascending
// within each).  Every hot ID occurs at least once (it was seen in the sample).
struct SortHot {
  const uint32_t* n_cold = nullptr;     // device word: number of cold keys (null: no hot plan)
  const uint32_t* hot_vals = nullptr;   // [n - n_cold] occurrence indices of the hot IDs
  const uint32_t* ids = nullptr;        // [256] hot IDs, ascending ([0, H) used)
  const uint16_t* bucket = nullptr;     // [1024] hot IDs whose key >> bshift is below the index
  const uint32_t* prefix = nullptr;     // [256] hot occurrences of the hot IDs before h; [H] = all
  const uint32_t* meta = nullptr;       // [0] = H
  int bshift = 0;
};
// Sorts ids (int64 [n], each checked against [0, R)) by value, stably.  The
// sorted keys and original occurrence indices are returned through
// *keys_out / *vals_out, which point into `ws`.  With `split` non-null and
// the hot-key plan, the output is split as described above.
hipError_t launch_sort_ids(const int64_t* ids, int64_t n, int64_t R, const SortPlan& plan, void* ws,
                           const uint32_t** keys_out, const uint32_t** vals_out, int32_t* err,
                           hipStream_t stream, SortHot* split = nullptr);

// ---- segments over the sorted keys: dedup, counts, decayed weighted sums
// Fused row apply: the optimiser runs on each active row (W_r > 0) as its
// segment is finished, with the same arithmetic as the separate row apply,
// instead of the mean making a round trip through agg.
struct RowApply {
  int mode = 0;          // 0 none, 1 Adagrad, 2 Adam
  float* p = nullptr;    // [R][D] table
  float* s1 = nullptr;   // [R][D] Adagrad accumulator or Adam m
  float* s2 = nullptr;   // [R][D] Adam v
  double lr = 0.0, eps = 0.0, beta1 = 0.0, beta2 = 0.0, bc1 = 1.0, bc2 = 1.0;
};

struct SegmentArgs {
  const uint32_t* keys;        // sorted IDs [N]
  const uint32_t* vals;        // occurrence index of each sorted entry [N]
  const float* rows;           // [N][D]
  const int64_t* offsets;      // [K+1]
  const float* w;              // [K]
  const int64_t* tokens;       // [K]
  int32_t* tag;                // [R] or null
  int64_t N, R, step, iota;
  int32_t K, D;
  int decay, norm;
  int64_t* unique_ids;
  int64_t* seg_offsets;
  int32_t* contrib_count;
  int32_t* active_count;
  float* agg;
  int64_t* num_unique;
  int32_t* err;
  // Split hot-key plan: keys/vals hold only the cold keys, *n_dev of them,
  // and the hot IDs (hot) are reduced apart; the outputs interleave both in
  // ID order.  Null n_dev: keys/vals hold all N occurrences.
  const uint32_t* n_dev = nullptr;
  SortHot hot;
  RowApply ap;            // mode 0: agg is written and no row is applied
};
size_t segments_workspace_bytes(int64_t N, int32_t D);
// Whether launch_segments applies the rows itself for this optimiser (ap.mode)
// at width D: Adagrad on rows of 20 to 32 floats, where it was measured
// faster than the aggregation followed by the separate row apply (Adam, with
// two state rows per update, was measured slower fused).
bool segments_fuse_apply(int32_t D, int mode);
hipError_t launch_segments(const SegmentArgs& a, void* ws, hipStream_t stream);

// ---- runs of equal keys in sorted keys[N]: per 1024-position tile, the number
// of runs that start before it (tile_base[ceil(N/1024)]); *total = number of runs
constexpr int64_t kRunTile = 1024;
size_t run_heads_workspace_bytes(int64_t N);
// n_dev (optional): the number of keys, on the device (at most N)
hipError_t launch_run_heads(const uint32_t* keys, int64_t N, uint32_t* tile_base, uint32_t* total, void* scan_ws,
                            hipStream_t stream, const uint32_t* n_dev = nullptr);

// ---- pull side: distinct IDs of a worker's request, the inverse map, the rows
struct PullArgs {
  const uint32_t* keys;   // sorted IDs [n]
  const uint32_t* vals;   // request position of each sorted entry [n]
  int64_t n, R;
  const float* table;     // [R][D]
  int32_t D;
  int64_t* unique_ids;    // [U] ascending
  int32_t* inverse;       // [n] index into unique_ids of each request position
  float* rows;            // [U][D]
  int64_t* num_unique;
};
size_t pull_workspace_bytes(int64_t n);
hipError_t launch_pull(const PullArgs& a, void* ws, hipStream_t stream);

// ---- storage keyed by 64-bit IDs: open-addressing index (ID -> row) + row pool
size_t hash_workspace_bytes(int64_t n);
hipError_t launch_hash_clear(int64_t* slot_ids, int32_t* slot_rows, int64_t capacity, hipStream_t stream);
hipError_t launch_hash_find_or_insert(int64_t* slot_ids, int32_t* slot_rows, int64_t capacity, const int64_t* ids,
                                      int64_t n, int64_t* rows_out, int64_t* num_rows, int64_t max_rows,
                                      int64_t* row_ids, int64_t* num_new, void* ws, int32_t* err,
                                      hipStream_t stream);
hipError_t launch_hash_rehash(const int64_t* old_ids, const int32_t* old_rows, int64_t old_capacity, int64_t* new_ids,
                              int32_t* new_rows, int64_t new_capacity, int32_t* err, hipStream_t stream);

}  // namespace gba
