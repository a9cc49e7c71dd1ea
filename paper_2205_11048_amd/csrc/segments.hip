// Embedding gradients by ID (Alg. 2, push responder): after the occurrences
// are sorted by ID, every run of equal IDs is one segment.  For each segment
// this computes its ID and start (dedup), c_r (number of contributions that
// hold the ID: the divisor of Alg. 2, the count of workers that sent the ID),
// W_r (contributions whose weight for the ID is non-zero), and the weighted
// sum of the rows divided by c_r (or by K).  The weight of a contribution for
// a row is its token weight, or in per-ID mode [max(0, tag[r] - tau_m + 1) <=
// iota] with the tag as it was before this step.
//
// Work is split by sorted position, not by segment, so a Zipf-hot ID with
// millions of occurrences is spread over many blocks and no floating-point
// atomics are used.  Two passes over the sorted positions:
//  * seg_meta: one lane per position (coalesced key and index loads) finds
//    the contribution of the occurrence through a bucket table in LDS, its
//    weight, and whether it starts a run of equal IDs or a new contribution
//    inside one.  It numbers the segments, writes their IDs and starts, and
//    packs (occurrence index, flags) into one word per position.
//  * seg_rows: a group of LPR lanes (one 16-byte column slice per lane) walks
//    128 consecutive positions from their packed words, keeping 8 row gathers
//    in flight and summing each run in float64.  Runs that cross group
//    boundaries are joined in LDS; runs that cross tile boundaries leave one
//    partial per tile end, joined by seg_fixup in a fixed order, so results
//    are deterministic.
//
// With the split hot-key plan the sort hands over the cold keys and, apart,
// the occurrences of each hot ID (a few hundred IDs holding about half of all
// occurrences under Zipf skew).  The passes above then run over the cold keys
// only and write each segment at its place among all IDs; each hot ID is one
// long segment, summed by hot_rows (per 4096-occurrence chunk, no per-position
// segment logic) and finished by hot_finish, both in a fixed order.
#include "gba_device.hpp"
#include "gba_internal.hpp"
#include "optim.hpp"

namespace gba {

constexpr int kSegBlock = 256;
constexpr int kSegWaves = kSegBlock / kWave;                 // 4
constexpr int kRounds = 4;                                   // 16-byte loads per lane in seg_heads
constexpr int64_t kMetaTile = (int64_t)kSegBlock * kRounds;  // 1024 positions: 4 per thread of a block
static_assert(kMetaTile == kRunTile, "run-head tiles are the per-position tiles");
constexpr int kGroupSpan = 128;                              // positions per lane group (most; hot_rows)
constexpr int kBase32Span = 32;                              // the segment count is kept every 32 positions
constexpr int kBatch = 8;                                    // positions per batch of a group
// Row gathers in flight per group: a batch's rows are gathered and summed in
// two parts of four, which leaves the fused row pass 121 VGPRs (4 waves per
// SIMD) instead of 139 (3): more waves in flight beat more loads per wave.
constexpr int kBatchPart = 4;
constexpr int kMaxBuckets = 1024;                            // contribution lookup buckets

// packed word of a sorted position
constexpr uint32_t kIndexMask = (1u << 28) - 1u;  // occurrence index j (N < 2^28)
constexpr uint32_t kNonUnit = 1u << 28;           // weight is neither 0 nor 1
constexpr uint32_t kHead = 1u << 29;              // first position of a segment
constexpr uint32_t kNewC = 1u << 30;              // first occurrence of a contribution in its segment
constexpr uint32_t kZeroW = 1u << 31;             // weight 0: the row is never read

enum : uint32_t { kValid = 1, kOpen = 2, kPass = 4 };            // group flags

static inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }
static inline size_t align_up(size_t x) { return (x + 255) & ~size_t(255); }

static int lanes_per_row(int D) {
  int l = 1;
  while (l < 64 && l * 4 < D) l <<= 1;
  return l;
}
// Positions per lane group of the cold row pass: 128 for large inputs, fewer
// below, so that a pass over a few million positions still has waves enough
// to keep the memory busy (each group walks its span in batches, one after
// the other).
static int rows_span(int64_t N) { return N >= (int64_t(1) << 25) ? 128 : (N >= (int64_t(1) << 23) ? 64 : 32); }
// positions per row-pass tile: 4 waves x (64 / LPR) groups x span positions
static int64_t rows_tile(int lpr, int span) { return (int64_t)kSegWaves * (kWave / lpr) * span; }

// Bucket width 2^q so that at most kMaxBuckets buckets cover [0, N).
static int bucket_shift(int64_t N) {
  int q = 0;
  while (((N - 1) >> q) >= kMaxBuckets) ++q;
  return q;
}

struct SegPartials {
  double* first_acc;   // [tiles][D] chain that began in an earlier tile
  double* last_acc;    // [tiles][D] chain that continues into the next tile
  int32_t* first_cc;
  int32_t* first_ww;
  int32_t* last_cc;
  int32_t* last_ww;
  u32x4* fix_list;       // per tile whose last chain continues into the next
                         // tile: (tile, segment, last tile of the segment, 0)
  uint32_t* fix_count;   // entries of fix_list (cleared before the row pass)
};

constexpr int kHotSlots = 256;   // at least the sort's largest number of hot IDs (+1)
constexpr int kRecipMax = 256;   // divisors with a reciprocal in the row pass's table

struct SegLayout {
  int64_t meta_tiles, row_tiles, hot_chunks;
  size_t off_heads, off_total, off_scan, off_buckets, off_packed, off_base32,
      off_cnt, off_first_acc, off_last_acc, off_fix, off_start, off_cnum, off_hot_acc, off_hot_cnt, bytes;
};

static SegLayout seg_layout(int64_t N, int32_t D) {
  SegLayout L{};
  L.meta_tiles = N > 0 ? ceil_div(N, kMetaTile) : 1;
  L.row_tiles = N > 0 ? ceil_div(N, rows_tile(lanes_per_row(D), rows_span(N))) : 1;
  const size_t mt = (size_t)L.meta_tiles, rt = (size_t)L.row_tiles;
  const size_t n = (size_t)(N > 0 ? N : 1);
  size_t o = 0;
  L.off_heads = o;     o += align_up(mt * 4);
  L.off_total = o;     o += 256;                     // head total
  L.off_scan = o;      o += align_up(run_heads_workspace_bytes(N));
  L.off_buckets = o;   o += align_up(kMaxBuckets * 4);
  L.off_packed = o;    o += align_up((n + kGroupSpan) * 4);   // padded: whole-group vector loads stay inside
  L.off_base32 = o;    o += align_up((n / kBase32Span + 2) * 4);
  L.off_cnt = o;       o += align_up(rt * 16);
  L.off_fix = o;       o += 256 + align_up(rt * 16);  // count, then the list
  L.off_first_acc = o; o += align_up(rt * (size_t)D * 8);
  L.off_last_acc = o;  o += align_up(rt * (size_t)D * 8);
  // the position where each (cold) segment starts, and its end
  L.off_start = o;     o += align_up((n + 1) * 4);
  // per hot ID: the cold segments below it, the chunk prefix of its run, and
  // the cold positions below it
  L.off_cnum = o;      o += align_up(3 * (kHotSlots + 1) * 4);
  // per chunk of a hot run: float64 sums and (contributions, active, first and last contribution)
  L.hot_chunks = (N > 0 ? ceil_div(N, rows_tile(lanes_per_row(D), kGroupSpan)) : 1) + kHotSlots;
  L.off_hot_acc = o;   o += align_up((size_t)L.hot_chunks * D * 8);
  L.off_hot_cnt = o;   o += align_up((size_t)L.hot_chunks * 16);
  L.bytes = o;
  return L;
}

size_t segments_workspace_bytes(int64_t N, int32_t D) { return seg_layout(N, D).bytes; }

// ------------------------------------------------------------------ helpers
// First index in [lo, hi) whose offset exceeds j, or hi (off non-decreasing).
__device__ __forceinline__ int count_le(const int32_t* off, int lo, int hi, uint32_t j) {
  int len = hi - lo;
  while (len > 0) {
    const int half = len >> 1;
    if ((uint32_t)off[lo + half] <= j) {
      lo += half + 1;
      len -= half + 1;
    } else {
      len = half;
    }
  }
  return lo;
}

// Entries of the ascending s[0, n) that are at most x (n <= 256): a fixed
// sequence of halving steps, with no loop for the compiler to keep registers
// live across.
__device__ __forceinline__ uint32_t count_at_most(const uint32_t* s, uint32_t n, int64_t x) {
  uint32_t pos = 0;
#pragma unroll
  for (uint32_t step = 128; step >= 1; step >>= 1) {
    const uint32_t next = pos + step;
    if (next <= n && (int64_t)s[next - 1] <= x) pos = next;
  }
  return pos;
}

// Hot IDs below `key` (split plan): the sort's bucket table narrows the
// search to the hot IDs that share the key's top bits, then halving.
__device__ __forceinline__ uint32_t hot_below(uint32_t key, const uint16_t* bucket, const uint32_t* ids, uint32_t H,
                                              int bshift) {
  const uint32_t t = key >> bshift;
  uint32_t lo = bucket[t];
  uint32_t hi = t + 1 < 1024u ? (uint32_t)bucket[t + 1] : H;
  while (lo < hi) {
    const uint32_t mid = (lo + hi) >> 1;
    if (ids[mid] < key) lo = mid + 1;
    else hi = mid;
  }
  return lo;
}

// Contribution m of occurrence j (off[m] <= j < off[m+1]): start from the
// bucket table, step past at most one boundary, else search the rest.
__device__ __forceinline__ int contribution_of(const int32_t* s_off, const int32_t* s_bucket, int q,
                                               int K, uint32_t j) {
  int m = s_bucket[j >> q];
  if ((uint32_t)s_off[m + 1] <= j) {
    ++m;
    // first index past m + 1 whose offset exceeds j, minus one
    if ((uint32_t)s_off[m + 1] <= j) m = count_le(s_off, m + 1, K, j) - 1;
  }
  return m < K ? m : K - 1;
}

// The same from the int64 offsets in global memory (rare path).
__device__ __forceinline__ int contribution_global(const int64_t* off, int K, uint32_t j) {
  int lo = 1, len = K;
  while (len > 0) {
    const int half = len >> 1;
    if (off[lo + half] <= (int64_t)j) {
      lo += half + 1;
      len -= half + 1;
    } else {
      len = half;
    }
  }
  const int m = lo - 1;
  return m < 0 ? 0 : (m < K ? m : K - 1);
}

// Adagrad on one lane's 4 floats of a row, with the row apply's arithmetic.  The fused row pass applies
// Adagrad only (segments_fuse_apply); Adam goes through the separate apply.
__device__ __forceinline__ void adagrad4(const RowApply& ap, f32x4& pv, f32x4& s1, f32x4 g) {
  float pe[4] = {pv.x, pv.y, pv.z, pv.w}, ae[4] = {s1.x, s1.y, s1.z, s1.w};
  const float ge[4] = {g.x, g.y, g.z, g.w};
  const OptF32 c = opt_f32(ap.lr, ap.eps);
#pragma unroll
  for (int e = 0; e < 4; ++e) adagrad_update_f32(pe[e], ae[e], ge[e], c);
  pv = f32x4{pe[0], pe[1], pe[2], pe[3]};
  s1 = f32x4{ae[0], ae[1], ae[2], ae[3]};
}

// Row r updated with mean g (one lane's 16 bytes): load, Adagrad, store.
__device__ __forceinline__ void apply_row_part(const RowApply& ap, int64_t r, int D, int lane, f32x4 g) {
  const int64_t at = r * D + lane * 4;
  f32x4 pv = load_stream(reinterpret_cast<const f32x4*>(ap.p + at));
  f32x4 s1 = load_stream(reinterpret_cast<const f32x4*>(ap.s1 + at));
  adagrad4(ap, pv, s1, g);
  store_stream(reinterpret_cast<f32x4*>(ap.p + at), pv);
  store_stream(reinterpret_cast<f32x4*>(ap.s1 + at), s1);
}

// out: the segment's place among all distinct IDs.  The mean goes to agg
// (when given) and, with the fused Adagrad apply (mode 1; a constant in the row pass),
// into the optimiser update of row `row`, or where row < 0 of the ID the
// position pass wrote for this place (written by an earlier launch).
__device__ __forceinline__ void finalize_segment(const SegmentArgs& a, int64_t seg, f64x4 acc,
                                                 int cc, int ww, int lane, bool lane_on, int mode,
                                                 int64_t row = -1) {
  if (seg < 0 || seg >= a.N) return;   // unreachable when the numbering is consistent
  const double div = (a.norm == GBA_NORM_BY_K) ? (double)a.K : (double)cc;
  const f32x4 g = narrow(div_rounded(acc, div));
  if (lane_on && a.agg)
    store_stream(reinterpret_cast<f32x4*>(a.agg + seg * (int64_t)a.D + lane * 4), g);   // read once, by the apply
  if (mode != 0 && lane_on && ww > 0) {
    const int64_t r = row >= 0 ? row : a.unique_ids[seg];
    if (r >= 0 && r < a.R) apply_row_part(a.ap, r, a.D, lane, g);   // always in range when the numbering is consistent
  }
  if (lane == 0) {
    a.contrib_count[seg] = cc;
    a.active_count[seg] = ww;
  }
}

// Loads the per-contribution tables every block keeps in LDS: offsets [K+1],
// token weights [K], staleness step - tau [K] and the bucket table [nb].
__device__ __forceinline__ void load_contrib_tables(const SegmentArgs& a, const int32_t* buckets, int nb,
                                                    int32_t* s_off, float* s_w, int32_t* s_sm,
                                                    int32_t* s_bucket) {
  for (int i = threadIdx.x; i <= a.K; i += kSegBlock) {
    int64_t o = a.offsets[i];
    o = o < 0 ? 0 : (o > a.N ? a.N : o);
    s_off[i] = (int32_t)o;
    if (i < a.K) {
      s_w[i] = a.w[i];
      int64_t sm = a.step - a.tokens[i];
      sm = sm < -(1 << 30) ? -(1 << 30) : (sm > (1 << 30) ? (1 << 30) : sm);
      s_sm[i] = (int32_t)sm;
    }
  }
  for (int i = threadIdx.x; i < nb; i += kSegBlock) s_bucket[i] = buckets[i];
}

// The same tables in two halves, for K < 2 * kSegBlock: issue() loads a
// thread's entries into registers with clamped indices (no branch, so the
// caller can issue more loads before any is waited for) and store() writes
// them to LDS.
struct ContribTableRegs {
  static constexpr int kR = 2;                            // K + 1 <= 2 * kSegBlock entries
  static constexpr int kB = kMaxBuckets / kSegBlock;      // bucket entries per thread
  int64_t off[kR], tok[kR];
  float w[kR];
  int32_t bucket[kB];

  __device__ __forceinline__ void issue(const SegmentArgs& a, const int32_t* buckets, int nb) {
#pragma unroll
    for (int r = 0; r < kR; ++r) {
      const int i = threadIdx.x + r * kSegBlock;
      off[r] = a.offsets[i <= a.K ? i : a.K];
      w[r] = a.w[i < a.K ? i : a.K - 1];
      tok[r] = a.tokens[i < a.K ? i : a.K - 1];
    }
#pragma unroll
    for (int r = 0; r < kB; ++r) {
      const int i = threadIdx.x + r * kSegBlock;
      bucket[r] = buckets[i < nb ? i : nb - 1];
    }
  }
  __device__ __forceinline__ void store(const SegmentArgs& a, int nb, int32_t* s_off, float* s_w, int32_t* s_sm,
                                        int32_t* s_bucket) const {
#pragma unroll
    for (int r = 0; r < kR; ++r) {
      const int i = threadIdx.x + r * kSegBlock;
      if (i <= a.K) {
        const int64_t o = off[r] < 0 ? 0 : (off[r] > a.N ? a.N : off[r]);
        s_off[i] = (int32_t)o;
      }
      if (i < a.K) {
        s_w[i] = w[r];
        int64_t sm = a.step - tok[r];
        sm = sm < -(1 << 30) ? -(1 << 30) : (sm > (1 << 30) ? (1 << 30) : sm);
        s_sm[i] = (int32_t)sm;
      }
    }
#pragma unroll
    for (int r = 0; r < kB; ++r) {
      const int i = threadIdx.x + r * kSegBlock;
      if (i < nb) s_bucket[i] = bucket[r];
    }
  }
};
static_assert(kMaxBuckets % kSegBlock == 0, "whole bucket rounds");

// ------------------------------------------------------------------ kernels
__global__ void check_offsets_kernel(const int64_t* __restrict__ off, int K, int64_t N,
                                     int32_t* __restrict__ err) {
  bool bad = false;
  for (int m = threadIdx.x; m < K; m += blockDim.x) bad |= off[m] > off[m + 1];
  if (threadIdx.x == 0) bad |= (off[0] != 0) || (off[K] != N);
  if (bad) raise_error(err, GBA_DERR_OFFSETS);
}

// bucket[b] = contribution of occurrence b << q.
__global__ void contrib_buckets_kernel(const int64_t* __restrict__ off, int K, int64_t N, int q,
                                       int nb, int32_t* __restrict__ bucket) {
  for (int b = threadIdx.x; b < nb; b += blockDim.x) {
    const int64_t j = (int64_t)b << q;
    int lo = 1, len = K;
    while (len > 0) {
      const int half = len >> 1;
      int64_t o = off[lo + half];
      o = o < 0 ? 0 : (o > N ? N : o);
      if (o <= j) {
        lo += half + 1;
        len -= half + 1;
      } else {
        len = half;
      }
    }
    const int m = lo - 1;
    bucket[b] = m < K ? m : K - 1;
  }
}

// Run heads per 1024-position tile, one wave per tile.  Lane l holds
// positions t0 + 4 (l + 64 c) + e (c, e < 4): each 16-byte load of the wave
// covers 1 KB of consecutive keys, and the key before a lane's first one is
// the last key of the lane before it.
__global__ void __launch_bounds__(kSegBlock)
seg_heads_kernel(const uint32_t* __restrict__ keys, int64_t N_arg, const uint32_t* __restrict__ n_dev, int64_t tiles,
                 uint32_t* __restrict__ heads) {
  const int lane = lane_id();
  const int64_t tile = (int64_t)blockIdx.x * kSegWaves + threadIdx.x / kWave;
  if (tile >= tiles) return;   // whole waves leave; no block-wide barrier follows
  const int64_t N = n_dev ? (int64_t)*n_dev : N_arg;
  const int64_t t0 = tile * kMetaTile;
  if (t0 >= N) {   // past the keys on the device (a grid sized for the most keys)
    if (lane == 0) heads[tile] = 0u;
    return;
  }
  uint32_t carry = t0 > 0 ? keys[t0 - 1] : 0u;   // position 0 is always a head
  uint32_t cnt = 0;
#pragma unroll
  for (int c = 0; c < kRounds; ++c) {
    const int64_t i0 = t0 + 4 * ((int64_t)lane + (int64_t)kWave * c);
    uint32_t k[4] = {0u, 0u, 0u, 0u};
    if (i0 + 3 < N) {
      const u32x4 v = *reinterpret_cast<const u32x4*>(keys + i0);
      k[0] = v.x; k[1] = v.y; k[2] = v.z; k[3] = v.w;
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e) k[e] = (i0 + e < N) ? keys[i0 + e] : 0u;
    }
    uint32_t prev = __shfl_up(k[3], 1, kWave);
    if (lane == 0) prev = carry;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int64_t p = i0 + e;
      if (p < N) cnt += (p == 0 || k[e] != prev) ? 1u : 0u;
      prev = k[e];
    }
    carry = __shfl(k[3], kWave - 1, kWave);
  }
  const uint32_t total = wave_sum(cnt);
  if (lane == 0) heads[tile] = total;
}

// U, the end of the last segment, and (split plan) the defaults of the hot
// IDs' places: above every cold segment, until the position pass finds a
// cold segment above them.
__global__ void __launch_bounds__(kSegBlock)
seg_finish_kernel(const SegmentArgs a, const uint32_t* __restrict__ total, uint32_t* __restrict__ seg_start,
                  uint32_t* __restrict__ cnum, uint32_t* __restrict__ cold_below, uint32_t* __restrict__ fix_count) {
  const uint32_t U = *total;
  const uint32_t H = a.n_dev ? *a.hot.meta : 0u;
  const int64_t n = a.n_dev ? (int64_t)*a.n_dev : a.N;
  if (threadIdx.x == 0) {
    *a.num_unique = (int64_t)U + H;
    a.seg_offsets[U + H] = a.N;
    seg_start[U] = (uint32_t)n;
    *fix_count = 0u;   // the row pass appends to the fixup list
  }
  for (uint32_t h = threadIdx.x; h < H; h += kSegBlock) {
    cnum[h] = U;
    cold_below[h] = (uint32_t)n;
  }
}

// Per-position pass: numbering, segment IDs and starts, packed words.
// kMetaTilesPerBlock consecutive 1024-position tiles per block; in a tile each
// lane takes 4 consecutive positions (16-byte loads and stores), and the
// segment numbers come from a scan of the lanes' head counts.
constexpr int kMetaTilesPerBlock = 4;
constexpr int kMetaPer = 4;   // consecutive positions per lane
static_assert(kSegBlock * kMetaPer == kMetaTile, "a block covers one tile per pass");
__global__ void __launch_bounds__(kSegBlock)
seg_meta_kernel(SegmentArgs a, const uint32_t* __restrict__ tile_seg_base,
                const int32_t* __restrict__ buckets, int q, int nbuckets, int64_t num_tiles,
                uint32_t* __restrict__ packed, uint32_t* __restrict__ base32, uint32_t* __restrict__ seg_start,
                uint32_t* __restrict__ cnum, uint32_t* __restrict__ cold_below) {
  extern __shared__ int32_t s_dyn[];
  __shared__ uint32_t s_wave_heads[kSegWaves];
  // split plan: the hot IDs, their buckets and the hot occurrences below each
  __shared__ uint32_t s_hbucket[512];
  __shared__ uint32_t s_hids[kHotSlots];
  __shared__ uint32_t s_hprefix[kHotSlots];
  const int K = a.K;
  const int64_t N = a.N;                                        // occurrences
  const int64_t n = a.n_dev ? (int64_t)*a.n_dev : a.N;          // sorted positions (the cold ones when split)
  const bool split = a.n_dev != nullptr;
  int32_t* s_off = s_dyn;
  float* s_w = reinterpret_cast<float*>(s_dyn + K + 1);
  int32_t* s_sm = s_dyn + 2 * K + 1;
  int32_t* s_bucket = s_dyn + 3 * K + 1;
  // The lookup tables' loads are issued first (branch-free when K is below
  // 512), then, when every position of the block exists, all loads of its
  // tiles, so that the tables are waited for while the tiles are in flight.
  const int64_t blk0 = (int64_t)blockIdx.x * kMetaTilesPerBlock * kMetaTile;
  if (blk0 >= n) return;   // the grid is sized for every occurrence
  const bool full = blk0 + kMetaTilesPerBlock * kMetaTile <= n;
  uint32_t H = 0;
  if (split) {
    H = *a.hot.meta;
    const uint32_t* b32 = reinterpret_cast<const uint32_t*>(a.hot.bucket);
    for (int i = threadIdx.x; i < 512; i += kSegBlock) s_hbucket[i] = b32[i];
    s_hids[threadIdx.x] = a.hot.ids[threadIdx.x];
    s_hprefix[threadIdx.x] = a.hot.prefix[threadIdx.x];
  }
  const uint16_t* hbucket = reinterpret_cast<const uint16_t*>(s_hbucket);
  const bool small_k = K < ContribTableRegs::kR * kSegBlock;
  ContribTableRegs tables;
  if (small_k) tables.issue(a, buckets, nbuckets);
  // Loaded unconditionally (a branch would make the compiler wait for them
  // where its paths join): a block that is not full clamps its indices into
  // the arrays (the key and value arrays are padded to 64 entries, so a
  // 16-byte load at the last multiple of 4 below N stays inside them) and
  // uses none of these values.
  u32x4 kv[kMetaTilesPerBlock], vv[kMetaTilesPerBlock];
  uint32_t kpv[kMetaTilesPerBlock], jpv[kMetaTilesPerBlock], sb[kMetaTilesPerBlock];
  {
    const int64_t last4 = (n - 1) & ~int64_t(kMetaPer - 1);
#pragma unroll
    for (int kt = 0; kt < kMetaTilesPerBlock; ++kt) {
      int64_t p0 = blk0 + kt * kMetaTile + (int64_t)threadIdx.x * kMetaPer;
      p0 = p0 < last4 ? p0 : last4;
      kv[kt] = *reinterpret_cast<const u32x4*>(a.keys + p0);
      vv[kt] = *reinterpret_cast<const u32x4*>(a.vals + p0);
      const int64_t pp = p0 > 0 ? p0 - 1 : 0;   // used by lane 0 only, when p0 > 0
      kpv[kt] = a.keys[pp];
      jpv[kt] = a.vals[pp];
      int64_t t = (int64_t)blockIdx.x * kMetaTilesPerBlock + kt;
      sb[kt] = tile_seg_base[t < num_tiles ? t : num_tiles - 1];
    }
  }
  if (small_k)
    tables.store(a, nbuckets, s_off, s_w, s_sm, s_bucket);
  else
    load_contrib_tables(a, buckets, nbuckets, s_off, s_w, s_sm, s_bucket);
  __syncthreads();

  const int w = threadIdx.x / kWave;
  const int lane = lane_id();
  // One tile: key/jv are this lane's 4 positions from p0, kprev/jprev the
  // position before p0 (when p0 > 0), seg_base the segments before the tile.
  auto tile_body = [&](int64_t p0, const uint32_t* key, const uint32_t* jv, uint32_t kprev, uint32_t jprev,
                       uint32_t seg_base) {
    int m[kMetaPer];
#pragma unroll
    for (int e = 0; e < kMetaPer; ++e)
      m[e] = (p0 + e < n && (int64_t)jv[e] < N) ? contribution_of(s_off, s_bucket, q, K, jv[e]) : 0;
    // the position before this lane's first: the previous lane's last, or
    // (first lane of a wave) the one loaded for it
    uint32_t kp = __shfl_up(key[kMetaPer - 1], 1, kWave);
    int mp = __shfl_up(m[kMetaPer - 1], 1, kWave);
    bool prev_ok = true;
    if (lane == 0) {
      prev_ok = p0 > 0 && p0 - 1 < n;
      if (prev_ok) {
        kp = kprev;
        mp = (int64_t)jprev < N ? contribution_of(s_off, s_bucket, q, K, jprev) : 0;
      }
    }
    uint32_t word[kMetaPer];
    uint32_t heads = 0, head_bits = 0;
#pragma unroll
    for (int e = 0; e < kMetaPer; ++e) {
      const bool valid = p0 + e < n;
      const bool head = valid && (e == 0 ? (!prev_ok || key[0] != kp) : key[e] != key[e - 1]);
      const bool newc = valid && (head || m[e] != (e == 0 ? mp : m[e - 1]));
      float wt = 0.0f;
      if (valid) {
        if (a.decay == GBA_DECAY_TOKEN) {
          wt = s_w[m[e]];
        } else {
          const int64_t tg = ((int64_t)key[e] < a.R) ? (int64_t)a.tag[key[e]] : -1;
          int64_t st = tg - a.step + (int64_t)s_sm[m[e]] + 1;
          st = st < 0 ? 0 : st;
          wt = (st <= a.iota) ? 1.0f : 0.0f;
        }
      }
      word[e] = (jv[e] & kIndexMask) | (head ? kHead : 0u) | (newc ? kNewC : 0u) |
                (wt == 0.0f ? kZeroW : 0u) | ((wt != 0.0f && wt != 1.0f) ? kNonUnit : 0u);
      heads += head ? 1u : 0u;
      head_bits |= head ? (1u << e) : 0u;
    }
    if (p0 + kMetaPer - 1 < n) {
      *reinterpret_cast<u32x4*>(packed + p0) = u32x4{word[0], word[1], word[2], word[3]};
    } else {
#pragma unroll
      for (int e = 0; e < kMetaPer; ++e)
        if (p0 + e < n) packed[p0 + e] = word[e];
    }
    // segment numbers: the tile's base, the waves before, the lanes before
    const uint32_t incl = wave_inclusive_scan(heads);
    if (lane == kWave - 1) s_wave_heads[w] = incl;
    __syncthreads();
    uint32_t before = seg_base + incl - heads;
    for (int k = 0; k < w; ++k) before += s_wave_heads[k];
    // segments that start before each group-aligned position
    if ((p0 & (kBase32Span - 1)) == 0 && p0 < n) base32[p0 / kBase32Span] = before;
#pragma unroll
    for (int e = 0; e < kMetaPer; ++e) {
      if ((head_bits >> e) & 1u) {
        // split plan: the hot IDs below this key come before it among all IDs
        // (and their occurrences before its start); those above the key
        // before it (none for position 0) lie between the two segments
        uint32_t below = 0;
        if (split) {
          below = hot_below(key[e], hbucket, s_hids, H, a.hot.bshift);
          const uint32_t kprev = e == 0 ? kp : key[e - 1];
          const uint32_t from = (p0 + e > 0) ? hot_below(kprev, hbucket, s_hids, H, a.hot.bshift) : 0u;
          for (uint32_t h = from; h < below; ++h) {
            cnum[h] = before;
            cold_below[h] = (uint32_t)(p0 + e);
          }
        }
        const int64_t out = (int64_t)before + below;
        if (out < N) {   // always true when the numbering is consistent
          a.unique_ids[out] = (int64_t)key[e];
          a.seg_offsets[out] = p0 + e + (split ? (int64_t)s_hprefix[below] : 0);
          seg_start[before] = (uint32_t)(p0 + e);
        }
        ++before;
      }
    }
    __syncthreads();   // s_wave_heads is rewritten by the next tile
  };

  if (full) {
#pragma unroll
    for (int kt = 0; kt < kMetaTilesPerBlock; ++kt) {
      const int64_t p0 = blk0 + kt * kMetaTile + (int64_t)threadIdx.x * kMetaPer;
      const uint32_t key[kMetaPer] = {kv[kt].x, kv[kt].y, kv[kt].z, kv[kt].w};
      const uint32_t jv[kMetaPer] = {vv[kt].x, vv[kt].y, vv[kt].z, vv[kt].w};
      tile_body(p0, key, jv, kpv[kt], jpv[kt], sb[kt]);
    }
    return;
  }
  for (int kt = 0; kt < kMetaTilesPerBlock; ++kt) {
    const int64_t tile = (int64_t)blockIdx.x * kMetaTilesPerBlock + kt;
    if (tile >= num_tiles) break;
    const int64_t p0 = tile * kMetaTile + (int64_t)threadIdx.x * kMetaPer;
    uint32_t key[kMetaPer] = {0u, 0u, 0u, 0u}, jv[kMetaPer] = {0u, 0u, 0u, 0u};
#pragma unroll
    for (int e = 0; e < kMetaPer; ++e)
      if (p0 + e < n) {
        key[e] = a.keys[p0 + e];
        jv[e] = a.vals[p0 + e];
      }
    uint32_t kprev = 0, jprev = 0;
    if (p0 > 0 && p0 - 1 < n) {
      kprev = a.keys[p0 - 1];
      jprev = a.vals[p0 - 1];
    }
    tile_body(p0, key, jv, kprev, jprev, tile_seg_base[tile]);
  }
}

// Per-group pass: gather the kept rows and sum every run in float64.  APPLY
// (1: Adagrad, on rows of 20 to 32 floats only) updates each finished
// segment's row in the table as well.
template <int LPR, int APPLY, int SPAN>
__global__ void __launch_bounds__(kSegBlock)
seg_rows_kernel(SegmentArgs a, const uint32_t* __restrict__ packed, const uint32_t* __restrict__ base32,
                SegPartials part, const uint32_t* __restrict__ seg_start, const uint32_t* __restrict__ cnum) {
  constexpr int GW = kWave / LPR;            // groups per wave
  constexpr int G = kSegWaves * GW;          // groups per block
  constexpr int64_t TILE = (int64_t)G * SPAN;
  static_assert(SPAN % kBatch == 0 && SPAN % kBase32Span == 0 && SPAN <= kGroupSpan, "whole batches per group");
  // With one lane per 16 bytes of a 32-float row (eight groups of eight lanes
  // per wave), a segment that closes inside a batch is parked in LDS (its
  // row, place and counts, one slot per group and batch position) and the
  // wave writes the batch's parked segments together afterwards, eight rows
  // per store with every lane busy, instead of each group storing as its
  // segments close while the other groups' lanes idle.
  // With a row apply the parked segment also keeps its row (its ID), and the
  // wave updates the batch's rows together: the table and state rows of
  // several rounds of parked segments are requested before the first is used.
  constexpr bool kPark = LPR == 8 && GW == kBatch;
  static_assert(APPLY == 0 || kPark, "the row apply is fused where segments are parked");
  static_assert(APPLY == 0 || APPLY == 1, "the fused row apply is Adagrad only");
  constexpr int kSlots = GW * kBatch;
  // rows gathered at a time: the batch in parts of kPart (registers: each
  // lane holds kPart 16-byte row pieces while they are in flight)
  constexpr int kPart = kBatchPart;
  __shared__ f32x4 s_park[kPark ? kSegWaves : 1][kPark ? kSlots : 1][LPR];
  __shared__ uint32_t s_park_out[kPark ? kSegWaves : 1][kSlots];
  __shared__ uint32_t s_park_cw[kPark ? kSegWaves : 1][kSlots];
  __shared__ uint32_t s_park_list[kPark ? kSegWaves : 1][kSlots];
  __shared__ uint32_t s_park_key[APPLY ? kSegWaves : 1][APPLY ? kSlots : 1];
  // per-lane chain sums at the end of the groups: in the parking area of the
  // lane's own wave when parking (free by then), else their own array
  static_assert(!kPark || sizeof(s_park[0]) >= kWave * sizeof(f64x4), "chain sums fit a wave's parking area");
  __shared__ f64x4 s_acc_own[kPark ? 1 : kSegBlock];
  auto s_acc_at = [&](int t) -> f64x4& {
    if (kPark) return reinterpret_cast<f64x4*>(&s_park[t / kWave][0][0])[t % kWave];
    return s_acc_own[t];
  };
  __shared__ int32_t s_cc[G], s_ww[G];
  __shared__ uint32_t s_seg[G], s_flags[G];
  __shared__ uint32_t s_cnum[kHotSlots];
  // rounded reciprocals of the small divisors (a segment's contribution count)
  __shared__ double s_recip[kRecipMax + 1];

  const int64_t N = a.N;                                   // occurrences
  const int64_t n = a.n_dev ? (int64_t)*a.n_dev : a.N;     // sorted positions
  const int D = a.D;
  if ((int64_t)blockIdx.x * TILE >= n) return;   // the grid is sized for every occurrence
  // split plan: hot ID h comes before cold segment s among all IDs when
  // cnum[h] <= s (cnum ascending)
  const uint32_t H = a.n_dev ? *a.hot.meta : 0u;
  if (threadIdx.x < H) s_cnum[threadIdx.x] = cnum[threadIdx.x];
  for (int i = threadIdx.x; i <= kRecipMax; i += kSegBlock) s_recip[i] = 1.0 / (double)i;
  __syncthreads();
  const bool by_k = a.norm == GBA_NORM_BY_K;
  const double recip_k = 1.0 / (double)a.K;
  const bool small_k = a.K <= kRecipMax;

  const int w = threadIdx.x / kWave;
  const int lane = lane_id();
  const int gl = lane % LPR;                 // lane inside its group
  const int grp = w * GW + lane / LPR;       // group inside the block
  const bool lane_on = gl * 4 < D;

  {
    const int64_t tile = blockIdx.x;
    const int64_t p0 = tile * TILE + (int64_t)grp * SPAN;
    const int nvalid = (n - p0) >= SPAN ? SPAN : (n - p0 > 0 ? (int)(n - p0) : 0);
    const uint32_t gbase = nvalid > 0 ? base32[p0 / kBase32Span] : 0u;
    f64x4 acc = {0.0, 0.0, 0.0, 0.0};
    int cc = 0, ww = 0;
    int64_t seg = (int64_t)gbase - 1;
    // hot IDs before segment seg among all IDs (its output is seg + hb)
    uint32_t hb = H ? count_at_most(s_cnum, H, seg) : 0u;
    const uint32_t hb0 = hb;
    // the first segment number that has hot ID hb before it
    uint32_t hnext = hb < H ? s_cnum[hb] : 0xffffffffu;   // positions (and segments) stay below 2^32 - 1
    bool first_open = false;
    bool in_first = true;
    f64x4 facc = {0.0, 0.0, 0.0, 0.0};
    int fcc = 0, fww = 0;
    bool owner = false;
    uint32_t parked = 0;   // batch positions at which a segment of this group was parked
    uint32_t cur_key = (APPLY && nvalid > 0) ? a.keys[p0] : 0u;   // row of the open segment (row apply)
    // Words of the batch at i0 (the packed array is padded by a group span, so
    // whole vectors stay in bounds past the group's end).
    auto load_words = [&](int i0, uint32_t (&word)[kBatch]) {
      // a group past its positions (waves loop to their longest group) reads the first words, ignored
      const u32x4* wp = reinterpret_cast<const u32x4*>(packed + (i0 < nvalid ? p0 + i0 : 0));
#pragma unroll
      for (int v = 0; v < kBatch / 4; ++v) {
        const u32x4 x = wp[v];
        word[4 * v] = x.x; word[4 * v + 1] = x.y; word[4 * v + 2] = x.z; word[4 * v + 3] = x.w;
      }
    };
    // Keys of the batch at i0, for the row apply (zero past the sorted positions).
    auto load_keys = [&](int i0, uint32_t (&kk)[kBatch]) {
      const int64_t pk = (i0 < nvalid) ? p0 + i0 : 0;
      if (pk + kBatch <= n) {
        const u32x4* kp = reinterpret_cast<const u32x4*>(a.keys + pk);
#pragma unroll
        for (int v = 0; v < kBatch / 4; ++v) {
          const u32x4 x = kp[v];
          kk[4 * v] = x.x; kk[4 * v + 1] = x.y; kk[4 * v + 2] = x.z; kk[4 * v + 3] = x.w;
        }
      } else {
#pragma unroll
        for (int u = 0; u < kBatch; ++u) kk[u] = (pk + u < n) ? a.keys[pk + u] : 0u;
      }
    };
    // Every lane issues all of a batch's gathers: one whose row is not needed
    // (past the group, a zero weight, a lane past D) reads the first 16
    // bytes of the rows, which stay in cache, and is zeroed when summed.  With
    // no load inside a branch, the compiler can count the loads in flight and
    // never waits for all of them at once.
    // rows u0 .. u0 + kPart - 1 of the batch into rv[0 .. kPart)
    auto gather = [&](int i0, int u0, const uint32_t (&word)[kBatch], f32x4 (&rv)[kPart], uint32_t& use) {
#pragma unroll
      for (int v = 0; v < kPart; ++v) {
        const int u = u0 + v;
        const uint32_t jv = word[u] & kIndexMask;
        const bool on = i0 + u < nvalid && !(word[u] & kZeroW) && lane_on && (int64_t)jv < N;
        use |= on ? (1u << u) : 0u;
        rv[v] = *reinterpret_cast<const f32x4*>(a.rows + (on ? (int64_t)jv * D + gl * 4 : 0));
      }
    };
    // positions u0 .. u0 + kPart - 1 of the batch, their rows in rv[0 .. kPart)
    auto sum_batch = [&](int i0, int u0, const uint32_t (&word)[kBatch], const uint32_t (&kk)[kBatch],
                         f32x4 (&rv)[kPart], uint32_t use, bool weighted) {
#pragma unroll
      for (int v = 0; v < kPart; ++v)
        if (!((use >> (u0 + v)) & 1u)) rv[v] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int v = 0; v < kPart; ++v) {
        const int u = u0 + v;
        const int i = i0 + u;
        // keep each row's float64 widening next to its use: hoisting all of
        // them costs registers and the waves that keep gathers in flight
        __builtin_amdgcn_sched_barrier(0);
        if (i < nvalid) {
          if (word[u] & kHead) {
            if (i > 0) {
              if (in_first && first_open) {
                facc = acc; fcc = cc; fww = ww; owner = true;
              } else if (kPark) {
                const int slot = (lane / LPR) * kBatch + u;
                const double div = by_k ? (double)a.K : (double)cc;
                // a segment has at most K contributions: the table covers every count when K is small
                const double y = by_k ? recip_k : (small_k ? s_recip[cc] : 1.0 / div);
                if (lane_on) s_park[w][slot][gl] = narrow(div_rounded(acc, div, y));
                if (gl == 0) {
                  s_park_out[w][slot] = (uint32_t)(seg + hb);
                  s_park_cw[w][slot] = (uint32_t)cc | ((uint32_t)ww << 16);
                  if (APPLY) s_park_key[w][slot] = cur_key;
                }
                parked |= 1u << u;
              } else {
                finalize_segment(a, seg + hb, acc, cc, ww, gl, lane_on, APPLY);
              }
              in_first = false;
            }
            ++seg;
            if (APPLY) cur_key = kk[u];
            if ((uint32_t)seg >= hnext) {
              do ++hb; while (hb < H && (int64_t)s_cnum[hb] <= seg);
              hnext = hb < H ? s_cnum[hb] : 0xffffffffu;
            }
            acc = f64x4{0.0, 0.0, 0.0, 0.0};
            cc = ww = 0;
          }
          const bool zero = word[u] & kZeroW;
          if (!weighted) {
            acc += widen(rv[v]);
          } else if (!zero) {
            double wd = 1.0;
            if (word[u] & kNonUnit)   // a weight other than 0 or 1: look up its contribution
              wd = (double)a.w[contribution_global(a.offsets, a.K, word[u] & kIndexMask)];
            acc = fma_widen(wd, rv[v], acc);
          }
          const int nc = (word[u] & kNewC) ? 1 : 0;
          cc += nc;
          ww += (nc && !zero) ? 1 : 0;
        }
      }
    };
    // The parked segments of a batch, written by the whole wave: lane L
    // stands for slot L (group L / 8, batch position L % 8).
    auto flush = [&]() {
      const bool mine = (parked >> gl) & 1u;
      const uint64_t m = __ballot(mine);
      if (mine) s_park_list[w][__popcll(m & lanemask_lt())] = (uint32_t)lane;
      __builtin_amdgcn_wave_barrier();
      const int E = __popcll(m);
      if (APPLY) {
        // kR rounds at a time: the table and state rows of all their active
        // segments are requested, then updated (a lane without one reads the
        // table's first 16 bytes and writes nothing)
        constexpr int kR = 4;
        for (int b = 0; b < E; b += kR * GW) {
          f32x4 pv[kR], sv[kR];
          uint32_t slot[kR];
          int64_t outv[kR], row[kR];
          bool act[kR];
#pragma unroll
          for (int r = 0; r < kR; ++r) {
            const int e = b + r * GW + lane / LPR;
            slot[r] = e < E ? s_park_list[w][e] : 0u;
            outv[r] = e < E ? (int64_t)s_park_out[w][slot[r]] : N;   // out < N when the numbering is consistent
            act[r] = outv[r] < N && (s_park_cw[w][slot[r]] >> 16) > 0 && lane_on &&
                     (int64_t)s_park_key[w][slot[r]] < a.R;   // sorted keys are below R
            row[r] = act[r] ? (int64_t)s_park_key[w][slot[r]] : 0;
            const int64_t at = act[r] ? row[r] * D + gl * 4 : 0;   // inactive lanes read the table's first 16 bytes
            pv[r] = load_stream(reinterpret_cast<const f32x4*>(a.ap.p + at));
            sv[r] = load_stream(reinterpret_cast<const f32x4*>(a.ap.s1 + at));
          }
#pragma unroll
          for (int r = 0; r < kR; ++r) {
            if (outv[r] >= N) continue;
            const f32x4 g = s_park[w][slot[r]][gl];
            if (lane_on && a.agg) store_stream(reinterpret_cast<f32x4*>(a.agg + outv[r] * D + gl * 4), g);
            if (gl == 0) {
              const uint32_t v = s_park_cw[w][slot[r]];
              a.contrib_count[outv[r]] = (int32_t)(v & 0xffffu);
              a.active_count[outv[r]] = (int32_t)(v >> 16);
            }
            if (act[r]) {
              const int64_t at = row[r] * D + gl * 4;
              adagrad4(a.ap, pv[r], sv[r], g);
              store_stream(reinterpret_cast<f32x4*>(a.ap.p + at), pv[r]);
              store_stream(reinterpret_cast<f32x4*>(a.ap.s1 + at), sv[r]);
            }
          }
        }
      } else {
        for (int b = 0; b < E; b += GW) {
          const int e = b + lane / LPR;
          if (e < E) {
            const uint32_t slot = s_park_list[w][e];
            const int64_t out = s_park_out[w][slot];
            if (out < N) {   // always true when the numbering is consistent
              if (lane_on) store_stream(reinterpret_cast<f32x4*>(a.agg + out * D + gl * 4), s_park[w][slot][gl]);
              if (gl == 0) {
                const uint32_t v = s_park_cw[w][slot];
                a.contrib_count[out] = (int32_t)(v & 0xffffu);
                a.active_count[out] = (int32_t)(v >> 16);
              }
            }
          }
        }
      }
      __builtin_amdgcn_wave_barrier();   // the next batch reuses the slots
      parked = 0;
    };
    // every group of a wave runs the wave's longest group's batches, so the
    // flush sees the whole wave
    int iters = nvalid;
    if (kPark) {
#pragma unroll
      for (int off = kWave / 2; off > 0; off >>= 1) {
        const int o = __shfl_xor(iters, off, kWave);
        iters = o > iters ? o : iters;
      }
    }
    for (int i0 = 0; i0 < iters; i0 += kBatch) {
      uint32_t word[kBatch], kk[kBatch];
      load_words(i0, word);
      if (APPLY) load_keys(i0, kk);
      if (i0 == 0) first_open = !(word[0] & kHead);
      // weights other than 0 and 1 are rare: unless some position of the
      // wave's batch has one, rows are added without a multiply (a weight-0
      // row is zeroed), a branch the whole wave takes together
      bool nonunit = false;
#pragma unroll
      for (int u = 0; u < kBatch; ++u) nonunit |= i0 + u < nvalid && (word[u] & kNonUnit);
      const bool weighted = __ballot(nonunit) != 0ull;
      uint32_t use = 0;
#pragma unroll
      for (int u0 = 0; u0 < kBatch; u0 += kPart) {
        f32x4 rv[kPart];
        gather(i0, u0, word, rv, use);
        sum_batch(i0, u0, word, kk, rv, use, weighted);
      }
      if (kPark) flush();
    }

    bool last_open = false, pass = false;
    if (nvalid > 0) {
      last_open = nvalid == SPAN && (p0 + SPAN) < n && !(packed[p0 + SPAN] & kHead);
      if (last_open) {
        pass = in_first && first_open;
        s_acc_at(threadIdx.x) = acc;
        if (gl == 0) {
          s_cc[grp] = cc;
          s_ww[grp] = ww;
          s_seg[grp] = (uint32_t)seg;
        }
      } else if (in_first && first_open) {
        facc = acc; fcc = cc; fww = ww; owner = true;
      } else {
        finalize_segment(a, seg + hb, acc, cc, ww, gl, lane_on, APPLY);
      }
    }
    if (gl == 0) s_flags[grp] = (nvalid > 0 ? kValid : 0u) | (last_open ? kOpen : 0u) | (pass ? kPass : 0u);
    __syncthreads();

    // a group whose first run began before it closes the chain of runs
    if (owner) {
      f64x4 tot = facc;
      int tcc = fcc, tww = fww;
      bool from_prev_tile = true;
      for (int gg = grp - 1; gg >= 0; --gg) {
        tot += s_acc_at(gg * LPR + gl);
        tcc += s_cc[gg];
        tww += s_ww[gg];
        if (!(s_flags[gg] & kPass)) {
          from_prev_tile = false;
          break;
        }
      }
      if (from_prev_tile) {
        if (lane_on) *reinterpret_cast<f64x4*>(part.first_acc + tile * D + gl * 4) = tot;
        if (gl == 0) {
          part.first_cc[tile] = tcc;
          part.first_ww[tile] = tww;
        }
      } else {
        finalize_segment(a, (int64_t)gbase - 1 + hb0, tot, tcc, tww, gl, lane_on, APPLY);
      }
    }
    // the chain that runs into the next tile
    if (grp == G - 1 && (s_flags[G - 1] & kOpen)) {
      f64x4 tot = s_acc_at((G - 1) * LPR + gl);
      int tcc = s_cc[G - 1], tww = s_ww[G - 1];
      int gg = G - 1;
      while (gg > 0 && (s_flags[gg] & kPass)) {
        --gg;
        tot += s_acc_at(gg * LPR + gl);
        tcc += s_cc[gg];
        tww += s_ww[gg];
      }
      if (s_flags[gg] & kPass) {   // the whole tile is inside one segment
        if (lane_on) *reinterpret_cast<f64x4*>(part.first_acc + tile * D + gl * 4) = tot;
        if (gl == 0) {
          part.first_cc[tile] = tcc;
          part.first_ww[tile] = tww;
        }
      } else {
        if (lane_on) *reinterpret_cast<f64x4*>(part.last_acc + tile * D + gl * 4) = tot;
        if (gl == 0) {
          part.last_cc[tile] = tcc;
          part.last_ww[tile] = tww;
          // one lane per tile: the fixup pass takes the tiles from this list,
          // with the segment and the last tile it covers
          const uint32_t seg = s_seg[G - 1];
          int64_t end = (int64_t)seg + 1 <= n ? (int64_t)seg_start[seg + 1] : n;   // written by the position pass
          end = end < 1 ? 1 : (end > n ? n : end);
          part.fix_list[atomicAdd(part.fix_count, 1u)] =
              u32x4{(uint32_t)tile, seg, (uint32_t)((end - 1) / TILE), hb};
        }
      }
    }
  }
}

// Joins, for each segment that runs past the end of the tile holding its
// head, the partial sums of every later tile it covers.  Only the tiles the
// row pass listed are visited (about a third of them for Zipf IDs), spread
// over a fixed grid.  A lane group takes one listed tile whose segment covers
// at most kFixShort (and at most 256/LPR) later tiles, which is nearly all of
// them (the hot IDs have their own pass), with all its loads in flight at
// once; a longer chain (some 1700 tiles for the hottest ID at 65M positions
// without the hot-key plan) is summed by the whole block, 256/LPR groups with
// eight loads in flight each.  Both add the tail of the first tile, then the
// later tiles' partials in tile order.
constexpr int kFixBlock = 256;
constexpr int64_t kFixGrid = 2048;
constexpr int kFixShort = 8;
template <int LPR>
__global__ void __launch_bounds__(kFixBlock)
seg_fixup_kernel(SegmentArgs a, SegPartials part) {
  constexpr int G = kFixBlock / LPR;
  // a chain of at most G later tiles is summed in the same order by both paths
  constexpr int kShort = kFixShort < G ? kFixShort : G;
  __shared__ f64x4 s_acc[kFixBlock];
  __shared__ int32_t s_cc[G], s_ww[G];
  __shared__ uint32_t s_long[G];
  __shared__ uint32_t s_nlong;
  const int lane = threadIdx.x % LPR;
  const int grp = threadIdx.x / LPR;
  const bool lane_on = lane * 4 < a.D;
  const int D = a.D;
  const uint32_t count = *part.fix_count;
  // the listed tiles in any order: each one's sum is taken in a fixed order
  for (uint32_t k0 = blockIdx.x * (uint32_t)G; k0 < count; k0 += gridDim.x * (uint32_t)G) {
    if (threadIdx.x == 0) s_nlong = 0u;
    __syncthreads();
    const uint32_t k = k0 + grp;
    if (k < count) {
      const u32x4 rec = part.fix_list[k];
      const int64_t b = rec.x, seg = rec.y, b_end = rec.z, hb = rec.w;   // hb: hot IDs before it (split plan)
      if (seg < a.N) {   // always true when the numbering is consistent
        if (b_end - b <= kShort) {
          f64x4 v[kShort];
          int32_t c[kShort], ww[kShort];
#pragma unroll
          for (int u = 0; u < kShort; ++u) {
            const int64_t bb = b + 1 + u;
            const int64_t bc = bb <= b_end ? bb : b;   // clamped: read, then ignored
            v[u] = lane_on ? *reinterpret_cast<const f64x4*>(part.first_acc + bc * D + lane * 4)
                           : f64x4{0.0, 0.0, 0.0, 0.0};
            c[u] = part.first_cc[bc];
            ww[u] = part.first_ww[bc];
          }
          f64x4 tot = lane_on ? *reinterpret_cast<const f64x4*>(part.last_acc + b * D + lane * 4)
                              : f64x4{0.0, 0.0, 0.0, 0.0};
          int tcc = part.last_cc[b], tww = part.last_ww[b];
#pragma unroll
          for (int u = 0; u < kShort; ++u) {
            if (b + 1 + u > b_end) break;
            tot += v[u];
            tcc += c[u];
            tww += ww[u];
          }
          finalize_segment(a, seg + hb, tot, tcc, tww, lane, lane_on, a.ap.mode);
        } else if (lane == 0) {
          s_long[atomicAdd(&s_nlong, 1u)] = k;
        }
      }
    }
    __syncthreads();
    const uint32_t nlong = s_nlong;
    for (uint32_t i = 0; i < nlong; ++i) {
      const u32x4 rec = part.fix_list[s_long[i]];
      const int64_t b = rec.x, seg = rec.y, b_end = rec.z, hb = rec.w;
      f64x4 acc = {0.0, 0.0, 0.0, 0.0};
      int cc = 0, ww = 0;
#pragma unroll 8
      for (int64_t bb = b + 1 + grp; bb <= b_end; bb += G) {
        if (lane_on) acc += *reinterpret_cast<const f64x4*>(part.first_acc + bb * D + lane * 4);
        cc += part.first_cc[bb];
        ww += part.first_ww[bb];
      }
      s_acc[threadIdx.x] = acc;
      if (lane == 0) {
        s_cc[grp] = cc;
        s_ww[grp] = ww;
      }
      __syncthreads();
      if (grp == 0) {
        f64x4 tot = lane_on ? *reinterpret_cast<const f64x4*>(part.last_acc + b * D + lane * 4)
                            : f64x4{0.0, 0.0, 0.0, 0.0};
        int tcc = part.last_cc[b], tww = part.last_ww[b];
        for (int g = 0; g < G; ++g) {
          tot += s_acc[g * LPR + lane];
          tcc += s_cc[g];
          tww += s_ww[g];
        }
        finalize_segment(a, seg + hb, tot, tcc, tww, lane, lane_on, a.ap.mode);
      }
      __syncthreads();   // s_acc is rewritten for the next long chain
    }
  }
}

// ------------------------------------------------------------ hot IDs (split plan)
// Each hot ID's occurrences are one segment, split into chunks of kGroupSpan
// occurrences per lane group, TILE per block.  The chunk prefix of the runs is
// rebuilt by every block from the hot occurrence counts.
struct HotPartials {
  double* acc;     // [chunks][D] float64 sums of the weighted rows
  int32_t* cnt;    // [chunks][4]: contributions, active contributions, first and last contribution
  uint32_t* cp;    // [H + 1] first chunk of each hot ID's run (written by block 0 of hot_rows)
};

// Weight of contribution m for the row with tag `tg` (per-ID mode) or its
// token weight, from the LDS tables.
__device__ __forceinline__ float row_weight(const SegmentArgs& a, const float* s_w, const int32_t* s_sm, int m,
                                           int64_t tg) {
  if (a.decay == GBA_DECAY_TOKEN) return s_w[m];
  int64_t st = tg - a.step + (int64_t)s_sm[m] + 1;
  st = st < 0 ? 0 : st;
  return st <= a.iota ? 1.0f : 0.0f;
}

template <int LPR>
__global__ void __launch_bounds__(kSegBlock)
hot_rows_kernel(SegmentArgs a, const int32_t* __restrict__ buckets, int q, int nbuckets, HotPartials hp) {
  constexpr int GW = kWave / LPR;            // groups per wave
  constexpr int G = kSegWaves * GW;          // groups per block
  constexpr int64_t TILE = (int64_t)G * kGroupSpan;
  extern __shared__ int32_t s_dyn[];
  __shared__ uint32_t s_cp[kHotSlots + 1];
  __shared__ uint32_t s_tmp[kSegWaves + 1];
  __shared__ f64x4 s_acc[kSegBlock];
  __shared__ int32_t s_c[G], s_a[G], s_first[G], s_last[G];
  const int K = a.K;
  const int D = a.D;
  int32_t* s_off = s_dyn;
  float* s_w = reinterpret_cast<float*>(s_dyn + K + 1);
  int32_t* s_sm = s_dyn + 2 * K + 1;
  int32_t* s_bucket = s_dyn + 3 * K + 1;
  const uint32_t H = *a.hot.meta;
  const int t = threadIdx.x;
  // chunks of every hot ID's run, and their prefix
  uint32_t nch = 0;
  if ((uint32_t)t < H) nch = (uint32_t)((a.hot.prefix[t + 1] - a.hot.prefix[t] + TILE - 1) / TILE);
  uint32_t total;
  const uint32_t ex = block_exclusive_scan<kSegBlock>(nch, s_tmp, &total);
  if ((uint32_t)t < H) s_cp[t] = ex;
  if (t == 0) s_cp[H] = total;
  if (blockIdx.x == 0) {
    if ((uint32_t)t < H) hp.cp[t] = ex;
    if (t == 0) hp.cp[H] = total;
  }
  const uint32_t b = blockIdx.x;
  if (b >= total) return;   // block-uniform; the grid is sized for the most chunks
  load_contrib_tables(a, buckets, nbuckets, s_off, s_w, s_sm, s_bucket);
  __syncthreads();
  // the run holding chunk b: the last h with s_cp[h] <= b
  uint32_t h = count_at_most(s_cp, H, (int64_t)b) - 1;
  const int64_t run_end = a.hot.prefix[h + 1];
  const int64_t c0 = (int64_t)a.hot.prefix[h] + (int64_t)(b - s_cp[h]) * TILE;
  const int64_t key = a.hot.ids[h];
  const int64_t tg = (a.decay == GBA_DECAY_ID_TAG && key < a.R) ? (int64_t)a.tag[key] : -1;

  const int w = t / kWave;
  const int lane = lane_id();
  const int gl = lane % LPR;
  const int grp = w * GW + lane / LPR;
  const bool lane_on = gl * 4 < D;
  const int64_t p0 = c0 + (int64_t)grp * kGroupSpan;
  const int64_t left = (p0 < run_end) ? run_end - p0 : 0;
  const int nvalid = left >= kGroupSpan ? kGroupSpan : (int)left;
  f64x4 acc = {0.0, 0.0, 0.0, 0.0};
  int cg = 0, ag = 0, first = -1, last = -1;
  for (int i0 = 0; i0 < nvalid; i0 += kBatch) {
    // the lanes of a group read the same indices (clamped into the run)
    uint32_t j[kBatch];
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      const int64_t pi = p0 + i0 + u;
      j[u] = a.hot.hot_vals[pi < run_end ? pi : run_end - 1];
    }
    int m[kBatch];
    float wt[kBatch];
    f32x4 rv[kBatch];
    uint32_t use = 0;
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      const bool valid = i0 + u < nvalid && (int64_t)j[u] < a.N;
      m[u] = valid ? contribution_of(s_off, s_bucket, q, K, j[u]) : 0;
      wt[u] = valid ? row_weight(a, s_w, s_sm, m[u], tg) : 0.0f;
      const bool on = valid && wt[u] != 0.0f && lane_on;
      use |= on ? (1u << u) : 0u;
      rv[u] = *reinterpret_cast<const f32x4*>(a.rows + (on ? (int64_t)j[u] * D + gl * 4 : 0));
    }
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      __builtin_amdgcn_sched_barrier(0);
      if (i0 + u < nvalid) {
        if ((use >> u) & 1u) acc = fma_widen((double)wt[u], rv[u], acc);
        const bool newc = m[u] != last;   // occurrences of one contribution are consecutive
        cg += newc ? 1 : 0;
        ag += (newc && wt[u] != 0.0f) ? 1 : 0;
        if (first < 0) first = m[u];
        last = m[u];
      }
    }
  }
  s_acc[t] = acc;
  if (gl == 0) {
    s_c[grp] = cg;
    s_a[grp] = ag;
    s_first[grp] = first;
    s_last[grp] = last;
  }
  __syncthreads();
  if (grp == 0) {
    // groups in order; a contribution that runs across two groups counts once
    f64x4 tot = {0.0, 0.0, 0.0, 0.0};
    int C = 0, A = 0, f = -1, l = -1;
    for (int g = 0; g < G; ++g) {
      if (s_first[g] < 0) continue;   // an empty group (past the end of the run)
      tot += s_acc[g * LPR + gl];
      C += s_c[g];
      A += s_a[g];
      if (s_first[g] == l) {
        C -= 1;
        if (row_weight(a, s_w, s_sm, l, tg) != 0.0f) A -= 1;
      }
      if (f < 0) f = s_first[g];
      l = s_last[g];
    }
    if (lane_on) *reinterpret_cast<f64x4*>(hp.acc + (int64_t)b * D + gl * 4) = tot;
    if (gl == 0) {
      int32_t* c = hp.cnt + (int64_t)b * 4;
      c[0] = C;
      c[1] = A;
      c[2] = f;
      c[3] = l;
    }
  }
}

// One block per hot ID: joins the chunks of its run in a fixed order and
// writes its place among all IDs (after the cold segments below it, cnum),
// its start (the cold occurrences below it plus the hot ones before it), c_r,
// W_r and the weighted sum divided by c_r (or K).  From 2^25 occurrences the
// blocks have 1024 threads (the hottest ID then has some 1,800 chunks, joined
// by 128 lane groups), below that 256.
template <int LPR, int BLOCK>
__global__ void __launch_bounds__(BLOCK)
hot_finish_kernel(SegmentArgs a, HotPartials hp, const uint32_t* __restrict__ cnum,
                  const uint32_t* __restrict__ cold_below) {
  constexpr int G = BLOCK / LPR;
  __shared__ f64x4 s_acc[BLOCK];
  __shared__ int32_t s_c[G], s_a[G];
  const uint32_t H = *a.hot.meta;
  const uint32_t h = blockIdx.x;
  if (h >= H) return;
  const int D = a.D;
  const int t = threadIdx.x;
  const int lane = t % LPR;
  const int grp = t / LPR;
  const bool lane_on = lane * 4 < D;
  const int64_t key = a.hot.ids[h];
  const int64_t tg = (a.decay == GBA_DECAY_ID_TAG && key < a.R) ? (int64_t)a.tag[key] : -1;
  // cold occurrences below the hot ID (found by the position pass)
  const uint32_t below_all = cold_below[h];
  const uint32_t b0 = hp.cp[h], b1 = hp.cp[h + 1];
  f64x4 acc = {0.0, 0.0, 0.0, 0.0};
  int C = 0, A = 0;
  // group grp takes chunks b0 + grp, b0 + grp + G, ... in that order, eight
  // loads in flight at a time
  constexpr int kFin = 8;
  for (uint32_t base = b0 + grp; base < b1; base += kFin * G) {
    f64x4 v[kFin];
    int32_t c0[kFin], c1[kFin], c2[kFin], prev_last[kFin];
#pragma unroll
    for (int u = 0; u < kFin; ++u) {
      const uint32_t bb = base + u * G;
      const uint32_t bc = bb < b1 ? bb : b1 - 1;   // clamped: read, then ignored
      v[u] = lane_on ? *reinterpret_cast<const f64x4*>(hp.acc + (int64_t)bc * D + lane * 4)
                     : f64x4{0.0, 0.0, 0.0, 0.0};
      const int32_t* c = hp.cnt + (int64_t)bc * 4;
      c0[u] = c[0];
      c1[u] = c[1];
      c2[u] = c[2];
      prev_last[u] = bc > b0 ? hp.cnt[(int64_t)(bc - 1) * 4 + 3] : -1;
    }
#pragma unroll
    for (int u = 0; u < kFin; ++u) {
      if (base + u * G >= b1) break;
      acc += v[u];
      C += c0[u];
      A += c1[u];
      if (c2[u] == prev_last[u]) {   // a contribution across two chunks counts once
        C -= 1;
        const int m = c2[u];
        float wm;
        if (a.decay == GBA_DECAY_TOKEN) {
          wm = a.w[m];
        } else {
          int64_t st = tg - a.tokens[m] + 1;
          st = st < 0 ? 0 : st;
          wm = st <= a.iota ? 1.0f : 0.0f;
        }
        if (wm != 0.0f) A -= 1;
      }
    }
  }
  s_acc[t] = acc;
  if (lane == 0) {
    s_c[grp] = C;
    s_a[grp] = A;
  }
  __syncthreads();
  if (grp == 0) {
    f64x4 tot = {0.0, 0.0, 0.0, 0.0};
    int tc = 0, ta = 0;
    for (int g = 0; g < G; ++g) {
      tot += s_acc[g * LPR + lane];
      tc += s_c[g];
      ta += s_a[g];
    }
    const int64_t out = (int64_t)h + cnum[h];
    if (out < a.N) {   // always true when the numbering is consistent
      finalize_segment(a, out, tot, tc, ta, lane, lane_on, a.ap.mode, (int64_t)key);
      if (lane == 0) {
        a.unique_ids[out] = key;
        a.seg_offsets[out] = (int64_t)below_all + a.hot.prefix[h];
      }
    }
  }
}

// Per-ID decay: every row with a non-zero weight now carries the current step.
__global__ void __launch_bounds__(kSegBlock)
tag_update_kernel(const int64_t* __restrict__ unique_ids, const int32_t* __restrict__ active_count,
                  const int64_t* __restrict__ num_unique, int32_t* __restrict__ tag, int32_t step) {
  const int64_t U = *num_unique;
  const int64_t stride = (int64_t)gridDim.x * kSegBlock;
  for (int64_t s = (int64_t)blockIdx.x * kSegBlock + threadIdx.x; s < U; s += stride)
    if (active_count[s] > 0) tag[unique_ids[s]] = step;
}

size_t run_heads_workspace_bytes(int64_t N) {
  return scan_workspace_bytes(N > 0 ? ceil_div(N, kMetaTile) : 1);
}

hipError_t launch_run_heads(const uint32_t* keys, int64_t N, uint32_t* tile_base, uint32_t* total, void* scan_ws,
                            hipStream_t stream, const uint32_t* n_dev) {
  const int64_t tiles = N > 0 ? ceil_div(N, kMetaTile) : 0;
  if (N > 0) {
    hipLaunchKernelGGL(seg_heads_kernel, dim3((unsigned)ceil_div(tiles, kSegWaves)), dim3(kSegBlock), 0, stream,
                       keys, N, n_dev, tiles, tile_base);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return launch_exclusive_scan_u32(tile_base, tile_base, tiles, total, scan_ws, stream);
}

template <int LPR>
static hipError_t launch_rows(const SegmentArgs& a, const uint32_t* packed, const uint32_t* base32,
                              SegPartials part, const uint32_t* seg_start, const uint32_t* cnum, HotPartials hp,
                              const int32_t* buckets, int q, int nb, const SegLayout& L, hipStream_t stream) {
  const int64_t tiles = L.row_tiles;
  const dim3 grid((unsigned)tiles), block(kSegBlock);
  if (a.ap.mode != 0 && !segments_fuse_apply(a.D, a.ap.mode)) return hipErrorInvalidValue;   // the caller applies
  const int span = rows_span(a.N);   // the layout's tiles were sized with the same span
#define GBA_ROWS_SPAN(AP, SP) \
  hipLaunchKernelGGL((seg_rows_kernel<LPR, AP, SP>), grid, block, 0, stream, a, packed, base32, part, seg_start, cnum)
#define GBA_ROWS_SPANS(AP)                 \
  if (span == 128) GBA_ROWS_SPAN(AP, 128); \
  else if (span == 64) GBA_ROWS_SPAN(AP, 64); \
  else GBA_ROWS_SPAN(AP, 32);
  if constexpr (LPR == 8) {
    if (a.ap.mode == 1) {
      GBA_ROWS_SPANS(1)
    } else {
      GBA_ROWS_SPANS(0)
    }
  } else {
    GBA_ROWS_SPANS(0)
  }
#undef GBA_ROWS_SPANS
#undef GBA_ROWS_SPAN
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  // the listed tiles (at most all of them) are spread over a fixed grid
  const int64_t fix_blocks = tiles < kFixGrid ? tiles : kFixGrid;
  hipLaunchKernelGGL(seg_fixup_kernel<LPR>, dim3((unsigned)fix_blocks), dim3(kFixBlock), 0, stream, a, part);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if (a.n_dev) {
    const size_t lds = (size_t)(3 * a.K + 1 + nb) * sizeof(int32_t);
    hipLaunchKernelGGL(hot_rows_kernel<LPR>, dim3((unsigned)L.hot_chunks), dim3(kSegBlock), lds, stream, a, buckets,
                       q, nb, hp);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if (a.N >= (int64_t(1) << 25))
      hipLaunchKernelGGL((hot_finish_kernel<LPR, 1024>), dim3(kHotSlots), dim3(1024), 0, stream, a, hp, cnum,
                         cnum + 2 * (kHotSlots + 1));
    else
      hipLaunchKernelGGL((hot_finish_kernel<LPR, 256>), dim3(kHotSlots), dim3(256), 0, stream, a, hp, cnum,
                         cnum + 2 * (kHotSlots + 1));
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  return hipSuccess;
}

bool segments_fuse_apply(int32_t D, int mode) { return mode == 1 && lanes_per_row(D) == 8; }

hipError_t launch_segments(const SegmentArgs& a, void* ws, hipStream_t stream) {
  const SegLayout L = seg_layout(a.N, a.D);
  char* base = static_cast<char*>(ws);
  uint32_t* heads = reinterpret_cast<uint32_t*>(base + L.off_heads);
  uint32_t* total = reinterpret_cast<uint32_t*>(base + L.off_total);
  void* scan_ws = base + L.off_scan;
  int32_t* buckets = reinterpret_cast<int32_t*>(base + L.off_buckets);
  uint32_t* packed = reinterpret_cast<uint32_t*>(base + L.off_packed);
  uint32_t* base32 = reinterpret_cast<uint32_t*>(base + L.off_base32);
  SegPartials part;
  int32_t* cnt = reinterpret_cast<int32_t*>(base + L.off_cnt);
  part.first_cc = cnt;
  part.first_ww = cnt + L.row_tiles;
  part.last_cc = cnt + 2 * L.row_tiles;
  part.last_ww = cnt + 3 * L.row_tiles;
  part.first_acc = reinterpret_cast<double*>(base + L.off_first_acc);
  part.last_acc = reinterpret_cast<double*>(base + L.off_last_acc);
  part.fix_count = reinterpret_cast<uint32_t*>(base + L.off_fix);
  part.fix_list = reinterpret_cast<u32x4*>(base + L.off_fix + 256);
  uint32_t* seg_start = reinterpret_cast<uint32_t*>(base + L.off_start);
  uint32_t* cnum = reinterpret_cast<uint32_t*>(base + L.off_cnum);
  HotPartials hp;
  hp.acc = reinterpret_cast<double*>(base + L.off_hot_acc);
  hp.cnt = reinterpret_cast<int32_t*>(base + L.off_hot_cnt);
  hp.cp = cnum + kHotSlots + 1;
  uint32_t* cold_below = cnum + 2 * (kHotSlots + 1);

  hipLaunchKernelGGL(check_offsets_kernel, dim3(1), dim3(256), 0, stream, a.offsets, a.K, a.N, a.err);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  e = launch_run_heads(a.keys, a.N, heads, total, scan_ws, stream, a.n_dev);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(seg_finish_kernel, dim3(1), dim3(kSegBlock), 0, stream, a, (const uint32_t*)total, seg_start,
                     cnum, cold_below, part.fix_count);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if (a.N <= 0) return hipSuccess;

  const int q = bucket_shift(a.N);
  const int nb = (int)(((a.N - 1) >> q) + 1);
  hipLaunchKernelGGL(contrib_buckets_kernel, dim3(1), dim3(256), 0, stream, a.offsets, a.K, a.N, q, nb,
                     buckets);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  const size_t lds = (size_t)(3 * a.K + 1 + nb) * sizeof(int32_t);
  hipLaunchKernelGGL(seg_meta_kernel, dim3((unsigned)ceil_div(L.meta_tiles, kMetaTilesPerBlock)),
                     dim3(kSegBlock), lds, stream, a, (const uint32_t*)heads, (const int32_t*)buckets, q, nb,
                     L.meta_tiles, packed, base32, seg_start, cnum, cold_below);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  switch (lanes_per_row(a.D)) {
    case 1: e = launch_rows<1>(a, packed, base32, part, seg_start, cnum, hp, buckets, q, nb, L, stream); break;
    case 2: e = launch_rows<2>(a, packed, base32, part, seg_start, cnum, hp, buckets, q, nb, L, stream); break;
    case 4: e = launch_rows<4>(a, packed, base32, part, seg_start, cnum, hp, buckets, q, nb, L, stream); break;
    case 8: e = launch_rows<8>(a, packed, base32, part, seg_start, cnum, hp, buckets, q, nb, L, stream); break;
    case 16: e = launch_rows<16>(a, packed, base32, part, seg_start, cnum, hp, buckets, q, nb, L, stream); break;
    case 32: e = launch_rows<32>(a, packed, base32, part, seg_start, cnum, hp, buckets, q, nb, L, stream); break;
    case 64: e = launch_rows<64>(a, packed, base32, part, seg_start, cnum, hp, buckets, q, nb, L, stream); break;
    default: return hipErrorInvalidValue;
  }
  if (e != hipSuccess) return e;
  if (a.decay == GBA_DECAY_ID_TAG) {
    int64_t blocks = ceil_div(a.N, kSegBlock);
    if (blocks > 4096) blocks = 4096;
    hipLaunchKernelGGL(tag_update_kernel, dim3((unsigned)blocks), dim3(kSegBlock), 0, stream,
                       (const int64_t*)a.unique_ids, (const int32_t*)a.active_count,
                       (const int64_t*)a.num_unique, a.tag, (int32_t)a.step);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace gba
