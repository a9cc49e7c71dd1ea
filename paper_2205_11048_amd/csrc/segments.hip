// Embedding gradients by ID (Alg. 2, push responder): after the occurrences
// are sorted by ID, every run of equal IDs is one segment.  For each segment
// this computes its ID and start (dedup), c_r (number of contributions that
// hold the ID: the divisor "number of workers that encountered the ID"),
// W_r (contributions whose weight for the ID is non-zero), and the weighted
// sum of the rows divided by c_r (or by K).  The weight of a contribution for
// a row is its token weight, or in per-ID mode [max(0, tag[r] - tau_m + 1) <=
// iota] with the tag as it was before this step.
//
// Work is split by sorted position, not by segment, so a Zipf-hot ID with
// millions of occurrences is spread over many blocks and no floating-point
// atomics are used.  A persistent block walks tiles of 1024 sorted positions.
// First every lane takes one position at a time (coalesced key and index
// loads): it finds the contribution of the occurrence through a bucket table
// in LDS, its weight, and whether it starts a run of equal IDs or a new
// contribution inside one; ballots turn these into bit masks in LDS.  Then a
// group of LPR lanes (one 16-byte column slice per lane) walks 256 / (64 /
// LPR) consecutive positions, keeping 8 row gathers in flight and summing
// each run in float64.  Runs that cross group boundaries are joined in LDS;
// runs that cross tile boundaries leave one partial per tile end, joined by a
// second launch in a fixed order, so results are deterministic.
#include "gba_device.hpp"
#include "gba_internal.hpp"

namespace gba {

constexpr int kSegBlock = 256;
constexpr int kSegWaves = kSegBlock / kWave;                 // 4
constexpr int kWaveSpan = 256;                               // positions per wave per tile
constexpr int kRounds = kWaveSpan / kWave;                   // 4
constexpr int64_t kSegTile = (int64_t)kSegWaves * kWaveSpan; // 1024 positions per tile
constexpr int kTileWords = (int)(kSegTile / 32);             // bit-mask words per tile
constexpr int kBatch = 8;                                    // row gathers in flight per group
static_assert(32 % kBatch == 0 && kBatch < 32, "a batch must not straddle a mask word");
constexpr int kMaxBuckets = 1024;                            // contribution lookup buckets

enum : uint32_t { kValid = 1, kOpen = 2, kPass = 4 };            // group flags
enum : uint32_t { kHasFirst = 1, kHasLast = 2, kBlockPass = 4 }; // tile flags

static inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }
static inline size_t align_up(size_t x) { return (x + 255) & ~size_t(255); }

static int lanes_per_row(int D) {
  int l = 1;
  while (l < 64 && l * 4 < D) l <<= 1;
  return l;
}

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
  uint32_t* last_seg;
  uint32_t* flags;
};

struct SegLayout {
  int64_t tiles;
  size_t off_heads, off_total, off_scan, off_buckets, off_flags, off_last_seg, off_cnt,
      off_first_acc, off_last_acc, bytes;
};

static SegLayout seg_layout(int64_t N, int32_t D) {
  SegLayout L{};
  L.tiles = N > 0 ? ceil_div(N, kSegTile) : 1;
  const size_t nt = (size_t)L.tiles;
  size_t o = 0;
  L.off_heads = o;     o += align_up(nt * 4);
  L.off_total = o;     o += 256;
  L.off_scan = o;      o += align_up(scan_workspace_bytes(L.tiles));
  L.off_buckets = o;   o += align_up(kMaxBuckets * 4);
  L.off_flags = o;     o += align_up(nt * 4);
  L.off_last_seg = o;  o += align_up(nt * 4);
  L.off_cnt = o;       o += align_up(nt * 16);
  L.off_first_acc = o; o += align_up(nt * (size_t)D * 8);
  L.off_last_acc = o;  o += align_up(nt * (size_t)D * 8);
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

__device__ __forceinline__ void finalize_segment(const SegmentArgs& a, int64_t seg, f64x4 acc,
                                                 int cc, int ww, int lane, bool lane_on) {
  if (seg < 0 || seg >= a.N) return;   // unreachable when the numbering is consistent
  const double div = (a.norm == GBA_NORM_BY_K) ? (double)a.K : (double)cc;
  if (lane_on)
    *reinterpret_cast<f32x4*>(a.agg + seg * (int64_t)a.D + lane * 4) = narrow(acc / div);
  if (lane == 0) {
    a.contrib_count[seg] = cc;
    a.active_count[seg] = ww;
  }
}

// popcount of bits [lo, hi) of a 256-bit mask held as four words
__device__ __forceinline__ int popc_range(const uint64_t* m, int lo, int hi) {
  int c = 0;
#pragma unroll
  for (int r = 0; r < kRounds; ++r) {
    const int a = lo > r * 64 ? lo - r * 64 : 0;
    const int b = hi < (r + 1) * 64 ? hi - r * 64 : 64;
    if (a < b) {
      const uint64_t hi_mask = b == 64 ? ~0ull : ((1ull << b) - 1);
      const uint64_t lo_mask = ~((1ull << a) - 1);
      c += __popcll(m[r] & hi_mask & lo_mask);
    }
  }
  return c;
}

// ------------------------------------------------------------------ kernels
__global__ void check_offsets_kernel(const int64_t* __restrict__ off, int K, int64_t N,
                                     int32_t* __restrict__ err) {
  bool bad = false;
  for (int m = threadIdx.x; m < K; m += blockDim.x) bad |= off[m] > off[m + 1];
  if (threadIdx.x == 0) bad |= (off[0] != 0) || (off[K] != N);
  if (bad) raise_error(err, GBA_DERR_OFFSETS);
}

// bucket[b] = contribution of occurrence b << q
__global__ void contrib_buckets_kernel(const int64_t* __restrict__ off, int K, int64_t N, int q,
                                       int nb, int32_t* __restrict__ bucket,
                                       uint32_t* __restrict__ tile_ctr) {
  if (threadIdx.x == 0) *tile_ctr = 0u;   // the reduction's tile counter starts at zero
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

__global__ void __launch_bounds__(kSegBlock)
seg_heads_kernel(const uint32_t* __restrict__ keys, int64_t N, uint32_t* __restrict__ heads) {
  __shared__ uint32_t tmp[kSegBlock / kWave + 1];
  const int64_t t0 = (int64_t)blockIdx.x * kSegTile;
  const int64_t t1 = (t0 + kSegTile < N) ? t0 + kSegTile : N;
  uint32_t c = 0;
  for (int64_t p = t0 + threadIdx.x; p < t1; p += kSegBlock) c += (p == 0 || keys[p] != keys[p - 1]);
  uint32_t total;
  block_exclusive_scan<kSegBlock>(c, tmp, &total);
  if (threadIdx.x == 0) heads[blockIdx.x] = total;
}

__global__ void seg_finish_kernel(const uint32_t* __restrict__ total, int64_t N,
                                  int64_t* __restrict__ num_unique, int64_t* __restrict__ seg_offsets) {
  const uint32_t U = *total;
  *num_unique = (int64_t)U;
  seg_offsets[U] = N;
}

// LDS index with one pad word per 32, so lane groups reading entries 32 apart
// hit different banks.
__host__ __device__ constexpr int pad(int i) { return i + (i >> 5); }

template <int LPR>
__global__ void __launch_bounds__(kSegBlock)
seg_reduce_kernel(SegmentArgs a, const uint32_t* __restrict__ tile_seg_base,
                  const int32_t* __restrict__ buckets, int q, int nbuckets, int64_t num_tiles,
                  uint32_t* __restrict__ tile_ctr, SegPartials part) {
  constexpr int GW = kWave / LPR;            // groups per wave
  constexpr int G = kSegWaves * GW;          // groups per block
  constexpr int PG = kWaveSpan / GW;         // positions per group
  extern __shared__ int32_t s_dyn[];
  __shared__ uint32_t s_j[pad((int)kSegTile)];
  __shared__ float s_wt[pad((int)kSegTile)];
  __shared__ uint32_t s_hb[kTileWords + 1];  // run heads (+ first position of the next tile)
  __shared__ uint32_t s_nb[kTileWords];      // first occurrence of a contribution in a run
  __shared__ uint32_t s_gb[G];               // segment number of each group's first head, in tile
  __shared__ f64x4 s_acc[kSegBlock];
  __shared__ int32_t s_cc[G], s_ww[G];
  __shared__ uint32_t s_seg[G], s_flags[G];
  __shared__ uint32_t s_tmp[kSegBlock / kWave + 1];
  __shared__ uint32_t s_bflags;
  __shared__ uint32_t s_next;

  const int K = a.K;
  const int64_t N = a.N;
  int32_t* s_off = s_dyn;                    // [K + 1]
  float* s_w = reinterpret_cast<float*>(s_dyn + K + 1);      // [K]
  int32_t* s_sm = s_dyn + 2 * K + 1;         // [K] staleness step - tau_m (per-ID decay)
  int32_t* s_bucket = s_dyn + 3 * K + 1;     // [nbuckets]
  for (int i = threadIdx.x; i <= K; i += kSegBlock) {
    int64_t o = a.offsets[i];
    o = o < 0 ? 0 : (o > N ? N : o);
    s_off[i] = (int32_t)o;
    if (i < K) {
      s_w[i] = a.w[i];
      int64_t sm = a.step - a.tokens[i];
      sm = sm < -(1 << 30) ? -(1 << 30) : (sm > (1 << 30) ? (1 << 30) : sm);
      s_sm[i] = (int32_t)sm;
    }
  }
  for (int i = threadIdx.x; i < nbuckets; i += kSegBlock) s_bucket[i] = buckets[i];
  __syncthreads();

  const int w = threadIdx.x / kWave;
  const int lane = lane_id();
  const int gl = lane % LPR;                 // lane inside its group
  const int gw = lane / LPR;                 // group inside the wave
  const int grp = w * GW + gw;               // group inside the block
  const bool lane_on = gl * 4 < a.D;
  const int D = a.D;

  // Tiles are taken from a counter, so blocks that become resident late (the
  // GPU may be shared with another stream's kernels) simply take fewer.
  if (threadIdx.x == 0) s_next = atomicAdd(tile_ctr, 1u);
  __syncthreads();
  for (int64_t tile = s_next; tile < num_tiles; tile = s_next) {
    const int64_t tile0 = tile * kSegTile;
    if (threadIdx.x == 0) {
      s_bflags = 0;
      const int64_t nx = tile0 + kSegTile;
      s_hb[kTileWords] = (nx < N) ? (a.keys[nx] != a.keys[nx - 1] ? 1u : 0u) : 1u;
    }

    // ---- per-position pass: contribution, weight, run and contribution starts
    const int64_t pw = tile0 + (int64_t)w * kWaveSpan;
    uint32_t carry_key = 0;
    int carry_m = -1;
    bool carry_ok = false;
    if (pw > 0 && pw < N) {
      carry_key = a.keys[pw - 1];
      const uint32_t jp = a.vals[pw - 1];
      carry_m = (int64_t)jp < N ? contribution_of(s_off, s_bucket, q, K, jp) : 0;
      carry_ok = true;
    }
    uint64_t hm[kRounds], nm[kRounds];
#pragma unroll
    for (int r = 0; r < kRounds; ++r) {
      const int64_t p = pw + r * kWave + lane;
      const bool valid = p < N;
      const uint32_t key = valid ? a.keys[p] : 0u;
      const uint32_t jv = valid ? a.vals[p] : 0u;
      const int m = (valid && (int64_t)jv < N) ? contribution_of(s_off, s_bucket, q, K, jv) : 0;
      uint32_t kp = __shfl_up(key, 1, kWave);
      int mp = __shfl_up(m, 1, kWave);
      bool prev_ok = true;
      if (lane == 0) {
        kp = carry_key;
        mp = carry_m;
        prev_ok = carry_ok;
      }
      const bool head = valid && (!prev_ok || key != kp);
      const bool newc = valid && (head || m != mp);
      float wt = 0.0f;
      if (valid) {
        if (a.decay == GBA_DECAY_TOKEN) {
          wt = s_w[m];
        } else {
          const int64_t tg = ((int64_t)key < a.R) ? (int64_t)a.tag[key] : -1;
          int64_t s = tg - a.step + (int64_t)s_sm[m] + 1;
          s = s < 0 ? 0 : s;
          wt = (s <= a.iota) ? 1.0f : 0.0f;
        }
      }
      const int pos = w * kWaveSpan + r * kWave + lane;
      s_j[pad(pos)] = jv;
      s_wt[pad(pos)] = wt;
      hm[r] = __ballot(head);
      nm[r] = __ballot(newc);
      carry_key = __shfl(key, kWave - 1, kWave);
      carry_m = __shfl(m, kWave - 1, kWave);
      carry_ok = (pw + r * kWave + kWave - 1) < N;
    }
#pragma unroll
    for (int r = 0; r < kRounds; ++r) {
      if (lane == 0) {
        s_hb[(w * kWaveSpan + r * kWave) / 32] = (uint32_t)hm[r];
        s_hb[(w * kWaveSpan + r * kWave) / 32 + 1] = (uint32_t)(hm[r] >> 32);
        s_nb[(w * kWaveSpan + r * kWave) / 32] = (uint32_t)nm[r];
        s_nb[(w * kWaveSpan + r * kWave) / 32 + 1] = (uint32_t)(nm[r] >> 32);
      }
    }
    // heads per group, in group order
    uint32_t gcount = 0;
    if (lane < GW) gcount = (uint32_t)popc_range(hm, lane * PG, (lane + 1) * PG);
    if (lane < GW) s_gb[w * GW + lane] = gcount;
    __syncthreads();
    uint32_t tile_heads;
    const uint32_t gex = block_exclusive_scan<kSegBlock>(threadIdx.x < G ? s_gb[threadIdx.x] : 0u, s_tmp,
                                                         &tile_heads);
    if (threadIdx.x < G) s_gb[threadIdx.x] = gex;
    __syncthreads();
    const uint32_t seg_base = tile_seg_base[tile];

    // ids and starts of the segments whose head lies in this tile
    {
      uint32_t before = 0;
#pragma unroll
      for (int r = 0; r < kRounds; ++r) {
        if ((hm[r] >> lane) & 1ull) {
          const int64_t p = pw + r * kWave + lane;
          const int64_t seg = (int64_t)seg_base + s_gb[w * GW] + before +
                              __popcll(hm[r] & lanemask_lt());
          if (seg < N) {
            a.unique_ids[seg] = (int64_t)a.keys[p];
            a.seg_offsets[seg] = p;
          }
        }
        before += (uint32_t)__popcll(hm[r]);
      }
    }

    // ---- per-group pass: gather the kept rows and sum every run in float64
    const int gpos0 = w * kWaveSpan + gw * PG;     // first position of the group in the tile
    const int64_t p0 = tile0 + gpos0;
    const int nvalid = (N - p0) >= PG ? PG : (N - p0 > 0 ? (int)(N - p0) : 0);
    f64x4 acc = {0.0, 0.0, 0.0, 0.0};
    int cc = 0, ww = 0;
    int64_t seg = (int64_t)seg_base + s_gb[grp] - 1;
    const bool first_open = nvalid > 0 && !((s_hb[gpos0 >> 5] >> (gpos0 & 31)) & 1u);
    bool in_first = true;
    f64x4 facc = {0.0, 0.0, 0.0, 0.0};
    int fcc = 0, fww = 0;
    bool owner = false;
    for (int i0 = 0; i0 < nvalid; i0 += kBatch) {
      f32x4 rv[kBatch];
      float wv[kBatch];
#pragma unroll
      for (int u = 0; u < kBatch; ++u) {
        const int i = i0 + u;
        const bool ok = i < nvalid;
        const uint32_t jv = ok ? s_j[pad(gpos0 + i)] : 0u;
        wv[u] = ok ? s_wt[pad(gpos0 + i)] : 0.0f;
        rv[u] = f32x4{0.f, 0.f, 0.f, 0.f};
        if (ok && wv[u] != 0.0f && lane_on && (int64_t)jv < N)
          rv[u] = *reinterpret_cast<const f32x4*>(a.rows + (int64_t)jv * D + gl * 4);
      }
      const int b0 = gpos0 + i0;
      constexpr uint32_t kBatchMask = (1u << kBatch) - 1u;   // kBatch divides 32
      const uint32_t hb = (s_hb[b0 >> 5] >> (b0 & 31)) & kBatchMask;
      const uint32_t nb = (s_nb[b0 >> 5] >> (b0 & 31)) & kBatchMask;
#pragma unroll
      for (int u = 0; u < kBatch; ++u) {
        const int i = i0 + u;
        if (i < nvalid) {
          if ((hb >> u) & 1u) {
            if (i > 0) {
              if (in_first && first_open) {
                facc = acc; fcc = cc; fww = ww; owner = true;
              } else {
                finalize_segment(a, seg, acc, cc, ww, gl, lane_on);
              }
              in_first = false;
            }
            ++seg;
            acc = f64x4{0.0, 0.0, 0.0, 0.0};
            cc = ww = 0;
          }
          if (wv[u] != 0.0f) acc += (double)wv[u] * widen(rv[u]);
          const int nc = (nb >> u) & 1u;
          cc += nc;
          ww += (nc && wv[u] != 0.0f) ? 1 : 0;
        }
      }
    }

    bool last_open = false, pass = false;
    if (nvalid > 0) {
      const int nxt = gpos0 + PG;                      // next position, may be in the next tile
      last_open = nvalid == PG && (p0 + PG) < N && !((s_hb[nxt >> 5] >> (nxt & 31)) & 1u);
      if (last_open) {
        pass = in_first && first_open;
        s_acc[threadIdx.x] = acc;
        if (gl == 0) {
          s_cc[grp] = cc;
          s_ww[grp] = ww;
          s_seg[grp] = (uint32_t)seg;
        }
      } else if (in_first && first_open) {
        facc = acc; fcc = cc; fww = ww; owner = true;
      } else {
        finalize_segment(a, seg, acc, cc, ww, gl, lane_on);
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
        tot += s_acc[gg * LPR + gl];
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
          atomicOr(&s_bflags, kHasFirst);
        }
      } else {
        finalize_segment(a, (int64_t)seg_base + s_gb[grp] - 1, tot, tcc, tww, gl, lane_on);
      }
    }
    // the chain that runs into the next tile
    if (grp == G - 1 && (s_flags[G - 1] & kOpen)) {
      f64x4 tot = s_acc[(G - 1) * LPR + gl];
      int tcc = s_cc[G - 1], tww = s_ww[G - 1];
      int gg = G - 1;
      while (gg > 0 && (s_flags[gg] & kPass)) {
        --gg;
        tot += s_acc[gg * LPR + gl];
        tcc += s_cc[gg];
        tww += s_ww[gg];
      }
      if (s_flags[gg] & kPass) {   // the whole tile is inside one segment
        if (lane_on) *reinterpret_cast<f64x4*>(part.first_acc + tile * D + gl * 4) = tot;
        if (gl == 0) {
          part.first_cc[tile] = tcc;
          part.first_ww[tile] = tww;
          atomicOr(&s_bflags, kHasFirst | kBlockPass);
        }
      } else {
        if (lane_on) *reinterpret_cast<f64x4*>(part.last_acc + tile * D + gl * 4) = tot;
        if (gl == 0) {
          part.last_cc[tile] = tcc;
          part.last_ww[tile] = tww;
          part.last_seg[tile] = s_seg[G - 1];
          atomicOr(&s_bflags, kHasLast);
        }
      }
    }
    __syncthreads();
    if (threadIdx.x == 0) {
      part.flags[tile] = s_bflags;
      s_next = atomicAdd(tile_ctr, 1u);
    }
    __syncthreads();
  }
}

// Joins, for each segment that runs past the end of the tile holding its
// head, the partial sums of every later tile it covers.
template <int LPR>
__global__ void __launch_bounds__(kSegBlock)
seg_fixup_kernel(SegmentArgs a, SegPartials part) {
  constexpr int G = kSegBlock / LPR;
  __shared__ f64x4 s_acc[kSegBlock];
  __shared__ int32_t s_cc[G], s_ww[G];
  const int64_t b = blockIdx.x;
  if (!(part.flags[b] & kHasLast)) return;
  const int lane = threadIdx.x % LPR;
  const int grp = threadIdx.x / LPR;
  const bool lane_on = lane * 4 < a.D;
  const int D = a.D;
  const int64_t seg = (int64_t)part.last_seg[b];
  if (seg + 1 > a.N) return;   // unreachable when the numbering is consistent
  int64_t end = a.seg_offsets[seg + 1];
  end = end < 1 ? 1 : (end > a.N ? a.N : end);
  const int64_t b_end = (end - 1) / kSegTile;
  f64x4 acc = {0.0, 0.0, 0.0, 0.0};
  int cc = 0, ww = 0;
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
    finalize_segment(a, seg, tot, tcc, tww, lane, lane_on);
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

template <int LPR>
static hipError_t launch_reduce(const SegmentArgs& a, const uint32_t* tile_base, const int32_t* buckets,
                                int q, int nb, uint32_t* tile_ctr, SegPartials part, int64_t tiles,
                                hipStream_t stream) {
  const size_t lds = (size_t)(3 * a.K + 1 + nb) * sizeof(int32_t);
  int dev = 0, cus = 0, per_cu = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (e == hipSuccess)
    e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, seg_reduce_kernel<LPR>, kSegBlock, lds);
  if (e != hipSuccess) return e;
  int64_t grid = (int64_t)(per_cu > 0 ? per_cu : 1) * (cus > 0 ? cus : 1);
  if (grid > tiles) grid = tiles;
  hipLaunchKernelGGL(seg_reduce_kernel<LPR>, dim3((unsigned)grid), dim3(kSegBlock), lds, stream, a,
                     tile_base, buckets, q, nb, tiles, tile_ctr, part);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  hipLaunchKernelGGL(seg_fixup_kernel<LPR>, dim3((unsigned)tiles), dim3(kSegBlock), 0, stream, a, part);
  return hipGetLastError();
}

hipError_t launch_segments(const SegmentArgs& a, void* ws, hipStream_t stream) {
  const SegLayout L = seg_layout(a.N, a.D);
  char* base = static_cast<char*>(ws);
  uint32_t* heads = reinterpret_cast<uint32_t*>(base + L.off_heads);
  uint32_t* total = reinterpret_cast<uint32_t*>(base + L.off_total);
  void* scan_ws = base + L.off_scan;
  int32_t* buckets = reinterpret_cast<int32_t*>(base + L.off_buckets);
  uint32_t* tile_ctr = total + 1;
  SegPartials part;
  part.flags = reinterpret_cast<uint32_t*>(base + L.off_flags);
  part.last_seg = reinterpret_cast<uint32_t*>(base + L.off_last_seg);
  int32_t* cnt = reinterpret_cast<int32_t*>(base + L.off_cnt);
  part.first_cc = cnt;
  part.first_ww = cnt + L.tiles;
  part.last_cc = cnt + 2 * L.tiles;
  part.last_ww = cnt + 3 * L.tiles;
  part.first_acc = reinterpret_cast<double*>(base + L.off_first_acc);
  part.last_acc = reinterpret_cast<double*>(base + L.off_last_acc);

  hipLaunchKernelGGL(check_offsets_kernel, dim3(1), dim3(256), 0, stream, a.offsets, a.K, a.N, a.err);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (a.N > 0) {
    hipLaunchKernelGGL(seg_heads_kernel, dim3((unsigned)L.tiles), dim3(kSegBlock), 0, stream, a.keys,
                       a.N, heads);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  e = launch_exclusive_scan_u32(heads, heads, a.N > 0 ? L.tiles : 0, total, scan_ws, stream);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(seg_finish_kernel, dim3(1), dim3(1), 0, stream, (const uint32_t*)total, a.N,
                     a.num_unique, a.seg_offsets);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if (a.N > 0) {
    const int q = bucket_shift(a.N);
    const int nb = (int)(((a.N - 1) >> q) + 1);
    hipLaunchKernelGGL(contrib_buckets_kernel, dim3(1), dim3(256), 0, stream, a.offsets, a.K, a.N, q,
                       nb, buckets, tile_ctr);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    switch (lanes_per_row(a.D)) {
      case 1: e = launch_reduce<1>(a, heads, buckets, q, nb, tile_ctr, part, L.tiles, stream); break;
      case 2: e = launch_reduce<2>(a, heads, buckets, q, nb, tile_ctr, part, L.tiles, stream); break;
      case 4: e = launch_reduce<4>(a, heads, buckets, q, nb, tile_ctr, part, L.tiles, stream); break;
      case 8: e = launch_reduce<8>(a, heads, buckets, q, nb, tile_ctr, part, L.tiles, stream); break;
      case 16: e = launch_reduce<16>(a, heads, buckets, q, nb, tile_ctr, part, L.tiles, stream); break;
      case 32: e = launch_reduce<32>(a, heads, buckets, q, nb, tile_ctr, part, L.tiles, stream); break;
      case 64: e = launch_reduce<64>(a, heads, buckets, q, nb, tile_ctr, part, L.tiles, stream); break;
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
  }
  return hipSuccess;
}

}  // namespace gba
