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
// atomics are used.  A group of LPR lanes (one 16-byte column slice per lane)
// walks 16 consecutive positions, gathering their rows and accumulating runs
// in float64.  Runs that cross group boundaries are joined in LDS; runs that
// cross block boundaries leave one partial per block end, joined by a second
// launch in a fixed order, so results are deterministic.
#include "gba_device.hpp"
#include "gba_internal.hpp"

namespace gba {

constexpr int kSegBlock = 256;
constexpr int kSegRun = 16;   // consecutive sorted positions per lane group

enum : uint32_t { kValid = 1, kOpen = 2, kPass = 4 };          // group flags
enum : uint32_t { kHasFirst = 1, kHasLast = 2, kBlockPass = 4 }; // block flags

static inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }
static inline size_t align_up(size_t x) { return (x + 255) & ~size_t(255); }

static int lanes_per_row(int D) {
  int l = 1;
  while (l < 64 && l * 4 < D) l <<= 1;
  return l;
}
static int64_t seg_tile(int lpr) { return (int64_t)(kSegBlock / lpr) * kSegRun; }

struct SegPartials {
  double* first_acc;   // [nb][D] chain that began in an earlier block
  double* last_acc;    // [nb][D] chain that continues into the next block
  int32_t* first_cc;
  int32_t* first_ww;
  int32_t* last_cc;
  int32_t* last_ww;
  uint32_t* last_seg;
  uint32_t* flags;
};

struct SegLayout {
  int64_t nb;
  size_t off_heads, off_total, off_scan, off_flags, off_last_seg, off_cnt, off_first_acc,
      off_last_acc, bytes;
};

static SegLayout seg_layout(int64_t N, int32_t D) {
  SegLayout L{};
  const int lpr = lanes_per_row(D);
  L.nb = N > 0 ? ceil_div(N, seg_tile(lpr)) : 1;
  const size_t nb = (size_t)L.nb;
  size_t o = 0;
  L.off_heads = o;     o += align_up(nb * 4);
  L.off_total = o;     o += 256;
  L.off_scan = o;      o += align_up(scan_workspace_bytes(L.nb));
  L.off_flags = o;     o += align_up(nb * 4);
  L.off_last_seg = o;  o += align_up(nb * 4);
  L.off_cnt = o;       o += align_up(nb * 16);
  L.off_first_acc = o; o += align_up(nb * (size_t)D * 8);
  L.off_last_acc = o;  o += align_up(nb * (size_t)D * 8);
  L.bytes = o;
  return L;
}

size_t segments_workspace_bytes(int64_t N, int32_t D) { return seg_layout(N, D).bytes; }

// ------------------------------------------------------------------ helpers
// Contribution m of occurrence j: the number of offsets[1..K] that are <= j.
__device__ __forceinline__ int contribution_of(const int32_t* s_off, int K, uint32_t j) {
  int base = 1, len = K;
  while (len > 0) {
    const int half = len >> 1;
    if ((uint32_t)s_off[base + half] <= j) {
      base += half + 1;
      len -= half + 1;
    } else {
      len = half;
    }
  }
  const int m = base - 1;
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

// ------------------------------------------------------------------ kernels
__global__ void check_offsets_kernel(const int64_t* __restrict__ off, int K, int64_t N,
                                     int32_t* __restrict__ err) {
  bool bad = false;
  for (int m = threadIdx.x; m < K; m += blockDim.x) bad |= off[m] > off[m + 1];
  if (threadIdx.x == 0) bad |= (off[0] != 0) || (off[K] != N);
  if (bad) raise_error(err, GBA_DERR_OFFSETS);
}

__global__ void __launch_bounds__(kSegBlock)
seg_heads_kernel(const uint32_t* __restrict__ keys, int64_t N, int64_t tile,
                 uint32_t* __restrict__ heads) {
  __shared__ uint32_t tmp[kSegBlock / kWave + 1];
  const int64_t t0 = (int64_t)blockIdx.x * tile;
  const int64_t t1 = (t0 + tile < N) ? t0 + tile : N;
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

template <int LPR>
__global__ void __launch_bounds__(kSegBlock)
seg_reduce_kernel(SegmentArgs a, const uint32_t* __restrict__ seg_base, SegPartials part) {
  constexpr int G = kSegBlock / LPR;
  constexpr int64_t TILE = (int64_t)G * kSegRun;
  extern __shared__ int32_t s_off[];
  __shared__ f64x4 s_acc[kSegBlock];
  __shared__ int32_t s_cc[G], s_ww[G];
  __shared__ uint32_t s_seg[G], s_flags[G];
  __shared__ uint32_t s_tmp[kSegBlock / kWave + 1];
  __shared__ uint32_t s_bflags;

  const int64_t N = a.N;
  for (int i = threadIdx.x; i <= a.K; i += kSegBlock) {
    int64_t o = a.offsets[i];
    o = o < 0 ? 0 : (o > N ? N : o);
    s_off[i] = (int32_t)o;
  }
  if (threadIdx.x == 0) s_bflags = 0;
  __syncthreads();

  const int lane = threadIdx.x % LPR;
  const int grp = threadIdx.x / LPR;
  const bool lane_on = lane * 4 < a.D;
  const int64_t b = blockIdx.x;
  const int64_t p0 = b * TILE + (int64_t)grp * kSegRun;
  const int nvalid = (N - p0) >= kSegRun ? kSegRun : (N - p0 > 0 ? (int)(N - p0) : 0);

  // sorted keys and occurrence indices of the group's positions
  uint32_t key[kSegRun], jj[kSegRun];
  if (nvalid > 0) {
    // the arrays are padded to a multiple of 64 entries, so whole vectors stay in bounds
    const u32x4* kp = reinterpret_cast<const u32x4*>(a.keys + p0);
    const u32x4* vp = reinterpret_cast<const u32x4*>(a.vals + p0);
#pragma unroll
    for (int q = 0; q < kSegRun / 4; ++q) {
      const u32x4 kv = kp[q], vv = vp[q];
      key[4 * q + 0] = kv.x; key[4 * q + 1] = kv.y; key[4 * q + 2] = kv.z; key[4 * q + 3] = kv.w;
      jj[4 * q + 0] = vv.x;  jj[4 * q + 1] = vv.y;  jj[4 * q + 2] = vv.z;  jj[4 * q + 3] = vv.w;
    }
  } else {
#pragma unroll
    for (int i = 0; i < kSegRun; ++i) key[i] = jj[i] = 0;
  }
  const bool has_prev = p0 > 0 && p0 < N;
  const uint32_t prev_key = has_prev ? a.keys[p0 - 1] : 0u;
  const uint32_t prev_j = has_prev ? a.vals[p0 - 1] : 0u;
  const bool has_next = p0 + kSegRun < N;
  const uint32_t next_key = has_next ? a.keys[p0 + kSegRun] : 0u;

  // contribution, weight, run heads and first occurrences of each contribution
  float wt[kSegRun];
  uint32_t head_mask = 0, newc_mask = 0;
  int mprev = has_prev ? contribution_of(s_off, a.K, prev_j) : -1;
  uint32_t kprev = prev_key;
  bool kprev_ok = has_prev;
#pragma unroll
  for (int i = 0; i < kSegRun; ++i) {
    wt[i] = 0.0f;
    if (i < nvalid) {
      const int m = contribution_of(s_off, a.K, jj[i]);
      const bool head = !kprev_ok || key[i] != kprev;
      const bool newc = head || m != mprev;
      if (a.decay == GBA_DECAY_TOKEN) {
        wt[i] = a.w[m];
      } else {
        const int64_t tg = ((int64_t)key[i] < a.R) ? (int64_t)a.tag[key[i]] : -1;
        int64_t s = tg - a.tokens[m] + 1;
        s = s < 0 ? 0 : s;
        wt[i] = (s <= a.iota) ? 1.0f : 0.0f;
      }
      head_mask |= (uint32_t)head << i;
      newc_mask |= (uint32_t)newc << i;
      kprev = key[i];
      kprev_ok = true;
      mprev = m;
    }
  }

  // gather the rows of the kept occurrences (excluded rows are never read)
  f32x4 rv[kSegRun];
#pragma unroll
  for (int i = 0; i < kSegRun; ++i) {
    rv[i] = f32x4{0.f, 0.f, 0.f, 0.f};
    if (i < nvalid && wt[i] != 0.0f && lane_on && (int64_t)jj[i] < N)
      rv[i] = *reinterpret_cast<const f32x4*>(a.rows + (int64_t)jj[i] * a.D + lane * 4);
  }

  // segment number of the group's first head
  uint32_t nheads_total;
  const uint32_t ex = block_exclusive_scan<kSegBlock>(lane == 0 ? (uint32_t)__popc(head_mask) : 0u,
                                                      s_tmp, &nheads_total);
  const int wl = threadIdx.x % kWave;
  const uint32_t gbase = seg_base[b] + (uint32_t)__shfl(ex, wl - lane, kWave);

  f64x4 acc = {0.0, 0.0, 0.0, 0.0};
  int cc = 0, ww = 0;
  int64_t seg = (int64_t)gbase - 1;
  const bool first_open = nvalid > 0 && !(head_mask & 1u);
  bool in_first = true;
  f64x4 facc = {0.0, 0.0, 0.0, 0.0};
  int fcc = 0, fww = 0;
  bool owner = false;
#pragma unroll
  for (int i = 0; i < kSegRun; ++i) {
    if (i < nvalid) {
      if ((head_mask >> i) & 1u) {
        if (i > 0) {
          if (in_first && first_open) {
            facc = acc; fcc = cc; fww = ww; owner = true;
          } else {
            finalize_segment(a, seg, acc, cc, ww, lane, lane_on);
          }
          in_first = false;
        }
        ++seg;
        acc = f64x4{0.0, 0.0, 0.0, 0.0};
        cc = ww = 0;
        if (lane == 0 && seg < N) {
          a.unique_ids[seg] = (int64_t)key[i];
          a.seg_offsets[seg] = p0 + i;
        }
      }
      if (wt[i] != 0.0f) acc += (double)wt[i] * widen(rv[i]);
      const int nc = (newc_mask >> i) & 1u;
      cc += nc;
      ww += (nc && wt[i] != 0.0f) ? 1 : 0;
    }
  }

  bool last_open = false, pass = false;
  if (nvalid > 0) {
    last_open = nvalid == kSegRun && has_next && next_key == key[kSegRun - 1];
    if (last_open) {
      pass = in_first && first_open;
      s_acc[threadIdx.x] = acc;
      if (lane == 0) {
        s_cc[grp] = cc;
        s_ww[grp] = ww;
        s_seg[grp] = (uint32_t)seg;
      }
    } else if (in_first && first_open) {
      facc = acc; fcc = cc; fww = ww; owner = true;
    } else {
      finalize_segment(a, seg, acc, cc, ww, lane, lane_on);
    }
  }
  if (lane == 0) s_flags[grp] = (nvalid > 0 ? kValid : 0u) | (last_open ? kOpen : 0u) | (pass ? kPass : 0u);
  __syncthreads();

  const int D = a.D;
  // a group whose first run began before it closes the chain of runs
  if (owner) {
    f64x4 tot = facc;
    int tcc = fcc, tww = fww;
    bool from_prev_block = true;
    for (int gg = grp - 1; gg >= 0; --gg) {
      tot += s_acc[gg * LPR + lane];
      tcc += s_cc[gg];
      tww += s_ww[gg];
      if (!(s_flags[gg] & kPass)) {
        from_prev_block = false;
        break;
      }
    }
    if (from_prev_block) {
      if (lane_on) *reinterpret_cast<f64x4*>(part.first_acc + b * D + lane * 4) = tot;
      if (lane == 0) {
        part.first_cc[b] = tcc;
        part.first_ww[b] = tww;
        atomicOr(&s_bflags, kHasFirst);
      }
    } else {
      finalize_segment(a, (int64_t)gbase - 1, tot, tcc, tww, lane, lane_on);
    }
  }
  // the chain that runs into the next block
  if (grp == G - 1 && (s_flags[G - 1] & kOpen)) {
    f64x4 tot = s_acc[(G - 1) * LPR + lane];
    int tcc = s_cc[G - 1], tww = s_ww[G - 1];
    int gg = G - 1;
    while (gg > 0 && (s_flags[gg] & kPass)) {
      --gg;
      tot += s_acc[gg * LPR + lane];
      tcc += s_cc[gg];
      tww += s_ww[gg];
    }
    if (s_flags[gg] & kPass) {   // the whole block is inside one segment
      if (lane_on) *reinterpret_cast<f64x4*>(part.first_acc + b * D + lane * 4) = tot;
      if (lane == 0) {
        part.first_cc[b] = tcc;
        part.first_ww[b] = tww;
        atomicOr(&s_bflags, kHasFirst | kBlockPass);
      }
    } else {
      if (lane_on) *reinterpret_cast<f64x4*>(part.last_acc + b * D + lane * 4) = tot;
      if (lane == 0) {
        part.last_cc[b] = tcc;
        part.last_ww[b] = tww;
        part.last_seg[b] = s_seg[G - 1];
        atomicOr(&s_bflags, kHasLast);
      }
    }
  }
  __syncthreads();
  if (threadIdx.x == 0) part.flags[b] = s_bflags;
}

// Joins, for each segment that runs past the end of the block holding its
// head, the partial sums of every later block it covers.
template <int LPR>
__global__ void __launch_bounds__(kSegBlock)
seg_fixup_kernel(SegmentArgs a, SegPartials part) {
  constexpr int G = kSegBlock / LPR;
  constexpr int64_t TILE = (int64_t)G * kSegRun;
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
  const int64_t b_end = (end - 1) / TILE;
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
static hipError_t launch_reduce(const SegmentArgs& a, const uint32_t* seg_base, SegPartials part,
                                int64_t nb, hipStream_t stream) {
  const size_t lds = (size_t)(a.K + 1) * sizeof(int32_t);
  hipLaunchKernelGGL(seg_reduce_kernel<LPR>, dim3((unsigned)nb), dim3(kSegBlock), lds, stream, a,
                     seg_base, part);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(seg_fixup_kernel<LPR>, dim3((unsigned)nb), dim3(kSegBlock), 0, stream, a, part);
  return hipGetLastError();
}

hipError_t launch_segments(const SegmentArgs& a, void* ws, hipStream_t stream) {
  const SegLayout L = seg_layout(a.N, a.D);
  char* base = static_cast<char*>(ws);
  uint32_t* heads = reinterpret_cast<uint32_t*>(base + L.off_heads);
  uint32_t* total = reinterpret_cast<uint32_t*>(base + L.off_total);
  void* scan_ws = base + L.off_scan;
  SegPartials part;
  part.flags = reinterpret_cast<uint32_t*>(base + L.off_flags);
  part.last_seg = reinterpret_cast<uint32_t*>(base + L.off_last_seg);
  int32_t* cnt = reinterpret_cast<int32_t*>(base + L.off_cnt);
  part.first_cc = cnt;
  part.first_ww = cnt + L.nb;
  part.last_cc = cnt + 2 * L.nb;
  part.last_ww = cnt + 3 * L.nb;
  part.first_acc = reinterpret_cast<double*>(base + L.off_first_acc);
  part.last_acc = reinterpret_cast<double*>(base + L.off_last_acc);

  hipLaunchKernelGGL(check_offsets_kernel, dim3(1), dim3(256), 0, stream, a.offsets, a.K, a.N, a.err);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int lpr = lanes_per_row(a.D);
  const int64_t tile = seg_tile(lpr);
  if (a.N > 0) {
    hipLaunchKernelGGL(seg_heads_kernel, dim3((unsigned)L.nb), dim3(kSegBlock), 0, stream, a.keys,
                       a.N, tile, heads);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  e = launch_exclusive_scan_u32(heads, heads, a.N > 0 ? L.nb : 0, total, scan_ws, stream);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(seg_finish_kernel, dim3(1), dim3(1), 0, stream, (const uint32_t*)total, a.N,
                     a.num_unique, a.seg_offsets);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if (a.N > 0) {
    switch (lpr) {
      case 1: e = launch_reduce<1>(a, heads, part, L.nb, stream); break;
      case 2: e = launch_reduce<2>(a, heads, part, L.nb, stream); break;
      case 4: e = launch_reduce<4>(a, heads, part, L.nb, stream); break;
      case 8: e = launch_reduce<8>(a, heads, part, L.nb, stream); break;
      case 16: e = launch_reduce<16>(a, heads, part, L.nb, stream); break;
      case 32: e = launch_reduce<32>(a, heads, part, L.nb, stream); break;
      case 64: e = launch_reduce<64>(a, heads, part, L.nb, stream); break;
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
