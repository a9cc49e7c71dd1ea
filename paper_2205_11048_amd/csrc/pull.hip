// Pull side of the PS (Alg. 2, pull responder): a worker sends the embedding
// IDs of its batch and receives their parameters.  The rows are looked up once
// per distinct ID: the request's IDs are sorted (the push path's radix sort),
// runs of equal IDs are numbered, every request position learns the number of
// its ID's run (the inverse map), and one row per distinct ID is gathered.  The
// worker expands rows[inverse[i]] locally, so a Zipf-skewed request moves
// U rows instead of n.
#include "gba_device.hpp"
#include "gba_internal.hpp"

namespace gba {

constexpr int kPullBlock = 256;
constexpr int kPullWaves = kPullBlock / kWave;
constexpr int kPullRounds = (int)(kRunTile / kPullBlock);   // 64 consecutive positions per wave round
constexpr int64_t kGatherMaxBlocks = 4096;

static inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }
static inline size_t align_up(size_t x) { return (x + 255) & ~size_t(255); }

struct PullLayout {
  size_t off_base, off_total, off_scan, bytes;
};

static PullLayout pull_layout(int64_t n) {
  PullLayout L{};
  const size_t tiles = (size_t)(n > 0 ? ceil_div(n, kRunTile) : 1);
  size_t o = 0;
  L.off_base = o;  o += align_up(tiles * 4);
  L.off_total = o; o += 256;
  L.off_scan = o;  o += align_up(run_heads_workspace_bytes(n));
  L.bytes = o;
  return L;
}

size_t pull_workspace_bytes(int64_t n) { return pull_layout(n).bytes; }

// One 1024-position tile per block; wave w takes positions [w * 256, +256) in
// four rounds of 64.  The run number of position p is the number of run heads
// at positions <= p, minus one.
__global__ void __launch_bounds__(kPullBlock)
pull_map_kernel(PullArgs a, const uint32_t* __restrict__ tile_base, const uint32_t* __restrict__ total) {
  __shared__ uint32_t s_wave_heads[kPullWaves];
  const int w = threadIdx.x / kWave;
  const int lane = lane_id();
  const int64_t tile = blockIdx.x;
  const int64_t pw = tile * kRunTile + (int64_t)w * (kPullRounds * kWave);
  const uint64_t le = lanemask_lt() | (1ull << lane);
  uint32_t carry = (pw > 0 && pw < a.n) ? a.keys[pw - 1] : 0u;
  bool carry_ok = pw > 0 && pw < a.n;
  uint64_t hm[kPullRounds];
  uint32_t keyr[kPullRounds], jr[kPullRounds];
#pragma unroll
  for (int r = 0; r < kPullRounds; ++r) {
    const int64_t p = pw + r * kWave + lane;
    const bool valid = p < a.n;
    const uint32_t key = valid ? a.keys[p] : 0u;
    jr[r] = valid ? a.vals[p] : 0u;
    uint32_t kp = __shfl_up(key, 1, kWave);
    bool prev_ok = true;
    if (lane == 0) {
      kp = carry;
      prev_ok = carry_ok;
    }
    const bool head = valid && (!prev_ok || key != kp);
    hm[r] = __ballot(head);
    keyr[r] = key;
    carry = __shfl(key, kWave - 1, kWave);
    carry_ok = true;
  }
  uint32_t wave_heads = 0;
#pragma unroll
  for (int r = 0; r < kPullRounds; ++r) wave_heads += (uint32_t)__popcll(hm[r]);
  if (lane == 0) s_wave_heads[w] = wave_heads;
  __syncthreads();
  uint32_t before = tile_base[tile];
  for (int k = 0; k < w; ++k) before += s_wave_heads[k];
  const uint32_t U = *total;
#pragma unroll
  for (int r = 0; r < kPullRounds; ++r) {
    const int64_t p = pw + r * kWave + lane;
    const uint32_t run = before + (uint32_t)__popcll(hm[r] & le) - 1u;
    if (p < a.n && run < U && (int64_t)jr[r] < a.n) {   // always true when the numbering is consistent
      a.inverse[jr[r]] = (int32_t)run;
      if ((hm[r] >> lane) & 1ull) a.unique_ids[run] = (int64_t)keyr[r];
    }
    before += (uint32_t)__popcll(hm[r]);
  }
}

__global__ void pull_finish_kernel(const uint32_t* __restrict__ total, int64_t* __restrict__ num_unique) {
  *num_unique = (int64_t)*total;
}

// rows[s] = table[unique_ids[s]] for s < U: a group of LPR lanes per row,
// 16-byte accesses, persistent grid (U is read on the device).
template <int LPR>
__global__ void __launch_bounds__(kPullBlock)
pull_gather_kernel(const float* __restrict__ table, const int64_t* __restrict__ unique_ids,
                   const uint32_t* __restrict__ total, int64_t R, int D, float* __restrict__ rows) {
  constexpr int G = kPullBlock / LPR;
  const int lane = threadIdx.x % LPR;
  const int grp = threadIdx.x / LPR;
  const int64_t U = *total;
  const int64_t stride = (int64_t)gridDim.x * G;
  for (int64_t s = (int64_t)blockIdx.x * G + grp; s < U; s += stride) {
    const int64_t r = unique_ids[s];
    if (r < 0 || r >= R) continue;   // unreachable: the IDs were range-checked by the sort
    for (int c = lane * 4; c < D; c += LPR * 4)
      *reinterpret_cast<f32x4*>(rows + s * (int64_t)D + c) =
          *reinterpret_cast<const f32x4*>(table + r * (int64_t)D + c);
  }
}

hipError_t launch_pull(const PullArgs& a, void* ws, hipStream_t stream) {
  const PullLayout L = pull_layout(a.n);
  char* base = static_cast<char*>(ws);
  uint32_t* tile_base = reinterpret_cast<uint32_t*>(base + L.off_base);
  uint32_t* total = reinterpret_cast<uint32_t*>(base + L.off_total);
  hipError_t e = launch_run_heads(a.keys, a.n, tile_base, total, base + L.off_scan, stream);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(pull_finish_kernel, dim3(1), dim3(1), 0, stream, (const uint32_t*)total, a.num_unique);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if (a.n <= 0) return hipSuccess;
  hipLaunchKernelGGL(pull_map_kernel, dim3((unsigned)ceil_div(a.n, kRunTile)), dim3(kPullBlock), 0, stream, a,
                     (const uint32_t*)tile_base, (const uint32_t*)total);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  int lpr = 1;
  while (lpr < 64 && lpr * 4 < a.D) lpr <<= 1;
  int64_t blocks = ceil_div(a.n, kPullBlock / lpr);
  if (blocks > kGatherMaxBlocks) blocks = kGatherMaxBlocks;
#define GBA_GATHER_CASE(LPR_)                                                                             \
  case LPR_:                                                                                              \
    hipLaunchKernelGGL((pull_gather_kernel<LPR_>), dim3((unsigned)blocks), dim3(kPullBlock), 0, stream,   \
                       a.table, (const int64_t*)a.unique_ids, (const uint32_t*)total, a.R, (int)a.D, a.rows); \
    break;
  switch (lpr) {
    GBA_GATHER_CASE(1)
    GBA_GATHER_CASE(2)
    GBA_GATHER_CASE(4)
    GBA_GATHER_CASE(8)
    GBA_GATHER_CASE(16)
    GBA_GATHER_CASE(32)
    GBA_GATHER_CASE(64)
    default:
      return hipErrorInvalidValue;
  }
#undef GBA_GATHER_CASE
  return hipGetLastError();
}

}  // namespace gba
