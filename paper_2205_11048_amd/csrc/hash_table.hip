// Embedding storage keyed by 64-bit IDs (the paper's PS keeps embeddings in
// expandable hash tables keyed by feature ID, Sec. 4.1 / Table 1 setting): an
// open-addressing index from ID to row, and a row pool that grows from a
// device counter.  The push and pull paths run unchanged on the row numbers;
// growing the index (rehash) re-inserts (ID, row) pairs and never moves rows.
//
// find-or-insert: (1) every position claims or finds its ID's slot
// (compare-and-swap on the slot's ID; IDs are never removed, so a non-empty
// slot never changes) and writes its row where the slot already has one; a
// slot that holds no row yet (claimed now, or by an earlier call that found
// the pool full) is listed once, by the one position whose compare-and-swap
// marks its row as pending, and every position of such a slot is listed as
// waiting; (2) the listed slots get the next rows of the pool, in list order
// (a slot past the end of the pool is left without a row, to be served by a
// later call); (3) the waiting positions read their slot's row.  No thread
// ever waits for another's write.  Each block of (1) takes a contiguous range
// of positions and writes its lists, in position order, into the same range
// of the list arrays, with its counts beside them: no list needs a global
// counter.  Once every ID is known, (2) and (3) find empty lists.
#include <algorithm>

#include "gba_device.hpp"
#include "gba_internal.hpp"

namespace gba {

constexpr int kHashBlock = 256;
constexpr int kHashWaves = kHashBlock / kWave;
constexpr int64_t kHashMaxBlocks = 8192;
constexpr int kHashScanBlock = 1024;   // scans the per-block counts of one call
static_assert(kHashMaxBlocks % kHashScanBlock == 0, "whole counts per scan thread");

static inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }
static inline size_t align_up(size_t x) { return (x + 255) & ~size_t(255); }

// Blocks of find-or-insert over n positions and the positions per block.
struct HashGrid {
  int64_t blocks, chunk;
};
static HashGrid hash_grid(int64_t n) {
  HashGrid g;
  const int64_t m = n > 0 ? n : 1;
  g.blocks = std::min<int64_t>(ceil_div(m, kHashBlock), kHashMaxBlocks);
  g.chunk = ceil_div(m, g.blocks);
  return g;
}

struct HashLayout {
  size_t off_pending, off_claimed, off_counts, off_prefix, bytes;
};

static HashLayout hash_layout(int64_t n) {
  HashLayout L{};
  const size_t m = (size_t)(n > 0 ? n : 1);
  size_t o = 0;
  L.off_pending = o; o += align_up(m * 8);    // (position, slot) of the positions waiting for a row
  L.off_claimed = o; o += align_up(m * 4);    // slots listed for a row by this call
  L.off_counts = o;  o += align_up(2 * kHashMaxBlocks * 4);         // per block: listed slots, waiting positions
  L.off_prefix = o;  o += align_up((kHashMaxBlocks + 1) * 4);       // listed slots of the blocks before; [blocks]: all
  L.bytes = o;
  return L;
}

size_t hash_workspace_bytes(int64_t n) { return hash_layout(n).bytes; }

// 64-bit finaliser of MurmurHash3 (Appleby): spreads consecutive or strided
// IDs over the whole index.
__device__ __forceinline__ uint64_t mix64(uint64_t h) {
  h ^= h >> 33;
  h *= 0xff51afd7ed558ccdull;
  h ^= h >> 33;
  h *= 0xc4ceb9fe1a85ec53ull;
  h ^= h >> 33;
  return h;
}

// Row of a slot: kNoRow until the pool hands it one; kPendingRow while it is
// listed for a row inside one find-or-insert.
constexpr int32_t kNoRow = -1;
constexpr int32_t kPendingRow = -2;

__global__ void __launch_bounds__(kHashBlock)
hash_clear_kernel(int64_t* __restrict__ slot_ids, int32_t* __restrict__ slot_rows, int64_t capacity) {
  const int64_t stride = (int64_t)gridDim.x * kHashBlock;
  for (int64_t s = (int64_t)blockIdx.x * kHashBlock + threadIdx.x; s < capacity; s += stride) {
    slot_ids[s] = GBA_EMPTY_ID;
    slot_rows[s] = -1;
  }
}

// Linear probing from the ID's home slot (h: the ID's hash).  Returns the
// slot that holds `id` (claimed here when *claimed), or -1 when every slot
// holds another ID.
__device__ __forceinline__ int64_t claim_or_find(int64_t* slot_ids, int64_t mask, int64_t id, uint64_t h,
                                                 bool* claimed) {
  int64_t s = (int64_t)(h & (uint64_t)mask);
  *claimed = false;
  for (int64_t probe = 0; probe <= mask; ++probe) {
    // a plain load may be stale only while the slot is empty: a filled slot
    // never changes, and the swap below decides every race for an empty one
    const int64_t cur = slot_ids[s];
    if (cur == id) return s;
    if (cur == GBA_EMPTY_ID) {
      const unsigned long long prev =
          atomicCAS(reinterpret_cast<unsigned long long*>(slot_ids + s), (unsigned long long)GBA_EMPTY_ID,
                    (unsigned long long)id);
      if ((int64_t)prev == GBA_EMPTY_ID) {
        *claimed = true;
        return s;
      }
      if ((int64_t)prev == id) return s;
    }
    s = (s + 1) & mask;
  }
  return -1;
}

// Block b takes positions [b * chunk, (b + 1) * chunk) in rounds of one
// position per thread, and lists its slots and waiting positions in position
// order at the same offsets of claimed_slots and pending; counts[b] and
// counts[kHashMaxBlocks + b] receive their numbers.
__global__ void __launch_bounds__(kHashBlock)
hash_claim_kernel(int64_t* __restrict__ slot_ids, int32_t* __restrict__ slot_rows, int64_t mask,
                  const int64_t* __restrict__ ids, int64_t n, int64_t chunk, int64_t* __restrict__ rows_out,
                  int2* __restrict__ pending, int32_t* __restrict__ claimed_slots, uint32_t* __restrict__ counts,
                  int32_t* __restrict__ err) {
  __shared__ uint32_t s_nc[kHashWaves], s_nw[kHashWaves];
  const int64_t p0 = (int64_t)blockIdx.x * chunk;
  const int64_t p1 = p0 + chunk < n ? p0 + chunk : n;
  const int w = threadIdx.x / kWave;
  uint32_t listed = 0, waiting = 0;   // the block's entries so far (the same in every thread)
  for (int64_t r0 = p0; r0 < p1; r0 += kHashBlock) {   // the same rounds for the whole block
    const int64_t i = r0 + threadIdx.x;
    bool claimed = false, waits = false;
    int64_t s = -1;
    if (i < p1) {
      const int64_t id = ids[i];
      int64_t row = -1;
      if (id == GBA_EMPTY_ID) {
        raise_error(err, GBA_DERR_ID_RANGE);
      } else {
        bool fresh = false;
        s = claim_or_find(slot_ids, mask, id, mix64((uint64_t)id), &fresh);
        if (s < 0) {
          raise_error(err, GBA_DERR_TABLE_FULL);
        } else {
          const int32_t r = slot_rows[s];
          if (r >= 0) {
            row = r;   // rows are handed out only by the next launch: a row never changes
          } else {
            // the slot has no row yet: exactly one position lists it (kNoRow
            // cannot turn into a row during this launch), and every position
            // of the slot reads its row after the rows are handed out
            if (r == kNoRow) claimed = atomicCAS(slot_rows + s, kNoRow, kPendingRow) == kNoRow;
            waits = true;
          }
        }
      }
      if (!waits) rows_out[i] = row;
    }
    // block-ordered appends: the waves before this one, then the lanes before
    // (a round with nothing to list, as every round once the IDs are known,
    // ends at the first barrier)
    if (!__syncthreads_or(claimed || waits)) continue;
    const uint64_t mc = __ballot(claimed), mw = __ballot(waits);
    if (lane_id() == 0) {
      s_nc[w] = (uint32_t)__popcll(mc);
      s_nw[w] = (uint32_t)__popcll(mw);
    }
    __syncthreads();
    uint32_t bc = listed, bw = waiting;
#pragma unroll
    for (int k = 0; k < kHashWaves; ++k) {
      const uint32_t a = s_nc[k], b = s_nw[k];
      bc += k < w ? a : 0u;
      bw += k < w ? b : 0u;
      listed += a;
      waiting += b;
    }
    if (claimed) claimed_slots[p0 + bc + __popcll(mc & lanemask_lt())] = (int32_t)s;
    if (waits) pending[p0 + bw + __popcll(mw & lanemask_lt())] = make_int2((int32_t)i, (int32_t)s);
    // s_nc and s_nw are rewritten only after the next round's first barrier
  }
  if (threadIdx.x == 0) {
    counts[blockIdx.x] = listed;
    counts[kHashMaxBlocks + blockIdx.x] = waiting;
  }
}

// Listed slots of the blocks before each block (prefix[b]) and of all of them
// (prefix[blocks]): one block of kHashScanBlock threads, a run of counts each.
__global__ void __launch_bounds__(kHashScanBlock)
hash_scan_kernel(const uint32_t* __restrict__ counts, int blocks, uint32_t* __restrict__ prefix) {
  __shared__ uint32_t tmp[kHashScanBlock / kWave + 1];
  constexpr int kPer = kHashMaxBlocks / kHashScanBlock;
  const int b0 = threadIdx.x * kPer;
  uint32_t c[kPer], sum = 0;
#pragma unroll
  for (int k = 0; k < kPer; ++k) {
    c[k] = b0 + k < blocks ? counts[b0 + k] : 0u;
    sum += c[k];
  }
  uint32_t total;
  uint32_t run = block_exclusive_scan<kHashScanBlock>(sum, tmp, &total);
#pragma unroll
  for (int k = 0; k < kPer; ++k) {
    if (b0 + k < blocks) prefix[b0 + k] = run;
    run += c[k];
  }
  if (threadIdx.x == 0) prefix[blocks] = total;
}

// Rows [num_rows, num_rows + listed) go to the listed slots in list order
// (block by block); block b of this launch serves the slots listed by block b
// of the claim launch.
__global__ void __launch_bounds__(kHashBlock)
hash_assign_kernel(const int64_t* __restrict__ slot_ids, int32_t* __restrict__ slot_rows,
                   const int32_t* __restrict__ claimed_slots, const uint32_t* __restrict__ counts,
                   const uint32_t* __restrict__ prefix, int64_t chunk, const int64_t* __restrict__ num_rows,
                   int64_t max_rows, int64_t* __restrict__ row_ids, int32_t* __restrict__ err) {
  const int64_t c = counts[blockIdx.x];
  if (c == 0) return;
  const int64_t r0 = *num_rows + (int64_t)prefix[blockIdx.x];
  const int32_t* list = claimed_slots + (int64_t)blockIdx.x * chunk;
  for (int64_t j = threadIdx.x; j < c; j += kHashBlock) {
    const int64_t s = list[j];
    const int64_t r = r0 + j;
    if (r >= max_rows) {   // the pool is full: the slot keeps no row, and a later call lists it again
      slot_rows[s] = kNoRow;
      raise_error(err, GBA_DERR_TABLE_FULL);
      continue;
    }
    slot_rows[s] = (int32_t)r;
    if (row_ids) row_ids[r] = slot_ids[s];
  }
}

__global__ void hash_count_kernel(const uint32_t* __restrict__ listed_total, int64_t max_rows,
                                  int64_t* __restrict__ num_rows, int64_t* __restrict__ num_new) {
  const int64_t c = *listed_total;
  int64_t r = *num_rows + c;
  *num_rows = r < max_rows ? r : max_rows;
  if (num_new) *num_new = c;
}

// The positions that waited for a row read it; one whose slot got none (the
// pool is full) gets -1 and reports the table full.  Block b serves the
// positions listed by block b of the claim launch.
__global__ void __launch_bounds__(kHashBlock)
hash_rows_kernel(const int32_t* __restrict__ slot_rows, const int2* __restrict__ pending,
                 const uint32_t* __restrict__ counts, int64_t chunk, int64_t* __restrict__ rows_out,
                 int32_t* __restrict__ err) {
  const int64_t c = counts[kHashMaxBlocks + blockIdx.x];
  const int2* list = pending + (int64_t)blockIdx.x * chunk;
  bool full = false;
  for (int64_t j = threadIdx.x; j < c; j += kHashBlock) {
    const int2 p = list[j];
    const int32_t r = slot_rows[p.y];
    full |= r < 0;
    rows_out[p.x] = r < 0 ? -1 : (int64_t)r;
  }
  if (full) raise_error(err, GBA_DERR_TABLE_FULL);
}

// Re-insert every (ID, row) of the old index into the new one; each ID is
// present once, so every claim succeeds without a race on its row.
__global__ void __launch_bounds__(kHashBlock)
hash_rehash_kernel(const int64_t* __restrict__ old_ids, const int32_t* __restrict__ old_rows, int64_t old_capacity,
                   int64_t* __restrict__ new_ids, int32_t* __restrict__ new_rows, int64_t new_mask,
                   int32_t* __restrict__ err) {
  const int64_t stride = (int64_t)gridDim.x * kHashBlock;
  for (int64_t s = (int64_t)blockIdx.x * kHashBlock + threadIdx.x; s < old_capacity; s += stride) {
    const int64_t id = old_ids[s];
    if (id == GBA_EMPTY_ID) continue;
    bool claimed = false;
    const int64_t t = claim_or_find(new_ids, new_mask, id, mix64((uint64_t)id), &claimed);
    if (t < 0) {
      raise_error(err, GBA_DERR_TABLE_FULL);
      continue;
    }
    new_rows[t] = old_rows[s];
  }
}

static dim3 grid_for(int64_t n) {
  int64_t b = ceil_div(n > 0 ? n : 1, kHashBlock);
  if (b > kHashMaxBlocks) b = kHashMaxBlocks;
  return dim3((unsigned)b);
}

hipError_t launch_hash_clear(int64_t* slot_ids, int32_t* slot_rows, int64_t capacity, hipStream_t stream) {
  hipLaunchKernelGGL(hash_clear_kernel, grid_for(capacity), dim3(kHashBlock), 0, stream, slot_ids, slot_rows,
                     capacity);
  return hipGetLastError();
}

hipError_t launch_hash_find_or_insert(int64_t* slot_ids, int32_t* slot_rows, int64_t capacity, const int64_t* ids,
                                      int64_t n, int64_t* rows_out, int64_t* num_rows, int64_t max_rows,
                                      int64_t* row_ids, int64_t* num_new, void* ws, int32_t* err,
                                      hipStream_t stream) {
  const HashLayout L = hash_layout(n);
  const HashGrid g = hash_grid(n);
  char* base = static_cast<char*>(ws);
  int2* pending = reinterpret_cast<int2*>(base + L.off_pending);
  int32_t* claimed = reinterpret_cast<int32_t*>(base + L.off_claimed);
  uint32_t* counts = reinterpret_cast<uint32_t*>(base + L.off_counts);
  uint32_t* prefix = reinterpret_cast<uint32_t*>(base + L.off_prefix);
  // every block of the claim launch writes its counts (none are cleared
  // beforehand, so the sequence can be captured in a graph)
  hipLaunchKernelGGL(hash_claim_kernel, dim3((unsigned)g.blocks), dim3(kHashBlock), 0, stream, slot_ids, slot_rows,
                     capacity - 1, ids, n, g.chunk, rows_out, pending, claimed, counts, err);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(hash_scan_kernel, dim3(1), dim3(kHashScanBlock), 0, stream, (const uint32_t*)counts,
                     (int)g.blocks, prefix);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  hipLaunchKernelGGL(hash_assign_kernel, dim3((unsigned)g.blocks), dim3(kHashBlock), 0, stream,
                     (const int64_t*)slot_ids, slot_rows, (const int32_t*)claimed, (const uint32_t*)counts,
                     (const uint32_t*)prefix, g.chunk, (const int64_t*)num_rows, max_rows, row_ids, err);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  hipLaunchKernelGGL(hash_count_kernel, dim3(1), dim3(1), 0, stream, (const uint32_t*)(prefix + g.blocks), max_rows,
                     num_rows, num_new);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  hipLaunchKernelGGL(hash_rows_kernel, dim3((unsigned)g.blocks), dim3(kHashBlock), 0, stream,
                     (const int32_t*)slot_rows, (const int2*)pending, (const uint32_t*)counts, g.chunk, rows_out,
                     err);
  return hipGetLastError();
}

hipError_t launch_hash_rehash(const int64_t* old_ids, const int32_t* old_rows, int64_t old_capacity, int64_t* new_ids,
                              int32_t* new_rows, int64_t new_capacity, int32_t* err, hipStream_t stream) {
  hipError_t e = launch_hash_clear(new_ids, new_rows, new_capacity, stream);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(hash_rehash_kernel, grid_for(old_capacity), dim3(kHashBlock), 0, stream, old_ids, old_rows,
                     old_capacity, new_ids, new_rows, new_capacity - 1, err);
  return hipGetLastError();
}

}  // namespace gba
