// Embedding storage keyed by 64-bit IDs (the paper's PS keeps embeddings in
// expandable hash tables keyed by feature ID, Sec. 4.1 / Table 1 setting): an
// open-addressing index from ID to row, and a row pool that grows from a
// device counter.  The push and pull paths run unchanged on the row numbers;
// growing the index (rehash) re-inserts (ID, row) pairs and never moves rows.
//
// find-or-insert is three launches, so no thread ever waits for another's
// write: (1) every position claims or finds its ID's slot (compare-and-swap on
// the slot's ID; IDs are never removed, so a non-empty slot never changes) and
// writes its row where the slot already has one; a slot that holds no row yet
// (claimed now, or by an earlier call that found the pool full) is appended to
// a list once, by the one position whose compare-and-swap marks its row as
// pending, and every position of such a slot to a second list, one list
// atomic per wave each; (2) the listed slots get the next rows of the pool, in
// list order (a slot past the end of the pool is left without a row, to be
// served by a later call); (3) the listed positions read their slot's row.
// Once every ID is known, (2) and (3) find empty lists.
#include "gba_device.hpp"
#include "gba_internal.hpp"

namespace gba {

constexpr int kHashBlock = 256;
constexpr int64_t kHashMaxBlocks = 8192;

static inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }
static inline size_t align_up(size_t x) { return (x + 255) & ~size_t(255); }

struct HashLayout {
  size_t off_pending, off_claimed, off_count, bytes;
};

static HashLayout hash_layout(int64_t n) {
  HashLayout L{};
  const size_t m = (size_t)(n > 0 ? n : 1);
  size_t o = 0;
  L.off_pending = o; o += align_up(m * 8);    // (position, slot) of the positions waiting for a row
  L.off_claimed = o; o += align_up(m * 4);    // slots listed for a row by this call
  L.off_count = o;   o += 256;                // [0] listed slots, [1] waiting positions
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

__global__ void hash_count_reset_kernel(uint32_t* __restrict__ counts) {
  counts[0] = 0u;
  counts[1] = 0u;
}

// Appends this lane's `value` to list[] when `on`, one atomic per wave.
template <typename T>
__device__ __forceinline__ void wave_append(bool on, T value, T* __restrict__ list, uint32_t* __restrict__ count) {
  const uint64_t m = __ballot(on);
  if (!m) return;
  const int leader = __ffsll((unsigned long long)m) - 1;
  uint32_t at = 0;
  if (lane_id() == leader) at = atomicAdd(count, (uint32_t)__popcll(m));
  at = __shfl(at, leader, kWave);
  if (on) list[at + __popcll(m & lanemask_lt())] = value;
}

__global__ void __launch_bounds__(kHashBlock)
hash_clear_kernel(int64_t* __restrict__ slot_ids, int32_t* __restrict__ slot_rows, int64_t capacity) {
  const int64_t stride = (int64_t)gridDim.x * kHashBlock;
  for (int64_t s = (int64_t)blockIdx.x * kHashBlock + threadIdx.x; s < capacity; s += stride) {
    slot_ids[s] = GBA_EMPTY_ID;
    slot_rows[s] = -1;
  }
}

// Linear probing from the ID's home slot.  Returns the slot that holds `id`
// (claimed here when *claimed), or -1 when every slot holds another ID.
__device__ __forceinline__ int64_t claim_or_find(int64_t* slot_ids, int64_t mask, int64_t id, bool* claimed) {
  int64_t s = (int64_t)(mix64((uint64_t)id) & (uint64_t)mask);
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

__global__ void __launch_bounds__(kHashBlock)
hash_claim_kernel(int64_t* __restrict__ slot_ids, int32_t* __restrict__ slot_rows, int64_t mask,
                  const int64_t* __restrict__ ids, int64_t n, int64_t* __restrict__ rows_out,
                  int2* __restrict__ pending, int32_t* __restrict__ claimed_slots, uint32_t* __restrict__ counts,
                  int32_t* __restrict__ err) {
  const int64_t stride = (int64_t)gridDim.x * kHashBlock;
  // every lane of a wave runs the same number of rounds, so the ballots of
  // the list appends see the whole wave
  for (int64_t base = (int64_t)blockIdx.x * kHashBlock + (threadIdx.x & ~(kWave - 1)); base < n; base += stride) {
    const int64_t i = base + lane_id();
    bool claimed = false, waits = false;
    int64_t s = -1;
    if (i < n) {
      const int64_t id = ids[i];
      int64_t row = -1;
      if (id == GBA_EMPTY_ID) {
        raise_error(err, GBA_DERR_ID_RANGE);
      } else {
        bool fresh = false;
        s = claim_or_find(slot_ids, mask, id, &fresh);
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
    wave_append(claimed, (int32_t)s, claimed_slots, counts);
    wave_append(waits, make_int2((int32_t)i, (int32_t)s), pending, counts + 1);
  }
}

// Rows [num_rows, num_rows + claimed) go to the claimed slots, in list order.
__global__ void __launch_bounds__(kHashBlock)
hash_assign_kernel(const int64_t* __restrict__ slot_ids, int32_t* __restrict__ slot_rows,
                   const int32_t* __restrict__ claimed_slots, const uint32_t* __restrict__ claimed_count,
                   const int64_t* __restrict__ num_rows, int64_t max_rows, int64_t* __restrict__ row_ids,
                   int32_t* __restrict__ err) {
  const int64_t c = *claimed_count;
  const int64_t r0 = *num_rows;
  const int64_t stride = (int64_t)gridDim.x * kHashBlock;
  for (int64_t j = (int64_t)blockIdx.x * kHashBlock + threadIdx.x; j < c; j += stride) {
    const int64_t s = claimed_slots[j];
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

__global__ void hash_count_kernel(const uint32_t* __restrict__ claimed_count, int64_t max_rows,
                                  int64_t* __restrict__ num_rows, int64_t* __restrict__ num_new) {
  const int64_t c = *claimed_count;
  int64_t r = *num_rows + c;
  *num_rows = r < max_rows ? r : max_rows;
  if (num_new) *num_new = c;
}

// The positions that waited for a row read it; one whose slot got none (the
// pool is full) gets -1 and reports the table full.
__global__ void __launch_bounds__(kHashBlock)
hash_rows_kernel(const int32_t* __restrict__ slot_rows, const int2* __restrict__ pending,
                 const uint32_t* __restrict__ counts, int64_t* __restrict__ rows_out, int32_t* __restrict__ err) {
  const int64_t c = counts[1];
  const int64_t stride = (int64_t)gridDim.x * kHashBlock;
  bool full = false;
  for (int64_t j = (int64_t)blockIdx.x * kHashBlock + threadIdx.x; j < c; j += stride) {
    const int2 p = pending[j];
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
    const int64_t t = claim_or_find(new_ids, new_mask, id, &claimed);
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
  char* base = static_cast<char*>(ws);
  int2* pending = reinterpret_cast<int2*>(base + L.off_pending);
  int32_t* claimed = reinterpret_cast<int32_t*>(base + L.off_claimed);
  uint32_t* count = reinterpret_cast<uint32_t*>(base + L.off_count);
  // the counter is cleared by a kernel, not a memset, so the sequence can be
  // captured in a graph
  hipLaunchKernelGGL(hash_count_reset_kernel, dim3(1), dim3(1), 0, stream, count);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (n > 0) {
    hipLaunchKernelGGL(hash_claim_kernel, grid_for(n), dim3(kHashBlock), 0, stream, slot_ids, slot_rows, capacity - 1,
                       ids, n, rows_out, pending, claimed, count, err);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(hash_assign_kernel, grid_for(n), dim3(kHashBlock), 0, stream, (const int64_t*)slot_ids,
                       slot_rows, (const int32_t*)claimed, (const uint32_t*)count, (const int64_t*)num_rows, max_rows,
                       row_ids, err);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  hipLaunchKernelGGL(hash_count_kernel, dim3(1), dim3(1), 0, stream, (const uint32_t*)count, max_rows, num_rows,
                     num_new);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if (n > 0) {
    hipLaunchKernelGGL(hash_rows_kernel, grid_for(n), dim3(kHashBlock), 0, stream, (const int32_t*)slot_rows,
                       (const int2*)pending, (const uint32_t*)count, rows_out, err);
    e = hipGetLastError();
  }
  return e;
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
