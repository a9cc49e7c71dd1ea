// Optimiser apply over the touched embedding rows only: gather the row and
// its optimiser state, update with the row's aggregated gradient, scatter
// back.  Rows without a non-zero-weight contribution are skipped (they are
// not updated at this global step; Alg. 2 updates embeddings by ID).
//
// A group of LPR lanes owns kRowBatch consecutive rows at a time and moves
// them as 16-byte non-temporal vectors (every row, state and gradient is
// touched once, so the L2 is left to the kernels that reuse lines); all of a
// batch's loads are issued before the first is used (a skipped row reads row
// 0 and is not written), so a group keeps kRowBatch rows in flight.  The grid
// is persistent and reads the row count from device memory, so no host round
// trip sits between the aggregation and the apply.
#include "gba_device.hpp"
#include "gba_internal.hpp"
#include "optim.hpp"

namespace gba {

constexpr int kRowsBlock = 256;
constexpr int64_t kRowsMaxBlocks = 4096;
constexpr int kRowBatch = 4;

static inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

template <int LPR, bool ADAM>
__global__ void __launch_bounds__(kRowsBlock)
rows_apply_kernel(float* __restrict__ p, float* __restrict__ s1, float* __restrict__ s2,
                  const float* __restrict__ g, const int64_t* __restrict__ rows,
                  const int32_t* __restrict__ active, const int64_t* __restrict__ num_rows,
                  int64_t n, int D, int64_t R, double lr, double eps, double b1, double b2,
                  double bc1, double bc2, int32_t* __restrict__ err) {
  constexpr int G = kRowsBlock / LPR;
  const int lane = threadIdx.x % LPR;
  const int grp = threadIdx.x / LPR;
  int64_t count = *num_rows;
  if (count > n) count = n;
  const OptF32 oc = opt_f32(lr, eps, b1, b2, bc1, bc2);
  bool bad = false;
  const int64_t stride = (int64_t)gridDim.x * G * kRowBatch;
  for (int64_t i0 = ((int64_t)blockIdx.x * G + grp) * kRowBatch; i0 < count; i0 += stride) {
    int64_t r[kRowBatch];
    bool on[kRowBatch];
#pragma unroll
    for (int k = 0; k < kRowBatch; ++k) {
      const int64_t i = i0 + k;
      const int64_t ic = i < count ? i : count - 1;
      const int64_t rk = rows[ic];
      const bool act = i < count && (!active || active[ic] > 0);
      const bool in_range = rk >= 0 && rk < R;
      bad |= act && !in_range;
      on[k] = act && in_range;
      r[k] = on[k] ? rk : 0;
    }
    for (int c = lane * 4; c < D; c += LPR * 4) {
      f32x4 pv[kRowBatch], av[kRowBatch], gv[kRowBatch], vv[ADAM ? kRowBatch : 1];
#pragma unroll
      for (int k = 0; k < kRowBatch; ++k) {
        const int64_t at = r[k] * (int64_t)D + c;
        const int64_t gi = on[k] ? i0 + k : 0;
        pv[k] = load_stream(reinterpret_cast<const f32x4*>(p + at));
        av[k] = load_stream(reinterpret_cast<const f32x4*>(s1 + at));
        if (ADAM) vv[ADAM ? k : 0] = load_stream(reinterpret_cast<const f32x4*>(s2 + at));
        gv[k] = load_stream(reinterpret_cast<const f32x4*>(g + gi * (int64_t)D + c));
      }
#pragma unroll
      for (int k = 0; k < kRowBatch; ++k) {
        if (!on[k]) continue;
        const int64_t at = r[k] * (int64_t)D + c;
        float pe[4] = {pv[k].x, pv[k].y, pv[k].z, pv[k].w};
        float ae[4] = {av[k].x, av[k].y, av[k].z, av[k].w};
        const float ge[4] = {gv[k].x, gv[k].y, gv[k].z, gv[k].w};
        if (ADAM) {
          const f32x4 vk = vv[ADAM ? k : 0];
          float ve[4] = {vk.x, vk.y, vk.z, vk.w};
#pragma unroll
          for (int e = 0; e < 4; ++e)
            adam_update_f32(pe[e], ae[e], ve[e], ge[e], oc);
          store_stream(reinterpret_cast<f32x4*>(s2 + at), f32x4{ve[0], ve[1], ve[2], ve[3]});
        } else {
#pragma unroll
          for (int e = 0; e < 4; ++e) adagrad_update_f32(pe[e], ae[e], ge[e], oc);
        }
        store_stream(reinterpret_cast<f32x4*>(p + at), f32x4{pe[0], pe[1], pe[2], pe[3]});
        store_stream(reinterpret_cast<f32x4*>(s1 + at), f32x4{ae[0], ae[1], ae[2], ae[3]});
      }
    }
  }
  if (bad) raise_error(err, GBA_DERR_ROW_RANGE);
}

template <bool ADAM>
static hipError_t launch_rows(float* p, float* s1, float* s2, const float* g, const int64_t* rows,
                              const int32_t* active, const int64_t* num_rows, int64_t n, int32_t D,
                              int64_t R, double lr, double eps, double b1, double b2, double bc1,
                              double bc2, int32_t* err, hipStream_t stream) {
  if (n <= 0) return hipSuccess;
  int lpr = 1;
  while (lpr < 64 && lpr * 4 < D) lpr <<= 1;
  const int G = kRowsBlock / lpr;
  int64_t blocks = ceil_div(n, (int64_t)G * kRowBatch);
  if (blocks > kRowsMaxBlocks) blocks = kRowsMaxBlocks;
  const dim3 grid((unsigned)blocks), block(kRowsBlock);
#define GBA_ROWS_CASE(L)                                                                          \
  case L:                                                                                         \
    hipLaunchKernelGGL((rows_apply_kernel<L, ADAM>), grid, block, 0, stream, p, s1, s2, g, rows,  \
                       active, num_rows, n, (int)D, R, lr, eps, b1, b2, bc1, bc2, err);           \
    break;
  switch (lpr) {
    GBA_ROWS_CASE(1)
    GBA_ROWS_CASE(2)
    GBA_ROWS_CASE(4)
    GBA_ROWS_CASE(8)
    GBA_ROWS_CASE(16)
    GBA_ROWS_CASE(32)
    GBA_ROWS_CASE(64)
    default:
      return hipErrorInvalidValue;
  }
#undef GBA_ROWS_CASE
  return hipGetLastError();
}

hipError_t launch_rows_adagrad(float* p, float* a, const float* g, const int64_t* rows,
                               const int32_t* active, const int64_t* num_rows, int64_t n, int32_t D,
                               int64_t R, double lr, double eps, int32_t* err, hipStream_t stream) {
  return launch_rows<false>(p, a, nullptr, g, rows, active, num_rows, n, D, R, lr, eps, 0.0, 0.0,
                            1.0, 1.0, err, stream);
}

hipError_t launch_rows_adam(float* p, float* m, float* v, const float* g, const int64_t* rows,
                            const int32_t* active, const int64_t* num_rows, int64_t n, int32_t D,
                            int64_t R, const AdamParams& hp, int32_t* err, hipStream_t stream) {
  return launch_rows<true>(p, m, v, g, rows, active, num_rows, n, D, R, hp.lr, hp.eps, hp.beta1,
                           hp.beta2, hp.bc1, hp.bc2, err, stream);
}

}  // namespace gba
