// Dense part of the push-step: the decayed weighted sum of the K dense
// gradients divided by N_a (Alg. 2), and the elementwise optimiser updates
// (Adagrad, Adam; Table 1 names them), separately or fused.
//
// The reduction streams K_eff * P floats from HBM.  A block of 8 waves owns
// 128 KB of the output at a time; each wave reads 16 KB of one gradient as 16
// consecutive 1 KB loads before moving to the next gradient, so the memory
// system sees long contiguous runs per gradient wherever the caller placed
// the K buffers (short runs from many buffers at once were measured to lose
// up to 15% of bandwidth to DRAM row conflicts, depending on the buffers'
// relative addresses).  Where P is too small for such blocks to give every
// compute unit one, threads take 4 vectors (or 1) instead of 16.  Each thread
// accumulates its vectors in float64 in buffer order, so the only rounding is
// the final one to float.
#include <algorithm>

#include "gba_device.hpp"
#include "gba_internal.hpp"
#include "optim.hpp"

namespace gba {

constexpr int kDenseBlock = 256;                                      // elementwise optimiser kernels
constexpr int kSumBlock = 512;                                        // the reduction: 8 waves
// f32x4 per thread: 16 (each wave reads 16 KB of one gradient in a row); 4 or
// 1 where P is too small for 16 to give every compute unit a block
constexpr int kDenseVecs = 16;
template <int VECS>
constexpr int64_t dense_span() { return (int64_t)kSumBlock * VECS; }   // vectors per block step
constexpr int64_t kDenseMaxBlocks = 65535;
constexpr int64_t kApplyMaxBlocks = 8192;
constexpr int64_t kDenseRoundsPerLaunch = 1;                           // rounds of resident blocks per launch

static inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

// Every block builds, in LDS, the ordered list of contributions whose weight
// is non-zero; excluded gradients are never touched (Eq. 1: they are not
// aggregated).  `aligned` tells whether every kept gradient allows 16-byte loads.
__device__ __forceinline__ int build_kept_list(const float* const* grads, const float* w, int K,
                                               uint16_t* kept, float* kw, uint32_t* tmp,
                                               int* aligned) {
  constexpr int kPer = (GBA_MAX_K + kSumBlock - 1) / kSumBlock;
  const int lo = threadIdx.x * kPer;
  uint32_t c = 0;
  bool al = true;
  for (int k = 0; k < kPer; ++k) {
    const int m = lo + k;
    if (m < K && w[m] != 0.0f) {
      ++c;
      al &= ((reinterpret_cast<uintptr_t>(grads[m]) & 15u) == 0);
    }
  }
  if (threadIdx.x == 0) *aligned = 1;
  __syncthreads();
  if (!al) *aligned = 0;
  uint32_t total;
  uint32_t pos = block_exclusive_scan<kSumBlock>(c, tmp, &total);
  for (int k = 0; k < kPer; ++k) {
    const int m = lo + k;
    if (m < K && w[m] != 0.0f) {
      kept[pos] = (uint16_t)m;
      kw[pos] = w[m];
      ++pos;
    }
  }
  __syncthreads();
  return (int)total;
}

// What the reduction does with each finished element g = sum / K: store it
// (kStoreOnly), and/or apply Adagrad or Adam to the dense parameters right
// away, which spares the round trip of g through memory (in the apply modes
// `out` may be null); or, for the early weighted sum, nothing yet: the
// float64 running sum is stored back (kAccumulate).
enum DenseMode : int { kStoreOnly = 0, kApplyAdagrad = 1, kApplyAdam = 2, kAccumulate = 3 };
struct DenseState {
  float* p;
  float* s1;   // Adagrad accumulator or Adam m
  float* s2;   // Adam v
  OptF32 c;    // the optimiser's float32 constants
};

template <int MODE>
__device__ __forceinline__ void finish_element(float g, int64_t e, float* out, const DenseState& st) {
  if (out) out[e] = g;
  if (MODE == kApplyAdagrad) {
    float pe = st.p[e], ae = st.s1[e];
    adagrad_update_f32(pe, ae, g, st.c);
    st.p[e] = pe;
    st.s1[e] = ae;
  } else if (MODE == kApplyAdam) {
    float pe = st.p[e], me = st.s1[e], ve = st.s2[e];
    adam_update_f32(pe, me, ve, g, st.c);
    st.p[e] = pe;
    st.s1[e] = me;
    st.s2[e] = ve;
  }
}

// One element, for the last P % 4 and for buffers that are not 16-byte aligned.
template <int MODE, bool CARRY>
__device__ __forceinline__ void finish_scalar(const float* const* grads, const uint16_t* kept, const float* kw,
                                              int nk, int64_t e, float* out, const DenseState& st,
                                              double* run, double denom, int reset) {
  double acc = CARRY ? run[e] : 0.0;
  for (int i = 0; i < nk; ++i) acc = __builtin_fma((double)kw[i], (double)grads[kept[i]][e], acc);   // exact product
  if (MODE == kAccumulate) {
    run[e] = acc;
  } else {
    finish_element<MODE>((float)(acc / denom), e, out, st);
    if (CARRY && reset) run[e] = 0.0;
  }
}

// Vectors q[j] = vb + 64 j (j < VECS, q < nvec) are finished: g in
// float first (which frees the float64 sums), then the optimiser, with the
// state of a whole group of vectors requested at once (16 for Adagrad, 8 for
// Adam: what fits the registers the sums held), so a block's finishing costs
// one or two memory latencies, not one per vector.
template <int MODE, int VECS>
__device__ __forceinline__ void finish_vectors(const f64x4* acc, double denom, int64_t vb, int64_t nvec,
                                               float* out, const DenseState& st) {
  f32x4 g[VECS];
#pragma unroll
  for (int j = 0; j < VECS; ++j) g[j] = narrow(acc[j] / denom);
  if (out) {
#pragma unroll
    for (int j = 0; j < VECS; ++j)
      if (vb + kWave * j < nvec) store_stream(reinterpret_cast<f32x4*>(out) + vb + kWave * j, g[j]);
  }
  if (MODE == kStoreOnly) return;
  constexpr int kGroup = (MODE == kApplyAdam) ? (VECS < 8 ? VECS : 8) : VECS;
#pragma unroll
  for (int j0 = 0; j0 < VECS; j0 += kGroup) {
    f32x4 pv[kGroup], sv[kGroup], vv[kGroup];
#pragma unroll
    for (int jj = 0; jj < kGroup; ++jj) {
      const int64_t q = vb + kWave * (j0 + jj);
      if (q < nvec) {
        pv[jj] = load_stream(reinterpret_cast<const f32x4*>(st.p) + q);
        sv[jj] = load_stream(reinterpret_cast<const f32x4*>(st.s1) + q);
        if (MODE == kApplyAdam) vv[jj] = load_stream(reinterpret_cast<const f32x4*>(st.s2) + q);
      }
    }
#pragma unroll
    for (int jj = 0; jj < kGroup; ++jj) {
      const int64_t q = vb + kWave * (j0 + jj);
      if (q >= nvec) continue;
      const f32x4 gj = g[j0 + jj];
      float pe[4] = {pv[jj].x, pv[jj].y, pv[jj].z, pv[jj].w};
      float se[4] = {sv[jj].x, sv[jj].y, sv[jj].z, sv[jj].w};
      const float ge[4] = {gj.x, gj.y, gj.z, gj.w};
      if (MODE == kApplyAdam) {
        float ve[4] = {vv[jj].x, vv[jj].y, vv[jj].z, vv[jj].w};
#pragma unroll
        for (int k = 0; k < 4; ++k) adam_update_f32(pe[k], se[k], ve[k], ge[k], st.c);
        store_stream(reinterpret_cast<f32x4*>(st.s2) + q, f32x4{ve[0], ve[1], ve[2], ve[3]});
      } else {
#pragma unroll
        for (int k = 0; k < 4; ++k) adagrad_update_f32(pe[k], se[k], ge[k], st.c);
      }
      store_stream(reinterpret_cast<f32x4*>(st.p) + q, f32x4{pe[0], pe[1], pe[2], pe[3]});
      store_stream(reinterpret_cast<f32x4*>(st.s1) + q, f32x4{se[0], se[1], se[2], se[3]});
    }
  }
}

// The weighted sum of the kept gradients, added in buffer order to a float64
// running sum that starts at 0 (the whole buffer at once) or at run[] (the
// early weighted sum, CARRY: contributions folded in as they arrive, in
// arrival order, so the result is bitwise the one-shot sum).  Then the
// MODE's finishing; with CARRY, `reset` clears run[] for the next step.
template <int MODE, bool CARRY, int VECS>
__global__ void __launch_bounds__(kSumBlock)
aggregate_dense_kernel(const float* const* __restrict__ grads, const float* __restrict__ w, int K,
                       int64_t P, float* __restrict__ out, DenseState st, double* __restrict__ run,
                       double denom, int reset, int64_t step0, int64_t step_end) {
  __shared__ uint16_t kept[GBA_MAX_K];
  __shared__ float kw[GBA_MAX_K];
  __shared__ uint32_t tmp[kSumBlock / kWave + 1];
  __shared__ int aligned;
  const int nk = build_kept_list(grads, w, K, kept, kw, tmp, &aligned);
  const int64_t stride = (int64_t)gridDim.x * kSumBlock;
  const bool outputs_aligned = ((reinterpret_cast<uintptr_t>(out) | reinterpret_cast<uintptr_t>(st.p) |
                                 reinterpret_cast<uintptr_t>(st.s1) | reinterpret_cast<uintptr_t>(st.s2)) &
                                15u) == 0 &&
                               (reinterpret_cast<uintptr_t>(run) & 31u) == 0;   // null pointers count as aligned
  if (aligned && outputs_aligned) {
    const int64_t nvec = P / 4;
    for (int64_t s = step0 + blockIdx.x; s < step_end; s += gridDim.x) {
      const int64_t b0 = s * dense_span<VECS>();
      // wave w covers vectors [b0 + w * 1024, +1024): lane l takes l, l + 64, ...
      const int64_t vb = b0 + (int64_t)(threadIdx.x / kWave) * (kWave * VECS) + (threadIdx.x % kWave);
      f64x4 acc[VECS];
#pragma unroll
      for (int j = 0; j < VECS; ++j) {
        acc[j] = f64x4{0.0, 0.0, 0.0, 0.0};
        if (CARRY && vb + kWave * j < nvec) acc[j] = reinterpret_cast<const f64x4*>(run)[vb + kWave * j];
      }
      // the next gradient's address is fetched while this one's loads are in
      // flight (global loads: the LDS and scalar reads for it do not wait on them)
      const f32x4* g_next = nk > 0 ? reinterpret_cast<const f32x4*>(grads[kept[0]]) : nullptr;
      for (int i = 0; i < nk; ++i) {
        const f32x4* g = g_next + vb;
        f32x4 x[VECS];
#pragma unroll
        for (int j = 0; j < VECS; ++j)
          x[j] = (vb + kWave * j < nvec) ? load_stream_global(g + kWave * j) : f32x4{0.f, 0.f, 0.f, 0.f};
        if (i + 1 < nk) g_next = reinterpret_cast<const f32x4*>(grads[kept[i + 1]]);
        const double wi = (double)kw[i];
#pragma unroll
        for (int j = 0; j < VECS; ++j) acc[j] = fma_widen(wi, x[j], acc[j]);
      }
      if (MODE == kAccumulate) {
#pragma unroll
        for (int j = 0; j < VECS; ++j)
          if (vb + kWave * j < nvec) reinterpret_cast<f64x4*>(run)[vb + kWave * j] = acc[j];
      } else {
        finish_vectors<MODE, VECS>(acc, denom, vb, nvec, out, st);
        if (CARRY && reset) {
#pragma unroll
          for (int j = 0; j < VECS; ++j)
            if (vb + kWave * j < nvec) reinterpret_cast<f64x4*>(run)[vb + kWave * j] = f64x4{0.0, 0.0, 0.0, 0.0};
        }
      }
    }
    // the last P % 4 elements
    const int64_t tail0 = nvec * 4;
    if (step0 == 0 && blockIdx.x == 0 && threadIdx.x < P - tail0)
      finish_scalar<MODE, CARRY>(grads, kept, kw, nk, tail0 + threadIdx.x, out, st, run, denom, reset);
  } else if (step0 == 0) {   // the first launch takes every element
    for (int64_t e = (int64_t)blockIdx.x * kSumBlock + threadIdx.x; e < P; e += stride)
      finish_scalar<MODE, CARRY>(grads, kept, kw, nk, e, out, st, run, denom, reset);
  }
}

// Block steps of a dense call over P elements and the steps each launch
// covers.  Where the steps outnumber two rounds of the blocks the GPU holds at
// once, they are launched one round at a time: blocks that start together read
// the same gradient at neighbouring offsets, while in one long launch the
// blocks drift apart until they read all K buffers at once, which costs
// bandwidth (DRAM row changes).  K == 0 (finishing a running sum) reads no
// gradients and takes one launch.
template <int MODE, bool CARRY, int VECS>
static void dense_rounds(int64_t P, int32_t K, int cus, int64_t* steps, int64_t* round) {
  *steps = std::max<int64_t>(ceil_div(P / 4, dense_span<VECS>()), 1);
  *round = *steps;
  int per_cu = 0;
  if (K > 0 && cus > 0 &&
      hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, aggregate_dense_kernel<MODE, CARRY, VECS>, kSumBlock,
                                                   0) == hipSuccess &&
      per_cu > 0 && *steps > 2 * kDenseRoundsPerLaunch * (int64_t)cus * per_cu)
    *round = kDenseRoundsPerLaunch * (int64_t)cus * per_cu;
}

// Compute units of the current device (0 if unknown).
static int device_cus() {
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess || hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) !=
                                              hipSuccess)
    return 0;
  return cus;
}

// Vectors per thread for P elements: the most that still give every compute
// unit a block step.
static int dense_vecs(int64_t P, int cus) {
  const int64_t nvec = P / 4;
  if (cus <= 0 || ceil_div(nvec, dense_span<kDenseVecs>()) >= cus) return kDenseVecs;
  if (ceil_div(nvec, dense_span<4>()) >= cus) return 4;
  return 1;
}

template <int MODE, bool CARRY, int VECS>
static hipError_t launch_dense_vecs(const float* const* grads, const float* w, int32_t K, int64_t P, float* out,
                                    const DenseState& st, double* run, double denom, int reset, int cus,
                                    hipStream_t stream) {
  // one block step per block; unaligned buffers fall back to a grid-stride
  // loop over single elements in the first launch
  int64_t steps = 0, round = 0;
  dense_rounds<MODE, CARRY, VECS>(P, K, cus, &steps, &round);
  for (int64_t s0 = 0; s0 < steps; s0 += round) {
    const int64_t s1 = std::min(steps, s0 + round);
    const int64_t blocks = std::min(s1 - s0, kDenseMaxBlocks);
    hipLaunchKernelGGL((aggregate_dense_kernel<MODE, CARRY, VECS>), dim3((unsigned)blocks), dim3(kSumBlock), 0,
                       stream, grads, w, (int)K, P, out, st, run, denom, reset, s0, s1);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

template <int MODE, bool CARRY>
static hipError_t launch_dense_mode(const float* const* grads, const float* w, int32_t K, int64_t P,
                                    float* out, const DenseState& st, double* run, double denom, int reset,
                                    hipStream_t stream) {
  if (P <= 0) return hipSuccess;
  const int cus = device_cus();
  switch (dense_vecs(P, cus)) {
    case 1: return launch_dense_vecs<MODE, CARRY, 1>(grads, w, K, P, out, st, run, denom, reset, cus, stream);
    case 4: return launch_dense_vecs<MODE, CARRY, 4>(grads, w, K, P, out, st, run, denom, reset, cus, stream);
    default:
      return launch_dense_vecs<MODE, CARRY, kDenseVecs>(grads, w, K, P, out, st, run, denom, reset, cus, stream);
  }
}

template <int MODE, bool CARRY>
static int64_t launch_count(int64_t P, int32_t K) {
  const int cus = device_cus();
  int64_t steps = 0, round = 0;
  switch (dense_vecs(P, cus)) {
    case 1: dense_rounds<MODE, CARRY, 1>(P, K, cus, &steps, &round); break;
    case 4: dense_rounds<MODE, CARRY, 4>(P, K, cus, &steps, &round); break;
    default: dense_rounds<MODE, CARRY, kDenseVecs>(P, K, cus, &steps, &round); break;
  }
  return ceil_div(steps, round);
}

int64_t dense_launch_count(int64_t P, int32_t K, int opt) {
  if (P <= 0) return 0;
  switch (opt) {
    case 1: return launch_count<kApplyAdagrad, false>(P, K);
    case 2: return launch_count<kApplyAdam, false>(P, K);
    case 3: return launch_count<kAccumulate, true>(P, K);
    default: return launch_count<kStoreOnly, false>(P, K);
  }
}

hipError_t launch_aggregate_dense(const float* const* grads, const float* w, int32_t K, int64_t P,
                                  float* out, hipStream_t stream) {
  return launch_dense_mode<kStoreOnly, false>(grads, w, K, P, out, DenseState{}, nullptr, (double)K, 0, stream);
}

static DenseState adagrad_state(float* p, float* a, double lr, double eps) {
  return DenseState{p, a, nullptr, opt_f32(lr, eps)};
}

static DenseState adam_state(float* p, float* m, float* v, const AdamParams& hp) {
  return DenseState{p, m, v, opt_f32(hp.lr, hp.eps, hp.beta1, hp.beta2, hp.bc1, hp.bc2)};
}

hipError_t launch_aggregate_apply_dense_adagrad(const float* const* grads, const float* w, int32_t K,
                                                int64_t P, float* out, float* p, float* a, double lr,
                                                double eps, hipStream_t stream) {
  return launch_dense_mode<kApplyAdagrad, false>(grads, w, K, P, out, adagrad_state(p, a, lr, eps), nullptr,
                                                 (double)K, 0, stream);
}

hipError_t launch_aggregate_apply_dense_adam(const float* const* grads, const float* w, int32_t K,
                                             int64_t P, float* out, float* p, float* m, float* v,
                                             const AdamParams& hp, hipStream_t stream) {
  return launch_dense_mode<kApplyAdam, false>(grads, w, K, P, out, adam_state(p, m, v, hp), nullptr, (double)K, 0,
                                              stream);
}

hipError_t launch_accumulate_dense(const float* const* grads, const float* w, int32_t J, int64_t P, double* run,
                                   hipStream_t stream) {
  return launch_dense_mode<kAccumulate, true>(grads, w, J, P, nullptr, DenseState{}, run, 1.0, 0, stream);
}

hipError_t launch_finalize_dense(double* run, int32_t K, int64_t P, float* out, int reset, hipStream_t stream) {
  return launch_dense_mode<kStoreOnly, true>(nullptr, nullptr, 0, P, out, DenseState{}, run, (double)K, reset,
                                             stream);
}

hipError_t launch_finalize_apply_dense_adagrad(double* run, int32_t K, int64_t P, float* out, float* p, float* a,
                                               double lr, double eps, int reset, hipStream_t stream) {
  return launch_dense_mode<kApplyAdagrad, true>(nullptr, nullptr, 0, P, out, adagrad_state(p, a, lr, eps), run,
                                                (double)K, reset, stream);
}

hipError_t launch_finalize_apply_dense_adam(double* run, int32_t K, int64_t P, float* out, float* p, float* m,
                                            float* v, const AdamParams& hp, int reset, hipStream_t stream) {
  return launch_dense_mode<kApplyAdam, true>(nullptr, nullptr, 0, P, out, adam_state(p, m, v, hp), run, (double)K,
                                             reset, stream);
}

// ---------------------------------------------------------------- optimisers
// Elementwise over n: threads take four consecutive elements with 16-byte
// non-temporal accesses when every array is 16-byte aligned (state and
// gradient are each touched once), else one element per thread.
__device__ __forceinline__ bool all_aligned16(const void* a, const void* b, const void* c, const void* d) {
  return ((reinterpret_cast<uintptr_t>(a) | reinterpret_cast<uintptr_t>(b) | reinterpret_cast<uintptr_t>(c) |
           reinterpret_cast<uintptr_t>(d)) & 15u) == 0;
}

__global__ void __launch_bounds__(kDenseBlock)
dense_adagrad_kernel(float* __restrict__ p, float* __restrict__ a, const float* __restrict__ g,
                     int64_t n, OptF32 c) {
  const int64_t stride = (int64_t)gridDim.x * kDenseBlock;
  const int64_t t0 = (int64_t)blockIdx.x * kDenseBlock + threadIdx.x;
  if (all_aligned16(p, a, g, p)) {
    const int64_t nvec = n / 4;
    for (int64_t v = t0; v < nvec; v += stride) {
      const f32x4 pv = load_stream(reinterpret_cast<const f32x4*>(p) + v);
      const f32x4 av = load_stream(reinterpret_cast<const f32x4*>(a) + v);
      const f32x4 gv = load_stream(reinterpret_cast<const f32x4*>(g) + v);
      float pe[4] = {pv.x, pv.y, pv.z, pv.w}, ae[4] = {av.x, av.y, av.z, av.w};
      const float ge[4] = {gv.x, gv.y, gv.z, gv.w};
#pragma unroll
      for (int k = 0; k < 4; ++k) adagrad_update_f32(pe[k], ae[k], ge[k], c);
      store_stream(reinterpret_cast<f32x4*>(p) + v, f32x4{pe[0], pe[1], pe[2], pe[3]});
      store_stream(reinterpret_cast<f32x4*>(a) + v, f32x4{ae[0], ae[1], ae[2], ae[3]});
    }
    // the last n % 4 elements
    for (int64_t e = nvec * 4 + threadIdx.x; blockIdx.x == 0 && e < n; e += kDenseBlock) {
      float pe = p[e], ae = a[e];
      adagrad_update_f32(pe, ae, g[e], c);
      p[e] = pe;
      a[e] = ae;
    }
  } else {
    for (int64_t e = t0; e < n; e += stride) {
      float pe = p[e], ae = a[e];
      adagrad_update_f32(pe, ae, g[e], c);
      p[e] = pe;
      a[e] = ae;
    }
  }
}

__global__ void __launch_bounds__(kDenseBlock)
dense_adam_kernel(float* __restrict__ p, float* __restrict__ m, float* __restrict__ v,
                  const float* __restrict__ g, int64_t n, OptF32 c) {
  const int64_t stride = (int64_t)gridDim.x * kDenseBlock;
  const int64_t t0 = (int64_t)blockIdx.x * kDenseBlock + threadIdx.x;
  if (all_aligned16(p, m, v, g)) {
    const int64_t nvec = n / 4;
    for (int64_t q = t0; q < nvec; q += stride) {
      const f32x4 pv = load_stream(reinterpret_cast<const f32x4*>(p) + q);
      const f32x4 mv = load_stream(reinterpret_cast<const f32x4*>(m) + q);
      const f32x4 vv = load_stream(reinterpret_cast<const f32x4*>(v) + q);
      const f32x4 gv = load_stream(reinterpret_cast<const f32x4*>(g) + q);
      float pe[4] = {pv.x, pv.y, pv.z, pv.w}, me[4] = {mv.x, mv.y, mv.z, mv.w};
      float ve[4] = {vv.x, vv.y, vv.z, vv.w};
      const float ge[4] = {gv.x, gv.y, gv.z, gv.w};
#pragma unroll
      for (int k = 0; k < 4; ++k) adam_update_f32(pe[k], me[k], ve[k], ge[k], c);
      store_stream(reinterpret_cast<f32x4*>(p) + q, f32x4{pe[0], pe[1], pe[2], pe[3]});
      store_stream(reinterpret_cast<f32x4*>(m) + q, f32x4{me[0], me[1], me[2], me[3]});
      store_stream(reinterpret_cast<f32x4*>(v) + q, f32x4{ve[0], ve[1], ve[2], ve[3]});
    }
    // the last n % 4 elements
    for (int64_t e = nvec * 4 + threadIdx.x; blockIdx.x == 0 && e < n; e += kDenseBlock) {
      float pe = p[e], me = m[e], ve = v[e];
      adam_update_f32(pe, me, ve, g[e], c);
      p[e] = pe;
      m[e] = me;
      v[e] = ve;
    }
  } else {
    for (int64_t e = t0; e < n; e += stride) {
      float pe = p[e], me = m[e], ve = v[e];
      adam_update_f32(pe, me, ve, g[e], c);
      p[e] = pe;
      m[e] = me;
      v[e] = ve;
    }
  }
}

hipError_t launch_dense_adagrad(float* p, float* a, const float* g, int64_t n, double lr, double eps,
                                hipStream_t stream) {
  if (n <= 0) return hipSuccess;
  int64_t blocks = ceil_div(ceil_div(n, 4), kDenseBlock);
  if (blocks > kApplyMaxBlocks) blocks = kApplyMaxBlocks;
  hipLaunchKernelGGL(dense_adagrad_kernel, dim3((unsigned)blocks), dim3(kDenseBlock), 0, stream, p,
                     a, g, n, opt_f32(lr, eps));
  return hipGetLastError();
}

hipError_t launch_dense_adam(float* p, float* m, float* v, const float* g, int64_t n,
                             const AdamParams& hp, hipStream_t stream) {
  if (n <= 0) return hipSuccess;
  int64_t blocks = ceil_div(ceil_div(n, 4), kDenseBlock);
  if (blocks > kApplyMaxBlocks) blocks = kApplyMaxBlocks;
  hipLaunchKernelGGL(dense_adam_kernel, dim3((unsigned)blocks), dim3(kDenseBlock), 0, stream, p, m,
                     v, g, n, opt_f32(hp.lr, hp.eps, hp.beta1, hp.beta2, hp.bc1, hp.bc2));
  return hipGetLastError();
}

}  // namespace gba
