// quant.hip - SLiM-Quant's scale search on the GPU (SLiM chapter, "SLiM-Quant quantization
// method": eq. error_summation with eq. quantization_error and eq. clipping_error, evaluated on a
// histogram of |w|; Alg. quantization for the coarse and fine candidate grids).
//
//   k_quant_clear   zero the histogram, the maximum and the status word (a kernel, not a memset,
//                   so that a captured graph replays it)
//   k_quant_absmax  max |w| of the tensor (float bits, compared as unsigned: every value is >= 0),
//                   and a status bit for non-finite weights
//   k_quant_hist    per-block histogram of |w| in LDS, added into the global one; bin
//                   b = floor(|w| bins / amax) exactly (see bin_of)
//   k_quant_cand    E(alpha) = E_quant + E_clip in float64 by the midpoint rule on the bin centres,
//                   one block per candidate: the ten coarse ones and the twenty fine ones around
//                   each of them
//   k_quant_pick    the search's order: the coarse minimum, its fine candidates, the argmin
#include <math.h>

#include "slim_device.h"
#include "slim_host.h"
#include "slim_timing.h"

namespace {

constexpr int kQThreads = 256;
constexpr int kQMaxBins = 20480;           // 80 KiB of LDS counters: two blocks per CU
constexpr int kQHistThreads = 1024;
constexpr int kQCoarse = 10, kQFine = 20;  // candidates of the two grids
constexpr int kQSearchThreads = 512;

__global__ void __launch_bounds__(kQThreads)
k_quant_clear(uint32_t* __restrict__ hist, int bins, uint32_t* __restrict__ amax_bits, int* __restrict__ status) {
  const int t = blockIdx.x * kQThreads + threadIdx.x;
  if (t < bins) hist[t] = 0u;
  if (t == 0) {
    *amax_bits = 0u;
    *status = 0;
  }
}

__global__ void __launch_bounds__(kQThreads)
k_quant_absmax(const float4* __restrict__ W, int64_t n4, uint32_t* __restrict__ amax_bits, int* __restrict__ status) {
  float m = 0.f;
  int bad = 0;
  for (int64_t i = (int64_t)blockIdx.x * kQThreads + threadIdx.x; i < n4; i += (int64_t)gridDim.x * kQThreads) {
    const float4 v = W[i];
    const float w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      if (!__builtin_isfinite(w[p])) bad = 1;
      m = fmaxf(m, fabsf(w[p]));
    }
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) m = fmaxf(m, __shfl_xor(m, off, 64));
  bad = __any(bad) ? 1 : 0;
  __shared__ float wm[kQThreads / 64];
  __shared__ int wb[kQThreads / 64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane == 0) {
    wm[wave] = m;
    wb[wave] = bad;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    float bm = wm[0];
    int bb = wb[0];
    for (int w = 1; w < kQThreads / 64; ++w) {
      bm = fmaxf(bm, wm[w]);
      bb |= wb[w];
    }
    // non-negative floats order like their bit patterns
    atomicMax(amax_bits, __float_as_uint(bm));
    if (bb) atomicOr(status, 1);
  }
}

// floor(a bins / amax) for 0 <= a <= amax, 0 < amax < inf, exactly: a bins is exact in float64 (a
// has 24 significant bits, bins at most 15), so is q amax for any integer q < 2^15; a first guess
// from the reciprocal is corrected by comparing those exact products. The result is clamped to
// [0, bins) whatever a is (a NaN weight, which the call reports, lands in some bin).
__device__ __forceinline__ int bin_of(float a, double bins_d, double amax, double inv_amax, int bins) {
  const double t = (double)a * bins_d;
  const double g = fmin(fmax(floor(t * inv_amax), 0.0), bins_d - 1.0);
  int b = (int)g;
  if ((double)(b + 1) * amax <= t) ++b;
  else if ((double)b * amax > t) --b;
  return b < 0 ? 0 : (b < bins ? b : bins - 1);
}

// Grid-stride over pairs of float4, both loads issued before the counting.
__global__ void __launch_bounds__(kQHistThreads)
k_quant_hist(const float4* __restrict__ W, int64_t n4, int bins, const uint32_t* __restrict__ amax_bits,
             uint32_t* __restrict__ hist) {
  __shared__ uint32_t hs[kQMaxBins];
  for (int b = threadIdx.x; b < bins; b += kQHistThreads) hs[b] = 0u;
  __syncthreads();
  const double amax = (double)__uint_as_float(*amax_bits);
  // all-zero weights: every magnitude in bin 0; an infinite maximum (reported by the call): likewise
  const bool binned = amax > 0.0 && amax < INFINITY;
  const double bins_d = (double)bins, inv = binned ? 1.0 / amax : 0.0;
  auto count4 = [&](const float4 v) {
    const float w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      const int b = binned ? bin_of(fabsf(w[p]), bins_d, amax, inv, bins) : 0;
      atomicAdd(&hs[b], 1u);
    }
  };
  const int64_t stride = (int64_t)gridDim.x * kQHistThreads;
  for (int64_t i = (int64_t)blockIdx.x * kQHistThreads + threadIdx.x; i < n4; i += 2 * stride) {
    const float4 v0 = W[i];
    const bool two = i + stride < n4;
    const float4 v1 = two ? W[i + stride] : make_float4(0.f, 0.f, 0.f, 0.f);
    count4(v0);
    if (two) count4(v1);
  }
  __syncthreads();
  for (int b = threadIdx.x; b < bins; b += kQHistThreads) {
    const uint32_t c = hs[b];
    if (c) atomicAdd(&hist[b], c);
  }
}

// Sum of one value per thread over the block, in a fixed order (wave butterflies, then the
// waves' sums in wave order); every thread gets the result.
__device__ double block_sum(double v, double* red) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  __syncthreads();
  if (lane == 0) red[wave] = v;
  __syncthreads();
  double s = 0.0;
  for (int w = 0; w < kQSearchThreads / 64; ++w) s += red[w];
  return s;
}

// The search's float64 expressions are evaluated as written, each product rounded before the sum
// it feeds (no fused multiply-add), so that every candidate and every per-bin term is the same
// number a plain float64 evaluation gives; only the order of the final sums differs.
#pragma clang fp contract(off)

// E(alpha) of Alg. quantization on the histogram: bin b stands for its count at the centre
// (b + 1/2) amax / bins; magnitudes up to alpha reconstruct on the grid of step alpha / qmax
// (eq. quantization_error), larger ones as alpha (eq. clipping_error).
// The thread's counts, bins b = threadIdx.x + kQSearchThreads i, sit in registers (loaded once for
// all candidates: a loop that loaded each count as it went waited for every load in turn).
constexpr int kQPerThread = kQMaxBins / kQSearchThreads;
__device__ double estimate_error(const uint32_t (&cnts)[kQPerThread], int bins, double amax, double alpha, double qmax,
                                 double total, double* red) {
  const double width = amax / (double)bins;
  const double delta = alpha / qmax;
  double sq = 0.0, sc = 0.0;
  // branch-free: a zero count, or the side a centre is not on, adds +0.0, which leaves a
  // non-negative sum unchanged; one bin at a time (the scheduler would otherwise interleave all the
  // divisions and spill)
#pragma unroll
  for (int i = 0; i < kQPerThread; ++i) {
    const int b = threadIdx.x + kQSearchThreads * i;
    const double cnt = (double)cnts[i];
    const double c = ((double)b + 0.5) * width;
    const double dq = delta * rint(c / delta) - c;
    const double dc = alpha - c;
    const bool in = c <= alpha;
    sq += in ? cnt * (dq * dq) : 0.0;
    sc += in ? 0.0 : cnt * (dc * dc);
    __builtin_amdgcn_sched_barrier(0);
  }
  const double q = block_sum(sq, red);
  const double s = block_sum(sc, red);
  return q / total + s / total;
}

// Every candidate the search can evaluate, one block each: the ten coarse ones i amax / 10, and
// for each of them the twenty fine ones (i amax / 10 - amax / 10) + j amax / 100 that the search
// evaluates if i is the coarse minimum (kQCand blocks; a non-positive one is marked NaN). Each
// block sums its candidate exactly as a single block evaluating the candidates in turn would, so
// the errors do not depend on this split; k_quant_pick then walks the search's order.
constexpr int kQCand = kQCoarse + kQCoarse * kQFine;
__global__ void __launch_bounds__(kQSearchThreads)
k_quant_cand(const uint32_t* __restrict__ hist, int bins, const uint32_t* __restrict__ amax_bits, int bits,
             double total, double* __restrict__ cand) {
  __shared__ double red[kQSearchThreads / 64];
  const double amax = (double)__uint_as_float(*amax_bits);
  if (amax == 0.0) return;
  const double qmax = (double)((1 << (bits - 1)) - 1);
  const double eta_low = amax / (double)kQCoarse;
  const int c = blockIdx.x;
  double a;
  if (c < kQCoarse) {
    a = (double)(c + 1) * eta_low;
  } else {
    const int i = (c - kQCoarse) / kQFine + 1, j = (c - kQCoarse) % kQFine;
    const double alpha_low = (double)i * eta_low, eta_high = eta_low / 10.0;
    a = (alpha_low - eta_low) + (double)j * eta_high;
  }
  double e = __builtin_nan("");
  if (a > 0.0) {     // uniform per block
    uint32_t cnts[kQPerThread];
#pragma unroll
    for (int i = 0; i < kQPerThread; ++i) {
      const int b = threadIdx.x + kQSearchThreads * i;
      cnts[i] = b < bins ? hist[b] : 0u;
    }
    e = estimate_error(cnts, bins, amax, a, qmax, total, red);
  }
  if (threadIdx.x == 0) {
    cand[2 * c] = a;
    cand[2 * c + 1] = e;
  }
}

// out: [0] alpha*, [1] E(alpha*), [2] amax, [3] candidates evaluated C, [4 + 2i] alpha_i,
// [5 + 2i] E(alpha_i) in evaluation order: the ten coarse candidates, then the positive fine ones
// around the first coarse minimum; alpha* is the first candidate of least error. One thread.
__global__ void __launch_bounds__(64)
k_quant_pick(const uint32_t* __restrict__ amax_bits, const double* __restrict__ cand, double* __restrict__ out) {
  if (threadIdx.x != 0) return;
  const double amax = (double)__uint_as_float(*amax_bits);
  if (amax == 0.0) {
    out[0] = 0.0;
    out[1] = 0.0;
    out[2] = 0.0;
    out[3] = 0.0;
    return;
  }
  int n = 0, ibest = 0;
  double best_a = 0.0, best_e = 0.0;
  for (int i = 0; i < kQCoarse; ++i) {
    const double a = cand[2 * i], e = cand[2 * i + 1];
    out[4 + 2 * n] = a;
    out[5 + 2 * n] = e;
    if (n == 0 || e < best_e) {
      best_a = a;
      best_e = e;
      ibest = i;
    }
    ++n;
  }
  for (int j = 0; j < kQFine; ++j) {
    const int c = kQCoarse + ibest * kQFine + j;
    const double a = cand[2 * c], e = cand[2 * c + 1];
    if (!(a > 0.0)) continue;
    out[4 + 2 * n] = a;
    out[5 + 2 * n] = e;
    if (e < best_e) {
      best_a = a;
      best_e = e;
    }
    ++n;
  }
  out[0] = best_a;
  out[1] = best_e;
  out[2] = amax;
  out[3] = (double)n;
}

}  // namespace

extern "C" int slim_quant_bins(int64_t N, int64_t K) {
  if (N < 1 || K < 1) return 512;
  const int64_t p = N * K / 1000;
  return (int)(p < 512 ? 512 : (p > 20000 ? 20000 : p));
}

extern "C" int slim_quant_search(const float* W, int64_t count, int bits, int64_t bins, uint32_t* hist,
                                 double* out, void* stream) {
  if (!W || !hist || !out) return SLIM_EINVAL;
  if (count < 4 || count % 4 || bits < 2 || bits > 8 || bins < 1 || bins > kQMaxBins) return SLIM_ESHAPE;
  if (count >= ((int64_t)1 << 40)) return SLIM_EUNSUPPORTED;
  if (!slim_aligned16(W) || ((uintptr_t)hist & 3u) || ((uintptr_t)out & 7u)) return SLIM_EALIGN;
  hipStream_t s = (hipStream_t)stream;
  // maximum, status and the candidates' errors live in one small device allocation for the
  // duration of the call
  uint32_t* d_aux = nullptr;
  if (hipMalloc(&d_aux, 16 + 2 * kQCand * sizeof(double)) != hipSuccess) return SLIM_EDEVICE;
  uint32_t* d_amax = d_aux;
  int* d_status = reinterpret_cast<int*>(d_aux + 1);
  double* d_cand = reinterpret_cast<double*>(d_aux + 4);
  int h_status = 0, rc = SLIM_OK;
  const int64_t n4 = count / 4;
  int64_t grid = (n4 + kQThreads - 1) / kQThreads;
  if (grid > 2048) grid = 2048;      // grid-stride: eight blocks per CU
  int64_t hgrid = (n4 + kQHistThreads - 1) / kQHistThreads;
  if (hgrid > 512) hgrid = 512;      // two blocks per CU
  do {
    {
      SlimKernelTimer timer("quant_clear", s);
      SLIM_LAUNCH(timer, k_quant_clear, dim3((unsigned)((bins + kQThreads - 1) / kQThreads)), dim3(kQThreads), s,
                  hist, (int)bins, d_amax, d_status);
    }
    {
      SlimKernelTimer timer("quant_absmax", s);
      SLIM_LAUNCH(timer, k_quant_absmax, dim3((unsigned)grid), dim3(kQThreads), s,
                  reinterpret_cast<const float4*>(W), n4, d_amax, d_status);
    }
    {
      SlimKernelTimer timer("quant_hist", s);
      SLIM_LAUNCH(timer, k_quant_hist, dim3((unsigned)hgrid), dim3(kQHistThreads), s,
                  reinterpret_cast<const float4*>(W), n4, (int)bins, (const uint32_t*)d_amax, hist);
    }
    {
      SlimKernelTimer timer("quant_search", s);
      SLIM_LAUNCH(timer, k_quant_cand, dim3(kQCand), dim3(kQSearchThreads), s, (const uint32_t*)hist, (int)bins,
                  (const uint32_t*)d_amax, bits, (double)count, d_cand);
    }
    {
      SlimKernelTimer timer("quant_pick", s);
      SLIM_LAUNCH(timer, k_quant_pick, dim3(1), dim3(64), s, (const uint32_t*)d_amax, (const double*)d_cand, out);
    }
    if (hipGetLastError() != hipSuccess) { rc = SLIM_EDEVICE; break; }
    if (hipMemcpyAsync(&h_status, d_status, sizeof(int), hipMemcpyDeviceToHost, s) != hipSuccess ||
        hipStreamSynchronize(s) != hipSuccess) { rc = SLIM_EDEVICE; break; }
    if (h_status & 1) rc = SLIM_ENONFINITE;
  } while (0);
  (void)hipFree(d_aux);
  return rc;
}
