// adapter_gemm.hip - the first, reducing product of the low-rank adapter path:
//   forward   T = X L        (X [M, K] activations, L [K, r] fp16, "NN")
//   backward  U = dY R^T     (dY [M, N],           R [r, N] fp16, "NT")
// Output fp32 [M, r]. 64 x 64 output tiles on 16x16x32 fp16 MFMA; the reduction may be split
// across blocks, in which case the last block to finish a tile sums the partial tiles in a
// fixed order (deterministic) and resets the tile's counter to zero.
#include "slim_device.h"
#include "slim_launch.h"

namespace {

constexpr int kT = 64;      // tile edge (rows of A = m, columns = adapter rank j)
constexpr int kBK = 64;     // reduction per LDS stage
constexpr int kLd = kBK + 8;

template <bool NT>
__global__ void __launch_bounds__(256)
k_adapter_gemm(const uint16_t* __restrict__ A, int a_bf16, int64_t M, int64_t Kd, const uint16_t* __restrict__ Bsrc,
               int64_t r, int64_t slice, int split, float* __restrict__ out, float* __restrict__ part,
               uint32_t* __restrict__ counters) {
  __shared__ __attribute__((aligned(16))) _Float16 As[kT][kLd];
  __shared__ __attribute__((aligned(16))) _Float16 Bt[kT][kLd];   // [j][k]
  __shared__ int last_flag;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave & 1, wj = wave >> 1;
  const int64_t m0 = (int64_t)blockIdx.x * kT, j0 = (int64_t)blockIdx.y * kT;
  const int s = blockIdx.z;
  const int64_t kbeg = (int64_t)s * slice, kend = min(Kd, kbeg + slice);
  f4_t acc[2][2];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b) acc[a][b] = f4_t{0.f, 0.f, 0.f, 0.f};

  for (int64_t k = kbeg; k < kend; k += kBK) {
    // A tile: 64 rows x 64 k = 512 vectors of 8
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int idx = tid + 256 * i, row = idx >> 3, kc = idx & 7;
      const int64_t gm = m0 + row, gk = k + 8 * kc;
      u32x4_t v = {0u, 0u, 0u, 0u};
      if (gm < M && gk < kend) v = *reinterpret_cast<const u32x4_t*>(A + gm * Kd + gk);
      *reinterpret_cast<h8_t*>(&As[row][8 * kc]) = load8_as_h(v, a_bf16 != 0);
    }
    // B tile, stored transposed as Bt[j][k]
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int idx = tid + 256 * i;
      if (NT) {  // R [r, Kd]: row j contiguous along k
        const int jr = idx >> 3, kc = idx & 7;
        const int64_t gj = j0 + jr, gk = k + 8 * kc;
        u32x4_t v = {0u, 0u, 0u, 0u};
        if (gj < r && gk < kend) v = *reinterpret_cast<const u32x4_t*>(Bsrc + gj * Kd + gk);
        *reinterpret_cast<u32x4_t*>(&Bt[jr][8 * kc]) = v;
      } else {   // L [Kd, r]: row k contiguous along j -> transpose on the way into LDS
        const int kr = idx >> 3, jc = idx & 7;
        const int64_t gk = k + kr, gj = j0 + 8 * jc;
        u32x4_t v = {0u, 0u, 0u, 0u};
        if (gk < kend && gj < r) v = *reinterpret_cast<const u32x4_t*>(Bsrc + gk * r + gj);
        const h8_t hv = __builtin_bit_cast(h8_t, v);
#pragma unroll
        for (int e = 0; e < 8; ++e) Bt[8 * jc + e][kr] = hv[e];
      }
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < kBK; kk += 32) {
      h8_t af[2], bf[2];
#pragma unroll
      for (int f = 0; f < 2; ++f) {
        af[f] = *reinterpret_cast<const h8_t*>(&As[32 * wm + 16 * f + (lane & 15)][kk + 8 * (lane >> 4)]);
        bf[f] = *reinterpret_cast<const h8_t*>(&Bt[32 * wj + 16 * f + (lane & 15)][kk + 8 * (lane >> 4)]);
      }
#pragma unroll
      for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int b = 0; b < 2; ++b) acc[a][b] = __builtin_amdgcn_mfma_f32_16x16x32_f16(af[a], bf[b], acc[a][b], 0, 0, 0);
    }
    __syncthreads();
  }

  const int tile = blockIdx.x * gridDim.y + blockIdx.y;
  if (split > 1) {
    // partial tile in register order: fully coalesced
    float* dst = part + ((int64_t)s * gridDim.x * gridDim.y + tile) * (kT * kT);
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
      for (int b = 0; b < 2; ++b)
#pragma unroll
        for (int v = 0; v < 4; ++v) dst[(((wave * 2 + a) * 2 + b) * 4 + v) * 64 + lane] = acc[a][b][v];
    __threadfence();
    __syncthreads();
    if (tid == 0) {
      const uint32_t done = atomicAdd(&counters[tile], 1u);
      last_flag = (done == (uint32_t)(split - 1));
    }
    __syncthreads();
    if (!last_flag) return;
    __threadfence();
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
      for (int b = 0; b < 2; ++b) acc[a][b] = f4_t{0.f, 0.f, 0.f, 0.f};
    for (int ss = 0; ss < split; ++ss) {
      const float* src = part + ((int64_t)ss * gridDim.x * gridDim.y + tile) * (kT * kT);
#pragma unroll
      for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int b = 0; b < 2; ++b)
#pragma unroll
          for (int v = 0; v < 4; ++v) acc[a][b][v] += src[(((wave * 2 + a) * 2 + b) * 4 + v) * 64 + lane];
    }
    if (tid == 0) counters[tile] = 0u;
  }
  // D[i][j] of a 16x16 fragment sits at lane (j + 16 * (i / 4)), element i % 4
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      const int64_t gj = j0 + 32 * wj + 16 * b + (lane & 15);
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int64_t gm = m0 + 32 * wm + 16 * a + 4 * (lane >> 4) + v;
        if (gm < M && gj < r) out[gm * r + gj] = acc[a][b][v];
      }
    }
}

}  // namespace

int slim_launch_adapter_gemm(bool nt, const uint16_t* A, int a_bf16, int64_t M, int64_t Kd, const uint16_t* B,
                             int64_t r, const SlimPlan& p, char* ws, hipStream_t s) {
  dim3 grid((unsigned)p.ad_tiles_m, (unsigned)p.ad_tiles_j, (unsigned)p.ad_split);
  float* out = reinterpret_cast<float*>(ws + p.off_t);
  float* part = reinterpret_cast<float*>(ws + p.off_tpart);
  uint32_t* counters = reinterpret_cast<uint32_t*>(ws + p.off_counters);
  if (nt)
    hipLaunchKernelGGL(k_adapter_gemm<true>, grid, dim3(256), 0, s, A, a_bf16, M, Kd, B, r, p.ad_slice, p.ad_split,
                       out, part, counters);
  else
    hipLaunchKernelGGL(k_adapter_gemm<false>, grid, dim3(256), 0, s, A, a_bf16, M, Kd, B, r, p.ad_slice, p.ad_split,
                       out, part, counters);
  return hipGetLastError() == hipSuccess ? SLIM_OK : SLIM_EDEVICE;
}
