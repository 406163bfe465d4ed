// adapter_gemm.hip - the adapter's first, reducing product for large M:
//   tm = act Q^T with act [M, red] (bf16/fp16) and Q [r, red] fp16 row-major:
//   forward  T = X L      (Q = L^T, from slim_pack_adapter)
//   backward U = dY R^T   (Q = R as given)
// Result fp16 (it only feeds the fp16 MFMA of the second product), in 32 x 16 tiles: element
// (m, j) at ((m / 32) (r / 16) + j / 16) 512 + (m % 32) 16 + j % 16, so that one 16-rank step of
// a 32-row operand fragment is 1 KB of contiguous memory. 64 x 64 output tiles
// on 16x16x32 fp16 MFMA, 64-wide reduction stages double-buffered in LDS and staged through
// registers one stage ahead. The reduction may be split across blocks; the last block of a tile
// sums the partials in split order (deterministic) through device-scope accesses.
#include "slim_device.h"
#include "slim_launch.h"
#include "slim_timing.h"

namespace {

constexpr int kT = 64;      // output tile edge (m and j)
constexpr int kBK = 64;     // reduction per stage
constexpr int kLd = kBK + 8;

__global__ void __launch_bounds__(256)
k_adapter_gemm(const uint16_t* __restrict__ A, int a_bf16, int64_t M, int64_t Kd, const uint16_t* __restrict__ Bsrc,
               int64_t r, int64_t slice, int split, uint16_t* __restrict__ out, float* __restrict__ part,
               uint32_t* __restrict__ counters) {
  __shared__ __attribute__((aligned(16))) _Float16 As[2][kT][kLd];
  __shared__ __attribute__((aligned(16))) _Float16 Bs[2][kT][kLd];   // [j][k]
  __shared__ int last_flag;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave & 1, wj = wave >> 1;
  const int g = lane >> 4;
  const int64_t m0 = (int64_t)blockIdx.x * kT, j0 = (int64_t)blockIdx.y * kT;
  const int s = blockIdx.z;
  const int64_t kbeg = (int64_t)s * slice, kend = min(Kd, kbeg + slice);
  const int nst = (int)((kend - kbeg + kBK - 1) / kBK);
  const bool bf16 = a_bf16 != 0;

  // loads are unconditional from clamped addresses; out-of-range elements are zeroed when stored
  // to LDS (a conditional load would make the compiler wait for it at the branch join)
  u32x4_t ar[2], br[2];
  bool aok[2], bok[2];
  auto load = [&](int t) {
    const int64_t k = kbeg + (int64_t)t * kBK;
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int q = tid + 256 * i;
      {  // A tile: 64 rows of m x 8 vectors
        const int row = q >> 3, kc = q & 7;
        const int64_t gm = m0 + row, gk = k + 8 * kc;
        aok[i] = gm < M && gk < kend;
        ar[i] = *reinterpret_cast<const u32x4_t*>(A + (gm < M ? gm : M - 1) * Kd + (gk < kend ? gk : kend - 8));
      }
      {  // Q [r, Kd]: row j contiguous along k
        const int jr = q >> 3, kc = q & 7;
        const int64_t gj = j0 + jr, gk = k + 8 * kc;
        bok[i] = gj < r && gk < kend;
        br[i] = *reinterpret_cast<const u32x4_t*>(Bsrc + (gj < r ? gj : r - 1) * Kd + (gk < kend ? gk : kend - 8));
      }
    }
  };
  auto store = [&](int buf) {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int q = tid + 256 * i;
      *reinterpret_cast<h8_t*>(&As[buf][q >> 3][8 * (q & 7)]) = aok[i] ? load8_as_h(ar[i], bf16) : zero_h8();
      *reinterpret_cast<u32x4_t*>(&Bs[buf][q >> 3][8 * (q & 7)]) = bok[i] ? br[i] : u32x4_t{0u, 0u, 0u, 0u};
    }
  };

  f4_t acc[2][2];
#pragma unroll
  for (int x = 0; x < 2; ++x)
#pragma unroll
    for (int y = 0; y < 2; ++y) acc[x][y] = f4_t{0.f, 0.f, 0.f, 0.f};

  if (nst > 0) {
    load(0);
    store(0);
    __syncthreads();
    if (nst > 1) load(1);
  }
  for (int t = 0; t < nst; ++t) {
    const int buf = t & 1;
#pragma unroll
    for (int kk = 0; kk < kBK; kk += 32) {
      h8_t af[2], bf[2];
#pragma unroll
      for (int f = 0; f < 2; ++f) {
        af[f] = *reinterpret_cast<const h8_t*>(&As[buf][32 * wm + 16 * f + (lane & 15)][kk + 8 * g]);
        bf[f] = *reinterpret_cast<const h8_t*>(&Bs[buf][32 * wj + 16 * f + (lane & 15)][kk + 8 * g]);
      }
#pragma unroll
      for (int x = 0; x < 2; ++x)
#pragma unroll
        for (int y = 0; y < 2; ++y) acc[x][y] = mfma16(af[x], bf[y], acc[x][y]);
    }
    if (t + 1 < nst) store(buf ^ 1);
    __syncthreads();
    if (t + 2 < nst) load(t + 2);
  }

  const int tile = blockIdx.x * gridDim.y + blockIdx.y;
  if (split > 1) {
    float* dst = part + ((int64_t)s * gridDim.x * gridDim.y + tile) * (kT * kT);
#pragma unroll
    for (int x = 0; x < 2; ++x)
#pragma unroll
      for (int y = 0; y < 2; ++y)
#pragma unroll
        for (int v = 0; v < 4; ++v) st_dev(dst + (((wave * 2 + x) * 2 + y) * 4 + v) * 64 + lane, acc[x][y][v]);
    drain_stores();
    __syncthreads();
    if (tid == 0) last_flag = counter_arrive(&counters[tile]) == (uint32_t)(split - 1);
    __syncthreads();
    if (!last_flag) return;
#pragma unroll
    for (int x = 0; x < 2; ++x)
#pragma unroll
      for (int y = 0; y < 2; ++y) acc[x][y] = f4_t{0.f, 0.f, 0.f, 0.f};
    for (int ss = 0; ss < split; ++ss) {
      const float* src = part + ((int64_t)ss * gridDim.x * gridDim.y + tile) * (kT * kT);
      float pv[16];
#pragma unroll
      for (int e = 0; e < 16; ++e) pv[e] = ld_dev(src + (wave * 16 + e) * 64 + lane);
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[e >> 3][(e >> 2) & 1][e & 3] += pv[e];
    }
    if (tid == 0) counter_reset(&counters[tile]);
  }
  // D[i][j] of a 16x16 fragment sits at lane (j + 16 * (i / 4)), element i % 4
#pragma unroll
  for (int x = 0; x < 2; ++x)
#pragma unroll
    for (int y = 0; y < 2; ++y) {
      const int64_t gj = j0 + 32 * wj + 16 * y + (lane & 15);
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int64_t gm = m0 + 32 * wm + 16 * x + 4 * g + v;
        if (gm < M && gj < r)
          out[((gm >> 5) * (r >> 4) + (gj >> 4)) * 512 + (gm & 31) * 16 + (gj & 15)] =
              __builtin_bit_cast(uint16_t, (_Float16)acc[x][y][v]);
      }
    }
}

}  // namespace

int slim_launch_adapter_gemm(const uint16_t* A, int a_bf16, int64_t M, int64_t Kd, const uint16_t* Q, int64_t r,
                             const SlimPlan& p, char* ws, hipStream_t s) {
  dim3 grid((unsigned)p.ad_tiles_m, (unsigned)p.ad_tiles_j, (unsigned)p.ad_split);
  uint16_t* out = reinterpret_cast<uint16_t*>(ws + p.off_t);
  float* part = reinterpret_cast<float*>(ws + p.off_tpart);
  uint32_t* counters = reinterpret_cast<uint32_t*>(ws + p.off_counters);
  SlimKernelTimer timer("adapter_gemm", s);
  SLIM_LAUNCH(timer, k_adapter_gemm, grid, dim3(256), s, A, a_bf16, M, Kd, Q, r, p.ad_slice, p.ad_split, out, part,
              counters);
  return hipGetLastError() == hipSuccess ? SLIM_OK : SLIM_EDEVICE;
}
