// adapter_gemm.hip - the adapter's first, reducing product for large M:
//   tm = act Q^T with act [M, red] fp16 and Q [r, red] fp16 row-major:
//   forward  T = X L      (Q = L^T, from slim_pack_adapter)
//   backward U = dY R^T   (Q = R as given)
// Result fp16 (it only feeds the fp16 MFMA of the second product), in 32 x 16 tiles: element
// (m, j) at ((m / 32) (r / 16) + j / 16) 512 + (m % 32) 16 + j % 16, so that one 16-rank step of
// a 32-row operand fragment is 1 KB of contiguous memory.
//
// 128 x 128 output tiles; wave (wm, wr) of the block's four owns rows 64 wm .. + 63 and ranks
// 64 wr .. + 63 as 2 x 2 fragments of 32x32x16 fp16 MFMA. Both operands are contiguous along the
// reduction, so both stream the same way: per 64-wide reduction chunk, 128 rows x 128 B of each go
// straight from memory to LDS (direct loads, 16 B per lane) into a ring of two stages, one chunk
// ahead (64 KB, so that two blocks share a CU and one's MFMAs overlap the other's loads, barriers
// and conversions: a block runs one wave per SIMD and its issue work, not memory, sets its pace);
// LDS rows are 128 B with the 16-byte column index XOR-swizzled by the row, so that
// fragment reads (32 rows at one column) hit distinct banks. Rows past M or r read as zero (the
// loads go through buffer resources whose extent ends with the matrix).
// The reduction may be split across blocks: each split then stores its fp32 partial in the same
// tiled order with plain stores, and k_adapter_finish (sparse_gemm.hip) sums the splits in order
// (deterministic) after the kernel boundary has made them visible.
// The activations are the fp16 copy k_rowprep writes, each row scaled by a power of two, so the
// result is T (or U) with the same row scaling; the tile kernel unscales its fp32 output.
#include <type_traits>

#include "slim_device.h"
#include "slim_launch.h"
#include "slim_timing.h"

namespace {

constexpr int kT = 128;     // output tile edge (m and j)
constexpr int kBK = 64;     // reduction per chunk
// direct loads per thread per chunk: 4 for the activation rows, 4 for the Q rows
constexpr int kLoads = 8;

__global__ void __launch_bounds__(256)
k_adapter_gemm(const uint16_t* __restrict__ A, int64_t M, int64_t Kd, const uint16_t* __restrict__ Q, int64_t r,
               int64_t slice, int split, uint16_t* __restrict__ out, float* __restrict__ part) {
  __shared__ __attribute__((aligned(16))) _Float16 as0[kT][kBK], as1[kT][kBK];
  __shared__ __attribute__((aligned(16))) _Float16 bs0[kT][kBK], bs1[kT][kBK];
  auto as_at = [&](int stg) -> _Float16(*)[kBK] { return stg == 0 ? as0 : as1; };
  auto bs_at = [&](int stg) -> _Float16(*)[kBK] { return stg == 0 ? bs0 : bs1; };
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave & 1, wr = wave >> 1, ha = lane >> 5;
  const int64_t m0 = (int64_t)blockIdx.x * kT, j0 = (int64_t)blockIdx.y * kT;
  const int s = blockIdx.z;
  const int64_t kbeg = (int64_t)s * slice, kend = min(Kd, kbeg + slice);
  const int nst = (int)((kend - kbeg) / kBK);   // slice and Kd are multiples of 64

  // direct loads: wave w writes rows 32 w .. 32 w + 31 of each operand tile, eight per load
  // (lane L: row + L / 8, LDS column slot L % 8 holding column (L % 8) ^ (row % 8))
  const rsrc_t ra = make_rsrc(A + m0 * Kd, (M - m0 < kT ? M - m0 : kT) * Kd * 2);
  const rsrc_t rq = make_rsrc(Q + j0 * Kd, (r - j0 < kT ? r - j0 : kT) * Kd * 2);
  const int lrow = lane >> 3, lslot = lane & 7;
  uint32_t xo[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int row = 32 * wave + 8 * i + lrow;
    xo[i] = ((uint32_t)row * (uint32_t)Kd + 8u * (uint32_t)(lslot ^ (row & 7))) * 2u;
  }
  auto dma = [&](int t, int stg) {
    const int ko = (int)((kbeg + (int64_t)(t < nst ? t : nst - 1) * kBK) * 2);
#pragma unroll
    for (int i = 0; i < 4; ++i)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(ra, (lds_ptr_t)&as_at(stg)[32 * wave + 8 * i][0], 16, xo[i], ko, 0, 0);
#pragma unroll
    for (int i = 0; i < 4; ++i)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rq, (lds_ptr_t)&bs_at(stg)[32 * wave + 8 * i][0], 16, xo[i], ko, 0, 0);
  };

  f16_t acc[2][2];
#pragma unroll
  for (int x = 0; x < 2; ++x)
#pragma unroll
    for (int y = 0; y < 2; ++y)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[x][y][v] = 0.f;

  // fragment read of step t: row `row` of a stage, 16-byte slot (2 t + L / 32) ^ (row % 8)
  auto frag = [&](const _Float16 (*tile)[kBK], int row, int t) {
    return *reinterpret_cast<const h8_t*>(&tile[row][8 * ((2 * t + ha) ^ (row & 7))]);
  };
  // steps of a chunk: 16-wide reductions; the fragments of step st + 1 are read while step st's
  // MFMAs run
  auto chunk = [&](int t, auto zc) {
    constexpr int z = decltype(zc)::value;
    // chunk t has landed once nothing is outstanding (the previous chunk's copy stores included);
    // with this wave's LDS reads returned, after the barrier no wave reads the stage refilled below
    __builtin_amdgcn_s_waitcnt(vmcnt_lgkm0_wait(0));
    asm volatile("s_barrier" ::: "memory");
    dma(t + 1, (z + 1) % 2);
    h8_t af[2][2], bf[2][2];
#pragma unroll
    for (int f = 0; f < 2; ++f) {
      af[0][f] = frag(as_at(z), 64 * wm + 32 * f + (lane & 31), 0);
      bf[0][f] = frag(bs_at(z), 64 * wr + 32 * f + (lane & 31), 0);
    }
#pragma unroll
    for (int st = 0; st < kBK / 16; ++st) {
      if (st + 1 < kBK / 16) {
#pragma unroll
        for (int f = 0; f < 2; ++f) {
          af[(st + 1) & 1][f] = frag(as_at(z), 64 * wm + 32 * f + (lane & 31), st + 1);
          bf[(st + 1) & 1][f] = frag(bs_at(z), 64 * wr + 32 * f + (lane & 31), st + 1);
        }
      }
#pragma unroll
      for (int x = 0; x < 2; ++x)
#pragma unroll
        for (int y = 0; y < 2; ++y) acc[x][y] = mfma32(af[st & 1][x], bf[st & 1][y], acc[x][y]);
    }
  };
  dma(0, 0);
  int t0 = 0;
  for (; t0 + 2 <= nst; t0 += 2) {
    chunk(t0, std::integral_constant<int, 0>{});
    chunk(t0 + 1, std::integral_constant<int, 1>{});
  }
  if (t0 < nst) chunk(t0, std::integral_constant<int, 0>{});
  // the ring's last loads (repeats of the final chunk) must land before the block's LDS is released
  __builtin_amdgcn_s_waitcnt(0);

  // D[i][j] of a 32x32 fragment: lane j + 32 * ((i / 4) % 2), element 4 * (i / 8) + i % 4; the
  // tiled index of (m, j) is ((m / 32) (r / 16) + j / 16) 512 + (m % 32) 16 + j % 16
  float* pdst = part + (int64_t)s * ((M + 31) / 32 * 32) * r;
#pragma unroll
  for (int y = 0; y < 2; ++y) {
    const int64_t gj = j0 + 64 * wr + 32 * y + (lane & 31);
    if (gj >= r) continue;
#pragma unroll
    for (int x = 0; x < 2; ++x)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int64_t gm = m0 + 64 * wm + 32 * x + 8 * (v >> 2) + 4 * ha + (v & 3);
        if (gm >= M) continue;
        const int64_t ti = ((gm >> 5) * (r >> 4) + (gj >> 4)) * 512 + (gm & 31) * 16 + (gj & 15);
        if (split > 1) pdst[ti] = acc[x][y][v];
        else out[ti] = __builtin_bit_cast(uint16_t, (_Float16)acc[x][y][v]);
      }
  }
}

}  // namespace

int slim_launch_adapter_gemm(const uint16_t* A, int64_t M, int64_t Kd, const uint16_t* Q, int64_t r, const SlimPlan& p,
                             char* ws, hipStream_t s) {
  dim3 grid((unsigned)p.ad_tiles_m, (unsigned)p.ad_tiles_j, (unsigned)p.ad_split);
  uint16_t* out = reinterpret_cast<uint16_t*>(ws + p.off_t);
  float* part = reinterpret_cast<float*>(ws + p.off_tpart);
  SlimKernelTimer timer("adapter_gemm", s);
  SLIM_LAUNCH(timer, k_adapter_gemm, grid, dim3(256), s, A, M, Kd, Q, r, p.ad_slice, p.ad_split, out, part);
  return hipGetLastError() == hipSuccess ? SLIM_OK : SLIM_EDEVICE;
}
