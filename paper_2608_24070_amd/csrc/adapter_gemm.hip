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
  // XCD-aware order: block b runs on XCD b % 8 (workgroups are dealt round robin), and XCD x takes
  // positions [x Q, (x + 1) Q) of an order that walks splits, then m tiles, then j tiles, so that the
  // blocks of one XCD share one split's slice of Q and read each activation tile once from its L2
  const int64_t tm = (M + kT - 1) / kT, tj = (r + kT - 1) / kT, total = tm * tj * split;
  const int64_t Qx = (total + 7) / 8;
  const int64_t pos = (int64_t)(blockIdx.x % 8) * Qx + blockIdx.x / 8;
  if (pos >= total) return;
  const int s = (int)(pos / (tm * tj));
  const int64_t rem = pos - (int64_t)s * tm * tj;
  const int64_t m0 = rem / tj * kT, j0 = rem % tj * kT;
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

// Wide variant for long reductions at large M and r a multiple of 256: 256 (m) x 256 (j) tiles of
// 8 waves, two per SIMD, wave (wm, wj) owning rows 128 wm .. + 127 and ranks 64 wj .. + 63 (4 x 2
// fragments): half the operand bytes per flop of the 128 x 128 tile. Per 32-wide reduction chunk,
// 256 rows x 64 B of each operand go to LDS by direct loads into a ring of four stages three ahead
// (128 KiB, one block per CU); LDS rows are 64 B with the 16-byte slot XOR-swizzled by (row / 4) % 4,
// so the eight consecutive rows a quarter-wave reads hit distinct banks. Reads are written out
// (ds_read_b128, one per fragment and step) with explicit waits, the next step's spread over the
// current step's MFMAs, and the chunk barrier sits between a chunk's two steps. Same outputs as
// k_adapter_gemm (fp16 T, or fp32 split partials, in the tiled order).
constexpr int kWT = 256, kWK = 32, kWThreads = 512, kWRing = 4;

__global__ void __launch_bounds__(kWThreads)
k_adapter_gemm_wide(const uint16_t* __restrict__ A, int64_t M, int64_t Kd, const uint16_t* __restrict__ Q, int64_t r,
                    int64_t slice, int split, uint16_t* __restrict__ out, float* __restrict__ part) {
  // the ring: activation chunks [m][32] in slots of 16 KiB at 0, Q chunks [j][32] at 64 KiB
  constexpr uint32_t kSlot = kWT * kWK * 2, kQBase = kWRing * kSlot;
  __shared__ __attribute__((aligned(16))) uint8_t lds[2 * kWRing * kSlot];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave & 1, wj = wave >> 1, ha = lane >> 5;
  const int64_t m0 = (int64_t)blockIdx.x * kWT, j0 = (int64_t)blockIdx.y * kWT;
  const int s = blockIdx.z;
  const int64_t kbeg = (int64_t)s * slice, kend = min(Kd, kbeg + slice);
  const int64_t nch = (kend - kbeg) / kWK;   // slice and Kd are multiples of 32

  // direct loads: each wave loads two 1 KiB pieces (16 rows, p = 2 wave + i) of each operand per
  // chunk; lane L writes LDS bytes 16 L of the piece, row 16 p + L / 4 at physical slot L % 4, which
  // holds logical slot (L % 4) ^ ((row / 4) % 4). Rows past M or r read as zero.
  const rsrc_t ra = make_rsrc(A + m0 * Kd, (M - m0 < kWT ? M - m0 : kWT) * Kd * 2);
  const rsrc_t rq = make_rsrc(Q + j0 * Kd, (r - j0 < kWT ? r - j0 : kWT) * Kd * 2);
  uint32_t vo[2];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int row = 16 * (2 * wave + i) + (lane >> 2), ls = (lane & 3) ^ ((row >> 2) & 3);
    vo[i] = ((uint32_t)row * (uint32_t)Kd + 8u * (uint32_t)ls) * 2u;
  }
  auto issue = [&](int64_t c, auto zc) {
    const uint32_t so = (uint32_t)((kbeg + (c < nch ? c : nch - 1) * kWK) * 2);   // past the end: a dead slot
    constexpr uint32_t z = decltype(zc)::value;
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const uint32_t o = z * kSlot + (uint32_t)(2 * wave + i) * 1024u;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(ra, (lds_ptr_t)&lds[o], 16, vo[i], so, 0, 0);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rq, (lds_ptr_t)&lds[kQBase + o], 16, vo[i], so, 0, 0);
    }
  };

  f16_t acc[4][2];
#pragma unroll
  for (int x = 0; x < 4; ++x)
#pragma unroll
    for (int y = 0; y < 2; ++y)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[x][y][v] = 0.f;

  auto rd = [](uint32_t addr, auto oc) -> u32x4_t {
    u32x4_t v;
    asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(v) : "v"(addr), "i"(decltype(oc)::value));
    return v;
  };
  // per-lane fragment addresses in slot 0 for step 0: row (base + L % 32), logical slot L / 32;
  // step 1 reads logical slots 2, 3, i.e. physical slot ^ 2: an immediate offset of +32 or -32 bytes
  // would depend on the row, so the step-1 addresses are kept too
  const uint32_t lb = (uint32_t)(uintptr_t)(lds_ptr_t)&lds[0];
  uint32_t aa[4][2], bb[2][2];
  auto off_of = [&](int row, int slot) { return (uint32_t)row * 64u + 16u * (uint32_t)(slot ^ ((row >> 2) & 3)); };
#pragma unroll
  for (int st = 0; st < 2; ++st) {
#pragma unroll
    for (int x = 0; x < 4; ++x) aa[x][st] = lb + off_of(128 * wm + 32 * x + (lane & 31), 2 * st + ha);
#pragma unroll
    for (int y = 0; y < 2; ++y) bb[y][st] = lb + kQBase + off_of(64 * wj + 32 * y + (lane & 31), 2 * st + ha);
  }
  struct Frags {
    u32x4_t a[4], b[2];
  };
  auto landed = [](Frags& F) {
    asm volatile("s_waitcnt lgkmcnt(0)"
                 : "+v"(F.a[0]), "+v"(F.a[1]), "+v"(F.a[2]), "+v"(F.a[3]), "+v"(F.b[0]), "+v"(F.b[1]));
  };
  // MFMAs I0 .. I1 - 1 of the step in F (i = 2 x + y); with RD the six reads of the step N (slot z,
  // step st) go one before each of the first six MFMAs of the range
  auto mma_rng = [&](const Frags& F, Frags& N, auto zc, auto stc, auto i0c, auto i1c, auto rdc) {
    using off = std::integral_constant<uint32_t, decltype(zc)::value * kSlot>;
    constexpr int st = decltype(stc)::value;
    constexpr int I0 = decltype(i0c)::value, I1 = decltype(i1c)::value;
#pragma unroll
    for (int i = I0; i < I1; ++i) {
      const int x = i >> 1, y = i & 1, k = i - I0;
      if (decltype(rdc)::value && k < 6) {
        if (k < 4) N.a[k] = rd(aa[k][st], off{});
        else N.b[k - 4] = rd(bb[k - 4][st], off{});
      }
      __builtin_amdgcn_sched_barrier(0);
      acc[x][y] = mfma32(__builtin_bit_cast(h8_t, F.a[x]), __builtin_bit_cast(h8_t, F.b[y]), acc[x][y]);
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  using I_0 = std::integral_constant<int, 0>;
  using I_1 = std::integral_constant<int, 1>;
  using I_8 = std::integral_constant<int, 8>;
  // Chunk c + 1 has landed for this wave once only the loads of c + 2 and c + 3 are outstanding
  // (8); the barrier then makes every wave's loads of c + 1 visible and ends every read of chunk c,
  // whose slot chunk c + 4 refills. Past the last chunk the steps read repeats and use none.
  Frags F0, F1;
  auto step = [&](int64_t c, auto zc) {
    constexpr int z = decltype(zc)::value;
    using zn = std::integral_constant<int, (z + 1) % kWRing>;
    mma_rng(F0, F1, zc, I_1{}, I_0{}, I_8{}, std::true_type{});
    landed(F1);
    __builtin_amdgcn_s_waitcnt(vmcnt_lgkm0_wait(8));
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
    mma_rng(F1, F0, zn{}, I_0{}, I_0{}, I_1{}, std::false_type{});
    issue(c + 4, zc);
    mma_rng(F1, F0, zn{}, I_0{}, I_1{}, I_8{}, std::true_type{});
    landed(F0);
  };
  issue(0, std::integral_constant<int, 0>{});
  issue(1, std::integral_constant<int, 1>{});
  issue(2, std::integral_constant<int, 2>{});
  __builtin_amdgcn_s_waitcnt(vmcnt_lgkm0_wait(8));
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_sched_barrier(0);
  issue(3, std::integral_constant<int, 3>{});
#pragma unroll
  for (int x = 0; x < 4; ++x) F0.a[x] = rd(aa[x][0], std::integral_constant<uint32_t, 0>{});
#pragma unroll
  for (int y = 0; y < 2; ++y) F0.b[y] = rd(bb[y][0], std::integral_constant<uint32_t, 0>{});
  landed(F0);
  for (int64_t c = 0; c < nch; c += kWRing) {
    step(c, std::integral_constant<int, 0>{});
    if (c + 1 < nch) step(c + 1, std::integral_constant<int, 1>{});
    if (c + 2 < nch) step(c + 2, std::integral_constant<int, 2>{});
    if (c + 3 < nch) step(c + 3, std::integral_constant<int, 3>{});
  }
  // no direct load may still be writing LDS when the workgroup ends
  __builtin_amdgcn_s_waitcnt(0);

  // D[i][j] of a 32x32 fragment: lane j + 32 * ((i / 4) % 2), element 4 * (i / 8) + i % 4; the
  // tiled index of (m, j) is ((m / 32) (r / 16) + j / 16) 512 + (m % 32) 16 + j % 16
  float* pdst = part + (int64_t)s * ((M + 31) / 32 * 32) * r;
#pragma unroll
  for (int y = 0; y < 2; ++y) {
    const int64_t gj = j0 + 64 * wj + 32 * y + (lane & 31);
    if (gj >= r) continue;
#pragma unroll
    for (int x = 0; x < 4; ++x)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int64_t gm = m0 + 128 * wm + 32 * x + 8 * (v >> 2) + 4 * ha + (v & 3);
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
  const int64_t nblk = (int64_t)p.ad_tiles_m * p.ad_tiles_j * p.ad_split;
  dim3 grid = p.ad_wide ? dim3((unsigned)p.ad_tiles_m, (unsigned)p.ad_tiles_j, (unsigned)p.ad_split)
                        : dim3((unsigned)(8 * ((nblk + 7) / 8)));
  uint16_t* out = reinterpret_cast<uint16_t*>(ws + p.off_t);
  float* part = reinterpret_cast<float*>(ws + p.off_tpart);
  SlimKernelTimer timer("adapter_gemm", s);
  if (p.ad_wide)
    SLIM_LAUNCH(timer, k_adapter_gemm_wide, grid, dim3(kWThreads), s, A, M, Kd, Q, r, p.ad_slice, p.ad_split, out, part);
  else
    SLIM_LAUNCH(timer, k_adapter_gemm, grid, dim3(256), s, A, M, Kd, Q, r, p.ad_slice, p.ad_split, out, part);
  return hipGetLastError() == hipSuccess ? SLIM_OK : SLIM_EDEVICE;
}
