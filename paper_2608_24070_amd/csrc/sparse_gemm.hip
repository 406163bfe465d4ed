// sparse_gemm.hip - the 2:4-sparse int4 contraction of the compressed linear layer and its
// input-gradient counterpart, with the low-rank adapter.
//
//   forward   Y[m, n]  = sum_k X[m, k] Wc[n, k]          + sum_j T[m, j] R[j, n],   T = X L
//   backward  dX[m, k] = sum_n dY[m, n] W^{R,C}[n, k]    + sum_j U[m, j] L[k, j],   U = dY R^T
//
// Both have the form
//   out[m, row] = sum_red act[m, red] A[row, red] + sum_j tm[m, j] P[row, j],  tm[m, j] = sum_red act[m, red] Q[j, red]
// with A the packed sparse operand (rows = N, red = K forward; rows = K, red = N backward) and the
// adapter factors in row-major [r x red] (Q) and [rows x r] (P) form: forward Q = L^T and P = R^T
// (from slim_pack_adapter), backward Q = R and P = L as given. Packed code words feed the sparse
// MFMA's compressed A operand directly; activations are the dense B operand as fp16; the
// accumulators hold out^T tiles (rows x m).
//
// Scales: forward, s16[n, k/128] varies along the output row and is applied while dequantising
// (fp16 product). Backward, s16[n, k/128] varies along the reduction n, so it multiplies the
// activations instead (B'[n, m] = dY[m, n] * s16[n, g], g fixed per 128-row group) and the codes
// enter the MFMA as exact integers.
//
// Two paths, chosen by the number of activation rows M:
//  * small M (<= 32, decode): k_decode splits the reduction across blocks so that every CU
//    streams a slice of the packed weight; the same launch computes the adapter's first product
//    in extra blocks (the two products share the activations, as in SLoPe's concatenated
//    adapter). Sparse units only store their partials; k_finish sums them in a fixed order and
//    adds the adapter's second product, so no sparse unit waits on another.
//  * large M: the adapter's first product runs as a dense GEMM (adapter_gemm.hip); k_tile then
//    computes 256 x 128 output tiles on 32x32x32 sparse MFMA with a double-buffered LDS
//    activation tile and adds the second adapter product in its epilogue.
// Every global load is issued unconditionally from a clamped, valid address and masked when
// used: a load under a branch makes the compiler wait for it at the join, which serialises
// what should be one round of memory traffic.
#include <type_traits>

#include "slim_device.h"
#include "slim_launch.h"
#include "slim_timing.h"

namespace {

struct LayerArgs {
  const uint32_t* codes;   // [rows, red/16] code words
  const uint32_t* meta;    // [rows, red/32] words = two index half-words
  const uint16_t* scales;  // forward [rows, red/128]; backward scalesT [rows/128, red]
  const uint16_t* act;     // [M, red] activations (bf16 or fp16 bits)
  int act_bf16;
  const uint16_t* act16;   // [M, red] fp16 activations for the large-M path (act, or a converted copy)
  int64_t M, rows, red;
  int64_t r;
  const uint16_t* ad_q;    // adapter first factor, row-major [r, red]
  const uint16_t* ad_p;    // adapter second factor, row-major [rows, r]
  uint16_t* tm;            // fp16 [M, r] adapter intermediate
  float* out;              // [M, rows]
  // small-M path
  int split;               // reduction splits of the sparse product
  int64_t row_tiles;       // 64-row tiles
  int ad_split;            // reduction splits of the adapter's first product
  int64_t ad_jblocks;      // 64-wide column blocks of the adapter rank
  float* part;             // sparse split partials
  float* tpart;            // adapter split partials
  uint32_t* tcounters;     // per adapter column block
  int finish;              // sparse partials go to k_finish (split > 1 or an adapter)
};

SLIM_DEV u32x4_t zero_u4() { return u32x4_t{0u, 0u, 0u, 0u}; }
SLIM_DEV int64_t clamp_hi(int64_t x, int64_t hi) { return x < hi ? x : hi; }

// bits of eight fp16 scales times eight activations (backward fold), rounded once to fp16.
SLIM_DEV h8_t act8_scaled(u32x4_t v, u32x4_t sv, bool bf16) {
  h8_t h;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    h[2 * i] = (_Float16)(act_to_f(v[i] & 0xFFFFu, bf16) * h_bits_to_f(sv[i] & 0xFFFFu));
    h[2 * i + 1] = (_Float16)(act_to_f(v[i] >> 16, bf16) * h_bits_to_f(sv[i] >> 16));
  }
  return h;
}

// Reduce split partials of one tile: every block stores its FM x 4 accumulator values per lane
// (device scope), the last one to arrive sums all S partials in split order.
template <int FM>
SLIM_DEV bool split_reduce(f4_t* acc, float* part_tile, int S, int s, uint32_t* counter, int* last_flag) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  constexpr int kPer = FM * 256;                    // floats per wave per split
  float* dst = part_tile + ((int64_t)s * 4 + wave) * kPer;
#pragma unroll
  for (int f = 0; f < FM; ++f)
#pragma unroll
    for (int v = 0; v < 4; ++v) st_dev(dst + (f * 4 + v) * 64 + lane, acc[f][v]);
  drain_stores();
  __syncthreads();
  if (tid == 0) *last_flag = counter_arrive(counter) == (uint32_t)(S - 1);
  __syncthreads();
  if (!*last_flag) return false;
#pragma unroll
  for (int f = 0; f < FM; ++f) acc[f] = f4_t{0.f, 0.f, 0.f, 0.f};
  const float* src = part_tile + (int64_t)wave * kPer;
  for (int s0 = 0; s0 < S; s0 += 8) {
    float pv[8][FM * 4];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int ss = s0 + j < S ? s0 + j : S - 1;
#pragma unroll
      for (int e = 0; e < FM * 4; ++e) pv[j][e] = ld_dev(src + (int64_t)ss * 4 * kPer + e * 64 + lane);
    }
#pragma unroll
    for (int j = 0; j < 8; ++j)
      if (s0 + j < S)
#pragma unroll
        for (int e = 0; e < FM * 4; ++e) acc[e >> 2][e & 3] += pv[j][e];
  }
  if (tid == 0) counter_reset(counter);
  return true;
}

// ============================================================ small-M: sparse split units
// Unit = 64 rows (16 per wave) x one slice of 4G quantisation groups. Lane group qa (lane / 16)
// of the 16x16x64 sparse MFMA owns G whole groups, so its code words (32 B per group), index
// words (16 B) and scales are contiguous: 4G loads per lane for the whole slice.
template <bool BWD, int FM, int G>
SLIM_DEV void decode_sparse_unit(const LayerArgs& a, int64_t u, _Float16* xs, int* last_flag) {
  constexpr int MC = 16 * FM;
  constexpr int SL = 512 * G;              // reduction positions per slice
  constexpr int LDX = SL + 8;
  constexpr int VPR = SL / 8;              // 16-byte activation vectors per row of the slice
  constexpr int XV = MC * VPR / 256;       // ... per thread
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int S = a.split;
  const int64_t rt = u / S;
  const int s = (int)(u - rt * S);
  const int64_t row0 = rt * 64;
  const int64_t nchunks = a.red / 128;
  const int64_t c0 = (int64_t)s * 4 * G;
  const int64_t red0 = c0 * 128;
  const bool bf16 = a.act_bf16 != 0;

  const int64_t lrow = clamp_hi(row0 + 16 * wave + (lane & 15), a.rows - 1);
  const int qa = lane >> 4;
  const int64_t cl = c0 + (int64_t)qa * G;      // first chunk (group) of this lane group
  u32x4_t cw[2 * G], mw[G];
  uint32_t sw[G];
#pragma unroll
  for (int gi = 0; gi < G; ++gi) {
    const int64_t ch = clamp_hi(cl + gi, nchunks - 1);
    const uint32_t* cp = a.codes + lrow * (a.red / 16) + ch * 8;
    cw[2 * gi] = *reinterpret_cast<const u32x4_t*>(cp);
    cw[2 * gi + 1] = *reinterpret_cast<const u32x4_t*>(cp + 4);
    mw[gi] = *reinterpret_cast<const u32x4_t*>(a.meta + lrow * (a.red / 32) + ch * 4);
    sw[gi] = BWD ? 0u : (uint32_t)a.scales[lrow * (a.red / 128) + ch];
  }
  const int64_t sgroup = row0 / 128;
  u32x4_t xv[XV], sv[XV];
#pragma unroll
  for (int i = 0; i < XV; ++i) {
    const int q = tid + 256 * i, m = q / VPR, vc = q % VPR;
    const int64_t pos = clamp_hi(red0 + 8 * vc, a.red - 8);
    xv[i] = *reinterpret_cast<const u32x4_t*>(a.act + clamp_hi(m, a.M - 1) * a.red + pos);
    if (BWD) sv[i] = *reinterpret_cast<const u32x4_t*>(a.scales + sgroup * a.red + pos);
  }
#pragma unroll
  for (int i = 0; i < XV; ++i) {
    const int q = tid + 256 * i, m = q / VPR, vc = q % VPR;
    const bool ok = m < a.M && red0 + 8 * vc < a.red;
    const h8_t h = BWD ? act8_scaled(xv[i], sv[i], bf16) : load8_as_h(xv[i], bf16);
    *reinterpret_cast<h8_t*>(&xs[m * LDX + 8 * vc]) = ok ? h : zero_h8();
  }
  __syncthreads();

  f4_t acc[FM];
#pragma unroll
  for (int f = 0; f < FM; ++f) acc[f] = f4_t{0.f, 0.f, 0.f, 0.f};
  const int qb = lane >> 4;
  const int pbase = 128 * G * (qb >> 1) + 8 * (qb & 1);
#pragma unroll
  for (int gi = 0; gi < G; ++gi) {
    const bool gok = cl + gi < nchunks;
    const h2_t s2 = splat_h2(sw[gi]);
#pragma unroll
    for (int t4 = 0; t4 < 8; ++t4) {
      const uint32_t word = cw[2 * gi + (t4 >> 2)][t4 & 3];
      h8_t av = BWD ? dequant_word_int(word) : dequant_word(word, s2);
      av = gok ? av : zero_h8();
      const int idx = (int)mw[gi][t4 >> 1];
      const int p0 = pbase + 16 * (8 * gi + t4);
#pragma unroll
      for (int f = 0; f < FM; ++f) {
        const _Float16* xr = xs + (16 * f + (lane & 15)) * LDX + p0;
        acc[f] = smfmac16(av, cat16(*reinterpret_cast<const h8_t*>(xr), *reinterpret_cast<const h8_t*>(xr + 256 * G)),
                          acc[f], idx, t4 & 1);
      }
    }
  }

  (void)last_flag;
  if (a.finish) {
    // k_finish sums the split partials (and adds the adapter); the kernel boundary orders them
    float* dst = a.part + ((rt * S + s) * 4 + wave) * (int64_t)(FM * 256);
#pragma unroll
    for (int f = 0; f < FM; ++f) *reinterpret_cast<f4_t*>(dst + f * 256 + 4 * lane) = acc[f];
    return;
  }

  // out^T fragment: lane (col + 16 * (row / 4)), element row % 4 -> 4 consecutive rows
  const int64_t rr = row0 + 16 * wave + 4 * (lane >> 4);
  if (rr < a.rows) {
#pragma unroll
    for (int f = 0; f < FM; ++f) {
      const int64_t m = 16 * f + (lane & 15);
      if (m < a.M) *reinterpret_cast<f4_t*>(a.out + m * a.rows + rr) = acc[f];
    }
  }
}

// ============================================================ small-M: adapter first-product units
// tm[m, j] = sum_red act[m, red] Q[j, red]. Unit = 64 adapter columns (16 per wave) x one slice
// of 256 reduction positions; both operands are read straight from global memory.
constexpr int kAdSlice = SLIM_DECODE_AD_SLICE;

template <int FM>
SLIM_DEV void decode_adapter_unit(const LayerArgs& a, int64_t v, int* last_flag) {
  constexpr int kSteps = kAdSlice / 32;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int SA = a.ad_split;
  const int64_t jb = v / SA;
  const int sa = (int)(v - jb * SA);
  const int64_t r0 = (int64_t)sa * kAdSlice;
  const bool bf16 = a.act_bf16 != 0;
  const int g = lane >> 4;
  const int64_t jcol = jb * 64 + 16 * wave + (lane & 15);
  const int64_t jl = clamp_hi(jcol, a.r - 1);

  u32x4_t aq[kSteps][FM], bq[kSteps];
#pragma unroll
  for (int t = 0; t < kSteps; ++t) {
    const int64_t rk = clamp_hi(r0 + 32 * t + 8 * g, a.red - 8);
#pragma unroll
    for (int f = 0; f < FM; ++f)
      aq[t][f] = *reinterpret_cast<const u32x4_t*>(a.act + clamp_hi(16 * f + (lane & 15), a.M - 1) * a.red + rk);
    bq[t] = *reinterpret_cast<const u32x4_t*>(a.ad_q + jl * a.red + rk);
  }
  f4_t acc[FM];
#pragma unroll
  for (int f = 0; f < FM; ++f) acc[f] = f4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int t = 0; t < kSteps; ++t) {
    const bool kok = r0 + 32 * t + 8 * g < a.red;
    const h8_t bv = (kok && jcol < a.r) ? __builtin_bit_cast(h8_t, bq[t]) : zero_h8();
#pragma unroll
    for (int f = 0; f < FM; ++f) {
      const h8_t av = (16 * f + (lane & 15) < a.M) ? load8_as_h(aq[t][f], bf16) : zero_h8();
      acc[f] = mfma16(av, bv, acc[f]);
    }
  }
  if (SA > 1 && !split_reduce<FM>(acc, a.tpart + jb * (int64_t)SA * 4 * FM * 256, SA, sa, &a.tcounters[jb], last_flag))
    return;
  // D[m][j] fragment: lane (j + 16 * (m / 4)), element m % 4
#pragma unroll
  for (int f = 0; f < FM; ++f)
#pragma unroll
    for (int vv = 0; vv < 4; ++vv) {
      const int64_t m = 16 * f + 4 * g + vv;
      if (m < a.M && jcol < a.r) a.tm[m * a.r + jcol] = __builtin_bit_cast(uint16_t, (_Float16)acc[f][vv]);
    }
}

// Blocks [0, jblocks * ad_split) are adapter units (dispatched first: their reduction is the
// longer path); the rest are sparse units.
template <bool BWD, int FM, int G>
__global__ void __launch_bounds__(256) k_decode(LayerArgs a) {
  __shared__ __attribute__((aligned(16))) _Float16 xs[16 * FM * (512 * G + 8)];
  __shared__ int last_flag;
  const int64_t nA = a.r > 0 ? a.ad_jblocks * a.ad_split : 0;
  const int64_t b = blockIdx.x;
  if (b < nA) decode_adapter_unit<FM>(a, b, &last_flag);
  else decode_sparse_unit<BWD, FM, G>(a, b - nA, xs, &last_flag);
}

// ============================================================ small-M: finish
// out[m, row] = sum_s part_s[m, row] + sum_j tm[m, j] P[row, j]. One wave per 16 output rows; the
// split partials are summed in split order (deterministic) and the adapter's second product is
// accumulated on top with 16x16x32 fp16 MFMA. The partials share the MFMA output layout, so each
// lane reads its own four values per split and fragment.
template <int FM>
__global__ void __launch_bounds__(64) k_finish(LayerArgs a) {
  constexpr int kSteps = FM == 1 ? 16 : 8;
  const int lane = threadIdx.x, g = lane >> 4;
  const int64_t row0 = (int64_t)blockIdx.x * 16;
  const int64_t lrow = clamp_hi(row0 + (lane & 15), a.rows - 1);
  const int64_t rr = row0 + 4 * g;
  const int64_t rt = row0 / 64;
  const int w16 = (int)((row0 % 64) / 16);
  const int S = a.split;
  f4_t acc[FM];
#pragma unroll
  for (int f = 0; f < FM; ++f) acc[f] = f4_t{0.f, 0.f, 0.f, 0.f};
  const float* src = a.part + (rt * S * 4 + w16) * (int64_t)(FM * 256);
  for (int s0 = 0; s0 < S; s0 += 8) {
    f4_t pv[8][FM];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int ss = s0 + j < S ? s0 + j : S - 1;
#pragma unroll
      for (int f = 0; f < FM; ++f)
        pv[j][f] = *reinterpret_cast<const f4_t*>(src + (int64_t)ss * 4 * FM * 256 + f * 256 + 4 * lane);
    }
#pragma unroll
    for (int j = 0; j < 8; ++j)
      if (s0 + j < S)
#pragma unroll
        for (int f = 0; f < FM; ++f) acc[f] = acc[f] + pv[j][f];
  }
  for (int64_t jbase = 0; jbase < a.r; jbase += 32 * kSteps) {
    u32x4_t aq[kSteps], bq[kSteps][FM];
#pragma unroll
    for (int t = 0; t < kSteps; ++t) {
      const int64_t jj = clamp_hi(jbase + 32 * t + 8 * g, a.r - 8);
      aq[t] = *reinterpret_cast<const u32x4_t*>(a.ad_p + lrow * a.r + jj);
#pragma unroll
      for (int f = 0; f < FM; ++f)
        bq[t][f] = *reinterpret_cast<const u32x4_t*>(a.tm + clamp_hi(16 * f + (lane & 15), a.M - 1) * a.r + jj);
    }
#pragma unroll
    for (int t = 0; t < kSteps; ++t) {
      const bool jok = jbase + 32 * t + 8 * g < a.r;
      const h8_t av = jok ? __builtin_bit_cast(h8_t, aq[t]) : zero_h8();
#pragma unroll
      for (int f = 0; f < FM; ++f) {
        const h8_t bv = (16 * f + (lane & 15) < a.M) ? __builtin_bit_cast(h8_t, bq[t][f]) : zero_h8();
        acc[f] = mfma16(av, bv, acc[f]);
      }
    }
  }
  if (rr < a.rows) {
#pragma unroll
    for (int f = 0; f < FM; ++f) {
      const int64_t m = 16 * f + (lane & 15);
      if (m < a.M) *reinterpret_cast<f4_t*>(a.out + m * a.rows + rr) = acc[f];
    }
  }
}

// ============================================================ large-M tile kernel
// Block = 4 waves; wave (wr, wc) owns rows [row0 + 128 wr, +128) as 4 fragments of 32 and columns
// [m0 + 64 wc, +64) as 2 fragments of 32 (a 128 x 64 accumulator on 32x32x32 sparse MFMA).
// Per 128-wide reduction chunk the fp16 activation tile [128 x 128] goes straight from memory to
// LDS (16-byte direct loads) into a ring of three buffers, two chunks ahead; the packed words
// go to registers two chunks ahead. LDS rows are 256 B with the 16-byte column
// index XOR-swizzled by the row, so the B-fragment reads (32 rows at one column) hit distinct
// banks. The backward also brings each wave's scale row (its 128-row group) into LDS.
constexpr int kTR = 256, kTC = 128, kTThreads = 256, kStages = 3;
// VMEM instructions per thread per chunk: 8 activation loads and 12 packed-word loads (codes,
// index words, scales); the backward has no scale words but one scale-row load. Chunk c's loads
// are issued in the body of chunk c - (kStages - 1); at least kStages - 2 whole bodies of loads
// follow them (more in the prologue, which issues them in the same order), so they are complete
// once at most that many are outstanding: the count the loop waits for before its barrier.
constexpr int kTileVmemFwd = 8 + 12, kTileVmemBwd = 8 + 8 + 1;
constexpr int kTileWaitFwd = (kStages - 2) * kTileVmemFwd, kTileWaitBwd = (kStages - 2) * kTileVmemBwd;

// s_waitcnt immediate (gfx9 layout) waiting for at most n outstanding vector-memory operations:
// vmcnt bits [3:0] and [15:14]; expcnt [6:4] and lgkmcnt [11:8] left at their maxima (no wait)
constexpr unsigned vmcnt_wait(int n) { return (unsigned)(n & 15) | ((unsigned)(n >> 4) << 14) | 0x0F70u; }
static_assert(vmcnt_wait(40) == 0x8F78u && vmcnt_wait(5) == 0x0F75u && kTileWaitFwd < 64, "s_waitcnt encoding");

struct TileA {
  u32x4_t cw[4];
  u32x2_t mw[4];
  uint32_t sw[4];
};

template <bool BWD>
SLIM_DEV void tile_load_a(const uint32_t* const* cp, const uint32_t* const* mp, const uint16_t* const* sp, int64_t c,
                          TileA& t) {
#pragma unroll
  for (int fn = 0; fn < 4; ++fn) {
    t.cw[fn] = *reinterpret_cast<const u32x4_t*>(cp[fn] + 8 * c);
    t.mw[fn] = *reinterpret_cast<const u32x2_t*>(mp[fn] + 4 * c);
    t.sw[fn] = BWD ? 0u : (uint32_t)sp[fn][c];
  }
}

template <bool BWD>
SLIM_DEV void tile_body(const LayerArgs& a) {
  // one array per stage (the stage of chunk c is c % 3, a constant in the loop unrolled by three),
  // so that reads of one stage are not ordered behind loads still landing in another
  __shared__ __attribute__((aligned(16))) _Float16 xs0[kTC][128], xs1[kTC][128], xs2[kTC][128];
  __shared__ __attribute__((aligned(16))) _Float16 ss0[BWD ? 4 : 1][512], ss1[BWD ? 4 : 1][512], ss2[BWD ? 4 : 1][512];
  auto xs_at = [&](int stg) -> _Float16(*)[128] { return stg == 0 ? xs0 : (stg == 1 ? xs1 : xs2); };
  auto ss_at = [&](int stg) -> _Float16(*)[512] { return stg == 0 ? ss0 : (stg == 1 ? ss1 : ss2); };
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wr = wave & 1, wc = wave >> 1;
  const int ha = lane >> 5;
  const int64_t row0 = (int64_t)blockIdx.x * kTR, m0 = (int64_t)blockIdx.y * kTC;
  const int64_t wrow0 = row0 + 128 * wr;
  const int64_t nch = a.red / 128;

  const uint32_t* cp[4];
  const uint32_t* mp[4];
  const uint16_t* sp[4];
#pragma unroll
  for (int fn = 0; fn < 4; ++fn) {
    const int64_t arow = clamp_hi(wrow0 + 32 * fn + (lane & 31), a.rows - 1);
    cp[fn] = a.codes + arow * (a.red / 16) + 4 * ha;
    mp[fn] = a.meta + arow * (a.red / 32) + 2 * ha;
    sp[fn] = a.scales + arow * (a.red / 128);
  }

  // activation chunk c -> stage c % kStages: wave w writes rows 32 w .. 32 w + 31, four per load
  // (lane L: row + L / 16, LDS column slot L % 16 holding column (L % 16) ^ (row % 16))
  const int lrow = lane >> 4, lslot = lane & 15;
  auto dma_x = [&](int64_t c, int stg) {
    const int64_t cc = clamp_hi(c, nch - 1);
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int row = 32 * wave + 4 * i + lrow;
      const uint16_t* src =
          a.act16 + clamp_hi(m0 + row, a.M - 1) * a.red + cc * 128 + 8 * (lslot ^ (row & 15));
      __builtin_amdgcn_global_load_lds(src, &xs_at(stg)[32 * wave + 4 * i][0], 16, 0, 0);
    }
    if (BWD) {
      // the wave's scale row s16[n, g] for this chunk (g = its 128-row group), four copies
      const int64_t g = clamp_hi(wrow0, a.rows - 1) / 128;
      const uint16_t* src = a.scales + g * a.red + cc * 128 + 8 * lslot;
      __builtin_amdgcn_global_load_lds(src, &ss_at(stg)[wave][0], 16, 0, 0);
    }
  };

  f16_t acc[4][2];
#pragma unroll
  for (int fn = 0; fn < 4; ++fn)
#pragma unroll
    for (int fm = 0; fm < 2; ++fm)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[fn][fm][v] = 0.f;

  // packed words: a ring of three register sets, chunk c in set c % 3, two chunks ahead; the
  // loop is unrolled by three so that the sets rotate without copies
  // (issued in the order the loop issues them, so the loop entry matches its back edge)
  TileA w[3];
  dma_x(0, 0);
  tile_load_a<BWD>(cp, mp, sp, 0, w[0]);
  dma_x(1, 1);
  tile_load_a<BWD>(cp, mp, sp, clamp_hi(1, nch - 1), w[1]);

  // one chunk: wait for its activations, refill the ring two chunks ahead, multiply
  auto chunk = [&](int64_t c, auto zc) {
    constexpr int z = decltype(zc)::value;
    const int stg = z;                      // c % 3 (c0 is a multiple of 3)
    // chunk c's activations (and packed words) have landed once at most kStages - 2 chunks of later
    // loads are outstanding.
    // The barrier is issued as a bare instruction: the builtin would also make this wave wait
    // for every direct-to-LDS load in flight, including the ones for the next two chunks.
    __builtin_amdgcn_s_waitcnt(vmcnt_wait(BWD ? kTileWaitBwd : kTileWaitFwd));
    asm volatile("s_barrier" ::: "memory");
    dma_x(c + kStages - 1, (z + 2) % 3);    // into the stage read in iteration c - 1
    tile_load_a<BWD>(cp, mp, sp, clamp_hi(c + 2, nch - 1), w[(z + 2) % 3]);
    // pin this chunk's packed words here: work on them cannot be scheduled into earlier chunks
    // (which would make those wait for loads that are meant to stay in flight)
    TileA& cur = w[z];
#pragma unroll
    for (int fn = 0; fn < 4; ++fn) {
      asm volatile("" : "+v"(cur.cw[fn]), "+v"(cur.mw[fn]), "+v"(cur.sw[fn]));
    }
#pragma unroll
    for (int st = 0; st < 4; ++st) {
      h8_t av[4];
      h16_t bv[2];
#pragma unroll
      for (int fn = 0; fn < 4; ++fn)
        av[fn] = BWD ? dequant_word_int(cur.cw[fn][st]) : dequant_word(cur.cw[fn][st], splat_h2(cur.sw[fn]));
      // B operand: columns (16-byte units) 2 st + ha and 2 st + ha + 8 of the chunk
      const int c16 = 2 * st + ha;
#pragma unroll
      for (int fm = 0; fm < 2; ++fm) {
        const int row = 64 * wc + 32 * fm + (lane & 31);
        const _Float16* rp = &xs_at(stg)[row][0];
        h8_t lo = *reinterpret_cast<const h8_t*>(rp + 8 * (c16 ^ (row & 15)));
        h8_t hi = *reinterpret_cast<const h8_t*>(rp + 8 * ((c16 + 8) ^ (row & 15)));
        if (BWD) {
          lo = mul_h8(lo, *reinterpret_cast<const h8_t*>(&ss_at(stg)[wave][8 * c16]));
          hi = mul_h8(hi, *reinterpret_cast<const h8_t*>(&ss_at(stg)[wave][8 * c16 + 64]));
        }
        bv[fm] = cat16(lo, hi);
      }
#pragma unroll
      for (int fn = 0; fn < 4; ++fn)
#pragma unroll
        for (int fm = 0; fm < 2; ++fm)
          acc[fn][fm] = smfmac32(av[fn], bv[fm], acc[fn][fm], (int)cur.mw[fn][st >> 1], st & 1);
    }
  };
  // full groups of three without guards (a load under a branch costs a full wait at the join),
  // then at most two chunks
  int64_t c0 = 0;
  for (; c0 + 3 <= nch; c0 += 3) {
    chunk(c0, std::integral_constant<int, 0>{});
    chunk(c0 + 1, std::integral_constant<int, 1>{});
    chunk(c0 + 2, std::integral_constant<int, 2>{});
  }
  if (c0 < nch) chunk(c0, std::integral_constant<int, 0>{});
  if (c0 + 1 < nch) chunk(c0 + 1, std::integral_constant<int, 1>{});
  // the ring's last loads (repeats of the final chunk) must land before the block's LDS is released
  __builtin_amdgcn_s_waitcnt(0);

  // adapter second product: out^T[row, m] += sum_j P[row, j] tm[m, j], on 32x32x16 fp16 MFMA;
  // both operands are row-major along j, 64 ranks per round of loads
  if (a.r > 0) {
    for (int64_t jb = 0; jb < a.r; jb += 64) {
      u32x4_t aq[4][4], bq[4][2];     // [kk][fn], [kk][fm]
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) {
        const int64_t jj = clamp_hi(jb + 16 * kk + 8 * ha, a.r - 8);
#pragma unroll
        for (int fn = 0; fn < 4; ++fn)
          aq[kk][fn] =
              *reinterpret_cast<const u32x4_t*>(a.ad_p + clamp_hi(wrow0 + 32 * fn + (lane & 31), a.rows - 1) * a.r + jj);
#pragma unroll
        for (int fm = 0; fm < 2; ++fm)
          bq[kk][fm] =
              *reinterpret_cast<const u32x4_t*>(a.tm + clamp_hi(m0 + 64 * wc + 32 * fm + (lane & 31), a.M - 1) * a.r + jj);
      }
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) {
        const bool jok = jb + 16 * kk + 8 * ha < a.r;
#pragma unroll
        for (int fn = 0; fn < 4; ++fn) {
          const h8_t av = jok ? __builtin_bit_cast(h8_t, aq[kk][fn]) : zero_h8();
#pragma unroll
          for (int fm = 0; fm < 2; ++fm) {
            const h8_t bv = (m0 + 64 * wc + 32 * fm + (lane & 31) < a.M) ? __builtin_bit_cast(h8_t, bq[kk][fm]) : zero_h8();
            acc[fn][fm] = mfma32(av, bv, acc[fn][fm]);
          }
        }
      }
    }
  }

  // D[i][j] of a 32x32 fragment: lane j + 32 * ((i / 4) % 2), element 4 * (i / 8) + i % 4
#pragma unroll
  for (int fm = 0; fm < 2; ++fm) {
    const int64_t m = m0 + 64 * wc + 32 * fm + (lane & 31);
    if (m >= a.M) continue;
#pragma unroll
    for (int fn = 0; fn < 4; ++fn)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int64_t rr = wrow0 + 32 * fn + 8 * q + 4 * ha;
        if (rr < a.rows) {
          const f4_t o = {acc[fn][fm][4 * q], acc[fn][fm][4 * q + 1], acc[fn][fm][4 * q + 2], acc[fn][fm][4 * q + 3]};
          *reinterpret_cast<f4_t*>(a.out + m * a.rows + rr) = o;
        }
      }
  }
}

template <bool BWD>
__global__ void __launch_bounds__(kTThreads) k_tile(LayerArgs a) {
  tile_body<BWD>(a);
}

// bf16 -> fp16 (round to nearest even), 8 values per thread
__global__ void __launch_bounds__(256) k_bf16_to_f16(const u32x4_t* __restrict__ src, u32x4_t* __restrict__ dst,
                                                     int64_t n8) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i < n8) dst[i] = __builtin_bit_cast(u32x4_t, load8_as_h(src[i], true));
}

// ------------------------------------------------------------------------------ launch
template <bool BWD, int FM, int G>
void launch_decode(const LayerArgs& a, const SlimPlan& p, hipStream_t s) {
  SlimKernelTimer timer(BWD ? "decode_bwd" : "decode_fwd", s);
  dim3 grid((unsigned)(p.sp_row_tiles * p.sp_split + (a.r > 0 ? p.ad_jblocks * p.ad_split : 0)));
  SLIM_LAUNCH(timer, (k_decode<BWD, FM, G>), grid, dim3(256), s, a);
}

template <int FM>
void launch_finish(const LayerArgs& a, bool bwd, hipStream_t s) {
  SlimKernelTimer timer(bwd ? "finish_bwd" : "finish_fwd", s);
  SLIM_LAUNCH(timer, (k_finish<FM>), dim3((unsigned)((a.rows + 15) / 16)), dim3(64), s, a);
}

template <bool BWD>
int launch_layer(const LayerArgs& a, const SlimPlan& p, const uint16_t* act, int act_bf16, char* ws, hipStream_t s) {
  if (p.decode) {
    if (p.dec_fm == 1) {
      if (p.dec_g == 1) launch_decode<BWD, 1, 1>(a, p, s);
      else launch_decode<BWD, 1, 2>(a, p, s);
    } else {
      launch_decode<BWD, 2, 1>(a, p, s);
    }
    if (hipGetLastError() != hipSuccess) return SLIM_EDEVICE;
    if (a.finish) {
      if (p.dec_fm == 1) launch_finish<1>(a, BWD, s);
      else launch_finish<2>(a, BWD, s);
      if (hipGetLastError() != hipSuccess) return SLIM_EDEVICE;
    }
    return SLIM_OK;
  }
  if (act_bf16) {
    // the tile kernel streams fp16 activations straight into LDS: convert them once
    SlimKernelTimer timer("to_f16", s);
    const int64_t n8 = a.M * a.red / 8;
    SLIM_LAUNCH(timer, k_bf16_to_f16, dim3((unsigned)((n8 + 255) / 256)), dim3(256), s,
                reinterpret_cast<const u32x4_t*>(act), reinterpret_cast<u32x4_t*>(const_cast<uint16_t*>(a.act16)), n8);
    if (hipGetLastError() != hipSuccess) return SLIM_EDEVICE;
  }
  if (a.r > 0) {
    int st = slim_launch_adapter_gemm(act, act_bf16, a.M, a.red, a.ad_q, a.r, p, ws, s);
    if (st != SLIM_OK) return st;
  }
  SlimKernelTimer timer(BWD ? "tile_bwd" : "tile_fwd", s);
  dim3 grid((unsigned)p.sp_row_tiles, (unsigned)p.sp_col_tiles);
  SLIM_LAUNCH(timer, (k_tile<BWD>), grid, dim3(kTThreads), s, a);
  return hipGetLastError() == hipSuccess ? SLIM_OK : SLIM_EDEVICE;
}

LayerArgs make_args(const SlimPlan& p, char* ws, const void* act, int dtype, int64_t M, int64_t rows, int64_t red,
                    const uint8_t* codes, const uint8_t* meta, const uint16_t* scales, const uint16_t* ad_q,
                    const uint16_t* ad_p, int64_t r, float* out) {
  LayerArgs a;
  a.codes = reinterpret_cast<const uint32_t*>(codes);
  a.meta = reinterpret_cast<const uint32_t*>(meta);
  a.scales = scales;
  a.act = reinterpret_cast<const uint16_t*>(act);
  a.act_bf16 = dtype == SLIM_BF16;
  a.M = M;
  a.rows = rows;
  a.red = red;
  a.r = r;
  a.ad_q = ad_q;
  a.ad_p = ad_p;
  a.tm = reinterpret_cast<uint16_t*>(ws + p.off_t);
  a.act16 = (!p.decode && dtype == SLIM_BF16) ? reinterpret_cast<const uint16_t*>(ws + p.off_x16) : a.act;
  a.out = out;
  a.split = p.sp_split;
  a.row_tiles = p.sp_row_tiles;
  a.ad_split = p.ad_split;
  a.ad_jblocks = p.ad_jblocks;
  a.part = reinterpret_cast<float*>(ws + p.off_ypart);
  a.tpart = reinterpret_cast<float*>(ws + p.off_tpart);
  a.tcounters = reinterpret_cast<uint32_t*>(ws + p.off_counters);
  a.finish = p.decode && (p.sp_split > 1 || r > 0);
  return a;
}

}  // namespace

extern "C" int slim_workspace_init(void* ws, size_t ws_bytes, void* stream) {
  if (!ws) return SLIM_EINVAL;
  if (ws_bytes < SLIM_COUNTER_SLOTS * 4) return SLIM_EWORKSPACE;
  return hipMemsetAsync(ws, 0, ws_bytes, (hipStream_t)stream) == hipSuccess ? SLIM_OK : SLIM_EDEVICE;
}

extern "C" int slim_linear(const void* X, int xdtype, int64_t M, int64_t N, int64_t K, const uint8_t* codes,
                           const uint8_t* meta, const uint16_t* scales, const uint16_t* Lt, const uint16_t* Rt,
                           int64_t r, float* Y, void* ws, size_t ws_bytes, void* stream) {
  SlimPlan p;
  int st = slim_check_linear(false, X, xdtype, M, N, K, codes, meta, scales, Lt, Rt, r, Y, ws, ws_bytes, &p);
  if (st != SLIM_OK) return st;
  char* w = reinterpret_cast<char*>(ws);
  const LayerArgs a = make_args(p, w, X, xdtype, M, N, K, codes, meta, scales, Lt, Rt, r, Y);
  return launch_layer<false>(a, p, reinterpret_cast<const uint16_t*>(X), xdtype == SLIM_BF16, w, (hipStream_t)stream);
}

extern "C" int slim_linear_bwd_dx(const void* dY, int dydtype, int64_t M, int64_t N, int64_t K,
                                  const uint8_t* codesT, const uint8_t* metaT, const uint16_t* scalesT,
                                  const uint16_t* L, const uint16_t* R, int64_t r, float* dX, void* ws,
                                  size_t ws_bytes, void* stream) {
  SlimPlan p;
  int st = slim_check_linear(true, dY, dydtype, M, N, K, codesT, metaT, scalesT, L, R, r, dX, ws, ws_bytes, &p);
  if (st != SLIM_OK) return st;
  char* w = reinterpret_cast<char*>(ws);
  const LayerArgs a = make_args(p, w, dY, dydtype, M, K, N, codesT, metaT, scalesT, R, L, r, dX);
  return launch_layer<true>(a, p, reinterpret_cast<const uint16_t*>(dY), dydtype == SLIM_BF16, w, (hipStream_t)stream);
}
