// sparse_gemm.hip - the 2:4-sparse int4 contraction of the compressed linear layer and its
// input-gradient counterpart, with the low-rank adapter.
//
//   forward   Y[m, n]  = sum_k X[m, k] Wc[n, k]          + sum_j T[m, j] R[j, n],   T = X L
//   backward  dX[m, k] = sum_n dY[m, n] W^{R,C}[n, k]    + sum_j U[m, j] L[k, j],   U = dY R^T
//
// Both are "out[m, row] = sum_red act[m, red] A[row, red] + sum_j tm[m, j] ap(row, j)" with A the
// packed sparse operand (rows = N, red = K forward; rows = K, red = N backward). Packed code
// words feed the sparse MFMA's compressed A operand directly; activations are the dense B
// operand as fp16. Accumulators hold out^T tiles (rows x m).
//
// Scales: forward, s16[n, k/128] varies along the output row and is applied while dequantising
// (fp16 product). Backward, s16[n, k/128] varies along the reduction n, so it multiplies the
// activations instead (B'[n, m] = dY[m, n] * s16[n, g], g fixed per 128-row group) and the codes
// enter the MFMA as exact integers.
//
// Two paths, chosen by the number of activation rows M:
//  * small M (<= 64, decode): k_decode splits the reduction across blocks so that every CU
//    streams a slice of the packed weight; the same launch also computes the adapter's first
//    product (X L, or dY R^T) as extra blocks (the two products share the activations, as in
//    SLoPe's concatenated adapter). Split partials are reduced by the last block of each tile
//    in a fixed order. k_adapter_out then adds the adapter's second product.
//  * large M (prefill/training): the adapter's first product runs as a dense GEMM
//    (adapter_gemm.hip), then k_tile computes 256 x 128 output tiles on 32x32x32 sparse MFMA
//    with a double-buffered LDS activation tile and adds the second adapter product in its
//    epilogue.
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
  int64_t M, rows, red;
  int64_t r;
  const uint16_t* ad_in;   // first adapter factor: forward L [red, r]; backward R [r, red]
  const uint16_t* ad_out;  // second adapter factor: forward R [r, rows]; backward L [rows, r]
  uint16_t* tm;            // fp16 [M, r] adapter intermediate (T forward, U backward)
  float* out;              // [M, rows]
  // small-M path
  int split;               // reduction splits of the sparse product
  int64_t cps;             // 128-wide chunks per split
  int64_t row_tiles;       // 64-row tiles
  int ad_split;            // reduction splits of the adapter's first product
  int64_t ad_slice;        // reduction positions per adapter split
  int64_t ad_jblocks;      // 64-wide column blocks of the adapter rank
  float* part;             // sparse split partials
  float* tpart;            // adapter split partials
  uint32_t* counters;      // per 64-row tile
  uint32_t* tcounters;     // per adapter column block
};

constexpr int kMaxChunks = 16;   // the plan keeps cps <= 13 and FM * cps <= 16

SLIM_DEV u32x4_t zero_u4() { return u32x4_t{0u, 0u, 0u, 0u}; }

// fp16 eight-vector from 16-bit activation bits (bf16 -> fp16 through fp32).
SLIM_DEV h8_t act8(u32x4_t v, bool bf16) { return load8_as_h(v, bf16); }

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

// ============================================================ small-M: sparse split units
template <bool BWD, int FM>
SLIM_DEV void decode_sparse_unit(const LayerArgs& a, int64_t u, _Float16* xs, int* last_flag) {
  constexpr int MC = 16 * FM;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int S = a.split;
  const int64_t rt = u / S;
  const int s = (int)(u - rt * S);
  const int64_t row0 = rt * 64;
  const int64_t c_beg = (int64_t)s * a.cps;
  const int nch = (int)min(a.cps, a.red / 128 - c_beg);
  const int ldx = (int)a.cps * 128 + 8;
  const int64_t red0 = c_beg * 128;
  const bool bf16 = a.act_bf16 != 0;

  // 1. packed words of every chunk of the slice, and the activation slice: one round of loads
  const int64_t arow = row0 + 16 * wave + (lane & 15);
  const int64_t lrow = arow < a.rows ? arow : a.rows - 1;
  const int qa = lane >> 4;
  const uint32_t* cp = a.codes + lrow * (a.red / 16) + c_beg * 8 + 2 * qa;
  const uint32_t* mp = a.meta + lrow * (a.red / 32) + c_beg * 4 + qa;
  const uint16_t* sp = a.scales + lrow * (a.red / 128) + c_beg;
  u32x2_t cw[kMaxChunks];
  uint32_t mw[kMaxChunks], sw[kMaxChunks];
#pragma unroll
  for (int i = 0; i < kMaxChunks; ++i) {
    if (i < nch) {
      cw[i] = *reinterpret_cast<const u32x2_t*>(cp + 8 * i);
      mw[i] = mp[4 * i];
      sw[i] = BWD ? 0u : (uint32_t)sp[i];
    }
  }
  const int vpr = nch * 16;          // 16-byte activation vectors per row of the slice
  const int nvec = MC * vpr;         // at most 256 * kMaxChunks
  const int64_t sgroup = row0 / 128;
  u32x4_t xv[kMaxChunks], sv[kMaxChunks];
#pragma unroll
  for (int i = 0; i < kMaxChunks; ++i) {
    const int q = tid + 256 * i;
    if (q < nvec) {
      const int m = q / vpr, vc = q - m * vpr;
      xv[i] = m < a.M ? *reinterpret_cast<const u32x4_t*>(a.act + m * a.red + red0 + 8 * vc) : zero_u4();
      if (BWD) sv[i] = *reinterpret_cast<const u32x4_t*>(a.scales + sgroup * a.red + red0 + 8 * vc);
    }
  }
#pragma unroll
  for (int i = 0; i < kMaxChunks; ++i) {
    const int q = tid + 256 * i;
    if (q < nvec) {
      const int m = q / vpr, vc = q - m * vpr;
      *reinterpret_cast<h8_t*>(&xs[m * ldx + 8 * vc]) = BWD ? act8_scaled(xv[i], sv[i], bf16) : act8(xv[i], bf16);
    }
  }
  __syncthreads();

  // 2. contraction: 16 rows per wave, FM 16-column fragments, two 16x16x64 steps per chunk
  f4_t acc[FM];
#pragma unroll
  for (int f = 0; f < FM; ++f) acc[f] = f4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int i = 0; i < kMaxChunks; ++i) {
    if (i < nch) {
      const h2_t s2 = splat_h2(sw[i]);
#pragma unroll
      for (int st = 0; st < 2; ++st) {
        const h8_t av = BWD ? dequant_word_int(cw[i][st]) : dequant_word(cw[i][st], s2);
        const int off = i * 128 + b_chunk_offset<16>(lane, st);
#pragma unroll
        for (int f = 0; f < FM; ++f) {
          const _Float16* xr = xs + (16 * f + (lane & 15)) * ldx + off;
          acc[f] = smfmac16(av, cat16(*reinterpret_cast<const h8_t*>(xr), *reinterpret_cast<const h8_t*>(xr + 64)),
                            acc[f], (int)mw[i], st);
        }
      }
    }
  }

  // 3. split reduction: the last block of the row tile sums the partials in split order
  if (S > 1) {
    float* dst = a.part + ((rt * S + s) * 4 + wave) * (FM * 256);
#pragma unroll
    for (int f = 0; f < FM; ++f)
#pragma unroll
      for (int v = 0; v < 4; ++v) st_dev(dst + (f * 4 + v) * 64 + lane, acc[f][v]);
    drain_stores();
    __syncthreads();
    if (tid == 0) *last_flag = counter_arrive(&a.counters[rt]) == (uint32_t)(S - 1);
    __syncthreads();
    if (!*last_flag) return;
#pragma unroll
    for (int f = 0; f < FM; ++f) acc[f] = f4_t{0.f, 0.f, 0.f, 0.f};
    const float* src = a.part + (rt * S * 4 + wave) * (FM * 256);
    for (int s0 = 0; s0 < S; s0 += 8) {
      float pv[8][FM * 4];
#pragma unroll
      for (int j = 0; j < 8; ++j)
        if (s0 + j < S)
#pragma unroll
          for (int e = 0; e < FM * 4; ++e) pv[j][e] = ld_dev(src + (int64_t)(s0 + j) * (4 * FM * 256) + e * 64 + lane);
#pragma unroll
      for (int j = 0; j < 8; ++j)
        if (s0 + j < S)
#pragma unroll
          for (int e = 0; e < FM * 4; ++e) acc[e >> 2][e & 3] += pv[j][e];
    }
    if (tid == 0) counter_reset(&a.counters[rt]);
  }

  // 4. store out^T fragment: lane (col + 16 * (row / 4)), element row % 4 -> 4 consecutive rows
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
// tm[m, j] = sum_red act[m, red] B(red, j) with B = L[red, j] (forward) or R[j, red] (backward).
// Unit = 64 adapter columns (one 16-column fragment per wave) x one reduction slice.
constexpr int kAdSlice = SLIM_DECODE_AD_SLICE;
constexpr int kLdL = 64 + 8;

template <bool BWD, int FM>
SLIM_DEV void decode_adapter_unit(const LayerArgs& a, int64_t v, _Float16* ls, int* last_flag) {
  constexpr int kSteps = kAdSlice / 32;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int SA = a.ad_split;
  const int64_t jb = v / SA;
  const int sa = (int)(v - jb * SA);
  const int64_t j0 = jb * 64;
  const int64_t r0 = (int64_t)sa * kAdSlice;
  const int nst = (int)min((int64_t)kSteps, (a.red - r0) / 32);
  const bool bf16 = a.act_bf16 != 0;
  const int g = lane >> 4;
  const int64_t jcol = j0 + 16 * wave + (lane & 15);

  // activation fragments (A operand: rows m) and adapter-factor fragments (B operand: columns j)
  h8_t af[kSteps][FM];
  u32x4_t bq[kSteps];
#pragma unroll
  for (int t = 0; t < kSteps; ++t) {
    if (t < nst) {
      const int64_t rk = r0 + 32 * t + 8 * g;
#pragma unroll
      for (int f = 0; f < FM; ++f) {
        const int64_t m = 16 * f + (lane & 15);
        af[t][f] = m < a.M ? act8(*reinterpret_cast<const u32x4_t*>(a.act + m * a.red + rk), bf16) : zero_h8();
      }
      if (BWD) bq[t] = jcol < a.r ? *reinterpret_cast<const u32x4_t*>(a.ad_in + jcol * a.red + rk) : zero_u4();
    }
  }
  if (!BWD) {
    // L[red, j] rows are contiguous along j: stage the [slice x 64] tile in LDS, read columns
    u32x4_t lv[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int q = tid + 256 * i, kr = q >> 3, jc = q & 7;
      const int64_t gk = r0 + kr, gj = j0 + 8 * jc;
      lv[i] = (kr < 32 * nst && gj < a.r) ? *reinterpret_cast<const u32x4_t*>(a.ad_in + gk * a.r + gj) : zero_u4();
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int q = tid + 256 * i, kr = q >> 3, jc = q & 7;
      *reinterpret_cast<u32x4_t*>(&ls[kr * kLdL + 8 * jc]) = lv[i];
    }
    __syncthreads();
  }
  f4_t acc[FM];
#pragma unroll
  for (int f = 0; f < FM; ++f) acc[f] = f4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int t = 0; t < kSteps; ++t) {
    if (t < nst) {
      h8_t bv;
      if (BWD) {
        bv = __builtin_bit_cast(h8_t, bq[t]);
      } else {
        const int col = 16 * wave + (lane & 15);
#pragma unroll
        for (int e = 0; e < 8; ++e) bv[e] = ls[(32 * t + 8 * g + e) * kLdL + col];
      }
#pragma unroll
      for (int f = 0; f < FM; ++f) acc[f] = mfma16(af[t][f], bv, acc[f]);
    }
  }
  // D[m][j] fragment: lane (j + 16 * (m / 4)), element m % 4
  auto store_tm = [&](const f4_t* res) {
#pragma unroll
    for (int f = 0; f < FM; ++f)
#pragma unroll
      for (int vv = 0; vv < 4; ++vv) {
        const int64_t m = 16 * f + 4 * g + vv;
        if (m < a.M && jcol < a.r) a.tm[m * a.r + jcol] = __builtin_bit_cast(uint16_t, (_Float16)res[f][vv]);
      }
  };
  if (SA == 1) {
    store_tm(acc);
    return;
  }
  float* dst = a.tpart + ((jb * SA + sa) * 4 + wave) * (FM * 256);
#pragma unroll
  for (int f = 0; f < FM; ++f)
#pragma unroll
    for (int vv = 0; vv < 4; ++vv) st_dev(dst + (f * 4 + vv) * 64 + lane, acc[f][vv]);
  drain_stores();
  __syncthreads();
  if (tid == 0) *last_flag = counter_arrive(&a.tcounters[jb]) == (uint32_t)(SA - 1);
  __syncthreads();
  if (!*last_flag) return;
#pragma unroll
  for (int f = 0; f < FM; ++f) acc[f] = f4_t{0.f, 0.f, 0.f, 0.f};
  const float* src = a.tpart + (jb * SA * 4 + wave) * (FM * 256);
  for (int s0 = 0; s0 < SA; s0 += 8) {
    float pv[8][FM * 4];
#pragma unroll
    for (int j = 0; j < 8; ++j)
      if (s0 + j < SA)
#pragma unroll
        for (int e = 0; e < FM * 4; ++e) pv[j][e] = ld_dev(src + (int64_t)(s0 + j) * (4 * FM * 256) + e * 64 + lane);
#pragma unroll
    for (int j = 0; j < 8; ++j)
      if (s0 + j < SA)
#pragma unroll
        for (int e = 0; e < FM * 4; ++e) acc[e >> 2][e & 3] += pv[j][e];
  }
  if (tid == 0) counter_reset(&a.tcounters[jb]);
  store_tm(acc);
}

// Blocks [0, row_tiles * split) are sparse units; the rest are adapter units.
template <bool BWD, int FM>
__global__ void __launch_bounds__(256) k_decode(LayerArgs a) {
  extern __shared__ __attribute__((aligned(16))) _Float16 lds[];
  __shared__ int last_flag;
  const int64_t nW = a.row_tiles * a.split;
  const int64_t b = blockIdx.x;
  if (b < nW) decode_sparse_unit<BWD, FM>(a, b, lds, &last_flag);
  else decode_adapter_unit<BWD, FM>(a, b - nW, lds, &last_flag);
}

// ============================================================ small-M: adapter second product
// out[m, row] += sum_j tm[m, j] ap(row, j), ap = R[j, row] (forward) or L[row, j] (backward).
// One wave per 16 output rows; all fragment loads are issued before the first MFMA.
template <bool BWD, int FM>
__global__ void __launch_bounds__(64) k_adapter_out(LayerArgs a) {
  constexpr int kMaxSteps = 8;                     // 256 adapter ranks per round of loads
  const int lane = threadIdx.x, g = lane >> 4;
  const int64_t row0 = (int64_t)blockIdx.x * 16;
  const int64_t row = row0 + (lane & 15);
  const int64_t lrow = row < a.rows ? row : a.rows - 1;
  f4_t acc[FM];
#pragma unroll
  for (int f = 0; f < FM; ++f) acc[f] = f4_t{0.f, 0.f, 0.f, 0.f};
  for (int64_t jbase = 0; jbase < a.r; jbase += 32 * kMaxSteps) {
    h8_t av[kMaxSteps], bv[kMaxSteps][FM];
#pragma unroll
    for (int t = 0; t < kMaxSteps; ++t) {
      const int64_t jj = jbase + 32 * t + 8 * g;
      if (jj < a.r) {
        if (BWD) {
          av[t] = __builtin_bit_cast(h8_t, *reinterpret_cast<const u32x4_t*>(a.ad_out + lrow * a.r + jj));
        } else {
#pragma unroll
          for (int e = 0; e < 8; ++e) av[t][e] = __builtin_bit_cast(_Float16, a.ad_out[(jj + e) * a.rows + lrow]);
        }
#pragma unroll
        for (int f = 0; f < FM; ++f) {
          const int64_t m = 16 * f + (lane & 15);
          bv[t][f] = m < a.M ? __builtin_bit_cast(h8_t, *reinterpret_cast<const u32x4_t*>(a.tm + m * a.r + jj))
                             : zero_h8();
        }
      } else {
        av[t] = zero_h8();
#pragma unroll
        for (int f = 0; f < FM; ++f) bv[t][f] = zero_h8();
      }
    }
#pragma unroll
    for (int t = 0; t < kMaxSteps; ++t)
      if (jbase + 32 * t < a.r)
#pragma unroll
        for (int f = 0; f < FM; ++f) acc[f] = mfma16(av[t], bv[t][f], acc[f]);
  }
  const int64_t rr = row0 + 4 * g;
  if (rr < a.rows) {
#pragma unroll
    for (int f = 0; f < FM; ++f) {
      const int64_t m = 16 * f + (lane & 15);
      if (m < a.M) {
        f4_t* p = reinterpret_cast<f4_t*>(a.out + m * a.rows + rr);
        *p = *p + acc[f];
      }
    }
  }
}

// ============================================================ large-M tile kernel
// Block = 4 waves; wave (wr, wc) owns rows [row0 + 128 wr, +128) as 4 fragments of 32 and columns
// [m0 + 64 wc, +64) as 2 fragments of 32 (a 128 x 64 accumulator on 32x32x32 sparse MFMA). Per
// 128-wide chunk: activations [128 x 128] in a double-buffered LDS tile (staged through
// registers one chunk ahead), packed words in registers two chunks ahead.
constexpr int kTR = 256, kTC = 128, kTLd = 136, kTThreads = 256;
constexpr int kTXV = kTC * 16 / kTThreads;      // 16-byte activation vectors per thread per chunk

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
__global__ void __launch_bounds__(kTThreads) k_tile(LayerArgs a) {
  __shared__ __attribute__((aligned(16))) _Float16 xs[2][kTC][kTLd];
  __shared__ __attribute__((aligned(16))) _Float16 ss[2][2][128];    // backward: scale row per row half
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wr = wave & 1, wc = wave >> 1;
  const int ha = lane >> 5;
  const int64_t row0 = (int64_t)blockIdx.x * kTR, m0 = (int64_t)blockIdx.y * kTC;
  const int64_t wrow0 = row0 + 128 * wr;
  const int64_t nch = a.red / 128;
  const bool bf16 = a.act_bf16 != 0;

  const uint32_t* cp[4];
  const uint32_t* mp[4];
  const uint16_t* sp[4];
#pragma unroll
  for (int fn = 0; fn < 4; ++fn) {
    int64_t arow = wrow0 + 32 * fn + (lane & 31);
    if (arow >= a.rows) arow = a.rows - 1;
    cp[fn] = a.codes + arow * (a.red / 16) + 4 * ha;
    mp[fn] = a.meta + arow * (a.red / 32) + 2 * ha;
    sp[fn] = a.scales + arow * (a.red / 128);
  }

  u32x4_t xr[kTXV];
  u32x4_t sr = zero_u4();
  auto load_x = [&](int64_t c) {
#pragma unroll
    for (int i = 0; i < kTXV; ++i) {
      const int q = tid + kTThreads * i, m = q >> 4, vc = q & 15;
      const int64_t gm = m0 + m;
      xr[i] = gm < a.M ? *reinterpret_cast<const u32x4_t*>(a.act + gm * a.red + c * 128 + 8 * vc) : zero_u4();
    }
    if (BWD && tid < 32) {
      // backward: scale row s16[n, g] of each row half's 128-row group, for this chunk
      const int h = tid >> 4, vc = tid & 15;
      int64_t gr = row0 + 128 * h;
      if (gr >= a.rows) gr = a.rows - 1;
      sr = *reinterpret_cast<const u32x4_t*>(a.scales + (gr / 128) * a.red + c * 128 + 8 * vc);
    }
  };
  auto store_x = [&](int buf) {
#pragma unroll
    for (int i = 0; i < kTXV; ++i) {
      const int q = tid + kTThreads * i, m = q >> 4, vc = q & 15;
      *reinterpret_cast<h8_t*>(&xs[buf][m][8 * vc]) = act8(xr[i], bf16);
    }
    if (BWD && tid < 32) *reinterpret_cast<u32x4_t*>(&ss[buf][tid >> 4][8 * (tid & 15)]) = sr;
  };

  f16_t acc[4][2];
#pragma unroll
  for (int fn = 0; fn < 4; ++fn)
#pragma unroll
    for (int fm = 0; fm < 2; ++fm)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[fn][fm][v] = 0.f;

  TileA cur, nxt;
  tile_load_a<BWD>(cp, mp, sp, 0, cur);
  load_x(0);
  if (nch > 1) tile_load_a<BWD>(cp, mp, sp, 1, nxt);
  store_x(0);
  __syncthreads();
  if (nch > 1) load_x(1);

  for (int64_t c = 0; c < nch; ++c) {
    const int buf = (int)(c & 1);
#pragma unroll
    for (int st = 0; st < 4; ++st) {
      h8_t av[4];
      h16_t bv[2];
#pragma unroll
      for (int fn = 0; fn < 4; ++fn)
        av[fn] = BWD ? dequant_word_int(cur.cw[fn][st]) : dequant_word(cur.cw[fn][st], splat_h2(cur.sw[fn]));
      const int off = b_chunk_offset<32>(lane, st);
#pragma unroll
      for (int fm = 0; fm < 2; ++fm) {
        const _Float16* p = &xs[buf][64 * wc + 32 * fm + (lane & 31)][off];
        h8_t lo = *reinterpret_cast<const h8_t*>(p), hi = *reinterpret_cast<const h8_t*>(p + 64);
        if (BWD) {
          lo = mul_h8(lo, *reinterpret_cast<const h8_t*>(&ss[buf][wr][off]));
          hi = mul_h8(hi, *reinterpret_cast<const h8_t*>(&ss[buf][wr][off + 64]));
        }
        bv[fm] = cat16(lo, hi);
      }
#pragma unroll
      for (int fn = 0; fn < 4; ++fn)
#pragma unroll
        for (int fm = 0; fm < 2; ++fm)
          acc[fn][fm] = smfmac32(av[fn], bv[fm], acc[fn][fm], (int)cur.mw[fn][st >> 1], st & 1);
    }
    if (c + 1 < nch) store_x(buf ^ 1);       // activations of chunk c+1 (loaded one chunk ago)
    __syncthreads();
    cur = nxt;
    if (c + 2 < nch) {
      tile_load_a<BWD>(cp, mp, sp, c + 2, nxt);
      load_x(c + 2);
    }
  }

  // adapter second product: out^T[row, m] += sum_j ap(row, j) tm[m, j], 32 ranks per round,
  // on 32x32x16 fp16 MFMA. Forward ap = R^T, staged through LDS transposed.
  if (a.r > 0) {
    constexpr int kAtLd = 40;
    _Float16(*at)[kAtLd] = reinterpret_cast<_Float16(*)[kAtLd]>(&xs[0][0][0]);   // [256][40]
    static_assert(kTR * kAtLd <= 2 * kTC * kTLd, "adapter slab must fit in the activation buffers");
    for (int64_t jb = 0; jb < a.r; jb += 32) {
      h8_t bv[2][2];       // [kk][fm]: tm[m][jb + 16 kk + 8 ha .. +7]
      h8_t av[2][4];       // [kk][fn]
#pragma unroll
      for (int kk = 0; kk < 2; ++kk) {
        const int64_t jj = jb + 16 * kk + 8 * ha;
#pragma unroll
        for (int fm = 0; fm < 2; ++fm) {
          const int64_t m = m0 + 64 * wc + 32 * fm + (lane & 31);
          bv[kk][fm] = (m < a.M && jj < a.r)
                           ? __builtin_bit_cast(h8_t, *reinterpret_cast<const u32x4_t*>(a.tm + m * a.r + jj))
                           : zero_h8();
        }
        if (BWD) {
#pragma unroll
          for (int fn = 0; fn < 4; ++fn) {
            int64_t rw = wrow0 + 32 * fn + (lane & 31);
            if (rw >= a.rows) rw = a.rows - 1;
            av[kk][fn] = jj < a.r ? __builtin_bit_cast(h8_t, *reinterpret_cast<const u32x4_t*>(a.ad_out + rw * a.r + jj))
                                  : zero_h8();
          }
        }
      }
      if (!BWD) {
        // R[jb .. jb+31][row0 .. row0+255] -> at[row][j]
        u32x4_t rv[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int q = tid + kTThreads * i, jr = q >> 5, nc = q & 31;
          const int64_t gj = jb + jr, gn = row0 + 8 * nc;
          rv[i] = (gj < a.r && gn < a.rows) ? *reinterpret_cast<const u32x4_t*>(a.ad_out + gj * a.rows + gn) : zero_u4();
        }
        __syncthreads();
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int q = tid + kTThreads * i, jr = q >> 5, nc = q & 31;
          const h8_t hv = __builtin_bit_cast(h8_t, rv[i]);
#pragma unroll
          for (int e = 0; e < 8; ++e) at[8 * nc + e][jr] = hv[e];
        }
        __syncthreads();
#pragma unroll
        for (int kk = 0; kk < 2; ++kk)
#pragma unroll
          for (int fn = 0; fn < 4; ++fn)
            av[kk][fn] = *reinterpret_cast<const h8_t*>(&at[128 * wr + 32 * fn + (lane & 31)][16 * kk + 8 * ha]);
      }
#pragma unroll
      for (int kk = 0; kk < 2; ++kk)
#pragma unroll
        for (int fn = 0; fn < 4; ++fn)
#pragma unroll
          for (int fm = 0; fm < 2; ++fm) acc[fn][fm] = mfma32(av[kk][fn], bv[kk][fm], acc[fn][fm]);
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

// ------------------------------------------------------------------------------ launch
template <bool BWD>
int launch_layer(const LayerArgs& a, const SlimPlan& p, const uint16_t* act, int act_bf16, char* ws, hipStream_t s) {
  if (p.decode) {
    {
      SlimKernelTimer timer(BWD ? "decode_bwd" : "decode_fwd", s);
      dim3 grid((unsigned)(p.sp_row_tiles * p.sp_split + (a.r > 0 ? p.ad_jblocks * p.ad_split : 0)));
      switch (p.dec_fm) {
        case 1: hipLaunchKernelGGL((k_decode<BWD, 1>), grid, dim3(256), p.lds_bytes, s, a); break;
        case 2: hipLaunchKernelGGL((k_decode<BWD, 2>), grid, dim3(256), p.lds_bytes, s, a); break;
        default: hipLaunchKernelGGL((k_decode<BWD, 4>), grid, dim3(256), p.lds_bytes, s, a); break;
      }
      if (hipGetLastError() != hipSuccess) return SLIM_EDEVICE;
    }
    if (a.r > 0) {
      SlimKernelTimer timer(BWD ? "adapter_out_bwd" : "adapter_out_fwd", s);
      dim3 grid((unsigned)((a.rows + 15) / 16));
      switch (p.dec_fm) {
        case 1: hipLaunchKernelGGL((k_adapter_out<BWD, 1>), grid, dim3(64), 0, s, a); break;
        case 2: hipLaunchKernelGGL((k_adapter_out<BWD, 2>), grid, dim3(64), 0, s, a); break;
        default: hipLaunchKernelGGL((k_adapter_out<BWD, 4>), grid, dim3(64), 0, s, a); break;
      }
      if (hipGetLastError() != hipSuccess) return SLIM_EDEVICE;
    }
    return SLIM_OK;
  }
  if (a.r > 0) {
    int st = slim_launch_adapter_gemm(BWD, act, act_bf16, a.M, a.red, a.ad_in, a.r, p, ws, s);
    if (st != SLIM_OK) return st;
  }
  SlimKernelTimer timer(BWD ? "tile_bwd" : "tile_fwd", s);
  dim3 grid((unsigned)p.sp_row_tiles, (unsigned)p.sp_col_tiles);
  hipLaunchKernelGGL((k_tile<BWD>), grid, dim3(kTThreads), 0, s, a);
  return hipGetLastError() == hipSuccess ? SLIM_OK : SLIM_EDEVICE;
}

LayerArgs make_args(const SlimPlan& p, char* ws, const void* act, int dtype, int64_t M, int64_t rows, int64_t red,
                    const uint8_t* codes, const uint8_t* meta, const uint16_t* scales, const uint16_t* ad_in,
                    const uint16_t* ad_out, int64_t r, float* out) {
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
  a.ad_in = ad_in;
  a.ad_out = ad_out;
  a.tm = reinterpret_cast<uint16_t*>(ws + p.off_t);
  a.out = out;
  a.split = p.sp_split;
  a.cps = p.sp_chunks_per_split;
  a.row_tiles = p.sp_row_tiles;
  a.ad_split = p.ad_split;
  a.ad_slice = p.ad_slice;
  a.ad_jblocks = p.ad_jblocks;
  a.part = reinterpret_cast<float*>(ws + p.off_ypart);
  a.tpart = reinterpret_cast<float*>(ws + p.off_tpart);
  a.counters = reinterpret_cast<uint32_t*>(ws + p.off_counters) + p.sp_counter_base;
  a.tcounters = reinterpret_cast<uint32_t*>(ws + p.off_counters);
  return a;
}

}  // namespace

extern "C" int slim_workspace_init(void* ws, size_t ws_bytes, void* stream) {
  if (!ws) return SLIM_EINVAL;
  if (ws_bytes < SLIM_COUNTER_SLOTS * 4) return SLIM_EWORKSPACE;
  return hipMemsetAsync(ws, 0, ws_bytes, (hipStream_t)stream) == hipSuccess ? SLIM_OK : SLIM_EDEVICE;
}

extern "C" int slim_linear(const void* X, int xdtype, int64_t M, int64_t N, int64_t K, const uint8_t* codes,
                           const uint8_t* meta, const uint16_t* scales, const uint16_t* L, const uint16_t* R,
                           int64_t r, float* Y, void* ws, size_t ws_bytes, void* stream) {
  SlimPlan p;
  int st = slim_check_linear(false, X, xdtype, M, N, K, codes, meta, scales, L, R, r, Y, ws, ws_bytes, &p);
  if (st != SLIM_OK) return st;
  char* w = reinterpret_cast<char*>(ws);
  const LayerArgs a = make_args(p, w, X, xdtype, M, N, K, codes, meta, scales, L, R, r, Y);
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
