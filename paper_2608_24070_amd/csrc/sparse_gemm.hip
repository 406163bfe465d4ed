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
//    computes 512 x 96 or 512 x 128 output tiles on 32x32x32 sparse MFMA, with activations and
//    packed words streamed into LDS rings by direct loads, and adds the second adapter product in
//    its epilogue.
// Every global load is issued unconditionally from a clamped (or, through a buffer resource,
// range-checked) address and masked when used: a load under a branch makes the compiler wait
// for it at the join, which serialises what should be one round of memory traffic.
#include <mutex>
#include <type_traits>

#include "slim_device.h"
#include "slim_launch.h"
#include "slim_timing.h"

namespace {

constexpr int kDecodeMaxUnits = SLIM_DECODE_MAX_UNITS;

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
  const uint16_t* ad_p;    // adapter second factor [rows, r]: 32 x 16 tiles (forward, from
                           // slim_pack_adapter) or row-major (backward, L as given)
  int p_tiled;             // ad_p is in 32 x 16 tiles
  // 4-bit adapters (slim_linear_qa): codes of Q = L^T [r, red/8 words] and P = R^T [rows, r/8 words]
  // with fp16 group-128 scales along the reduction of each product; null for fp16 adapters
  const uint32_t* q4;
  const uint16_t* q4s;     // [r, ceil(red/128)]
  const uint32_t* p4;
  const uint16_t* p4s;     // [rows, ceil(r/128)]
  const uint16_t* ad_pb;   // large M: the factor in 32 x 16 tiles (ad_p, or a re-laid copy)
  uint16_t* tm;            // fp16 adapter intermediate of the row-scaled activations: row-major
                           // [M, r] (small M), 32 x 16 tiles (large M)
  float* trinv;            // small M: 2^-e per row of tm (written by the adapter units)
  const float* rowinv;     // large M: 2^-e per activation row (the rows were scaled by 2^e), or null
  float* out;              // [M, rows]
  // small-M path
  int split;               // reduction splits of the sparse product
  int64_t row_tiles;       // 64-row tiles (small M) or 512-row tiles (large M)
  int64_t units;           // small M: row tiles per sparse block
  int64_t col_tiles;       // 96- or 128-column tiles (large M)
  int ad_split;            // reduction splits of the adapter's first product
  int ad_sub;              // small M: slices of SLIM_DECODE_AD_SLICE positions per adapter wave
  int64_t ad_jblocks;      // 16-wide column blocks of the adapter rank (small M)
  float* part;             // sparse split partials
  float* tpart;            // adapter split partials
  uint32_t* tcounters;     // per adapter column block
  int finish;              // sparse partials go to k_finish (split > 1 or an adapter)
};

SLIM_DEV u32x4_t zero_u4() { return u32x4_t{0u, 0u, 0u, 0u}; }
SLIM_DEV int64_t clamp_hi(int64_t x, int64_t hi) { return x < hi ? x : hi; }

// Reduce the split partials of one adapter column block, run by wave 0 of each unit (the unit's
// sum is in its registers): every unit stores its FM x 4 accumulator values per lane (device
// scope, one 16-byte store per fragment) and its per-row maxima of |activation| (16 words per
// fragment), and the last one to arrive sums all S partials in split order and takes the maxima's
// maximum. A partial is [FM][64 lanes][4] fp32; the maxima follow all S partials, [S][FM][16].
template <int FM>
SLIM_DEV bool split_reduce_wave(f4_t* acc, uint32_t* amx, float* part, int S, int s, uint32_t* counter) {
  const int lane = threadIdx.x & 63;
  const rsrc_t pr = make_rsrc(part, (int64_t)S * FM * 1088);
  auto off = [&](int ss, int f) { return (uint32_t)(((ss * FM + f) * 256 + 4 * lane) * 4); };
  auto moff = [&](int ss, int f) { return (uint32_t)(S * FM * 1024 + ((ss * FM + f) * 16 + (lane & 15)) * 4); };
#pragma unroll
  for (int f = 0; f < FM; ++f) {
    st_dev4(pr, off(s, f), acc[f]);
    if (lane < 16) st_dev1(pr, moff(s, f), amx[f]);
  }
  drain_stores();
  uint32_t prev = 0;
  if (lane == 0) prev = counter_arrive(counter);
  if (__shfl(prev, 0) != (uint32_t)(S - 1)) return false;
#pragma unroll
  for (int f = 0; f < FM; ++f) acc[f] = f4_t{0.f, 0.f, 0.f, 0.f};
  constexpr int kR = 16 / FM;   // partials per load round
  for (int s0 = 0; s0 < S; s0 += kR) {
    f4_t pv[kR][FM];
    uint32_t pm[kR][FM];
#pragma unroll
    for (int j = 0; j < kR; ++j) {
      const int ss = s0 + j < S ? s0 + j : S - 1;
#pragma unroll
      for (int f = 0; f < FM; ++f) {
        pv[j][f] = ld_dev4(pr, off(ss, f));
        pm[j][f] = ld_dev1(pr, moff(ss, f));
      }
    }
#pragma unroll
    for (int j = 0; j < kR; ++j)
      if (s0 + j < S)
#pragma unroll
        for (int f = 0; f < FM; ++f) {
          acc[f] = acc[f] + pv[j][f];
          amx[f] = max(amx[f], pm[j][f]);
        }
  }
  if (lane == 0) counter_reset(counter);
  return true;
}

// ============================================================ small-M: sparse split units
// Unit = 64 rows (16 per wave, one 16-row block of the packed layout) x one slice of 4G
// quantisation groups. Lane group qa (lane / 16) of the 16x16x64 sparse MFMA owns G whole
// groups: per group one row's code words (32 B), index words (16 B) and scale, which the 16 lanes
// of a lane group (16 rows of one block) read from one contiguous piece.
//
// A block runs up to NU units of one slice, consecutive row tiles [rt0, rt1): it stages the
// slice's activations in LDS once and loads each unit's packed words while the unit before is
// computed. Results stay in registers until every load has been issued and are stored at the end:
// a store between the loads would make the compiler's wait for one unit's words also wait for
// the next unit's. In the backward the staged activations carry the scales of a 128-row group,
// so a block runs at most the two row tiles of one group (rt0 even).
template <int G>
struct DecodeWords {
  u32x4_t cw[2 * G], mw[G];
  uint32_t sw[G];
};

template <bool BWD, int G>
SLIM_DEV void decode_load_words(const LayerArgs& a, int64_t rt, int64_t cl, int lane, int wave, DecodeWords<G>& w) {
  const int64_t nchunks = a.red / 128;
  const int64_t lrow = clamp_hi(rt * 64 + 16 * wave + (lane & 15), a.rows - 1);
#pragma unroll
  for (int gi = 0; gi < G; ++gi) {
    const int64_t ch = clamp_hi(cl + gi, nchunks - 1);
    const int64_t slot = packed_slot(lrow, ch, nchunks);
    const uint32_t* cp = a.codes + 8 * slot;
    w.cw[2 * gi] = *reinterpret_cast<const u32x4_t*>(cp);
    w.cw[2 * gi + 1] = *reinterpret_cast<const u32x4_t*>(cp + 4);
    w.mw[gi] = *reinterpret_cast<const u32x4_t*>(a.meta + 4 * slot);
    w.sw[gi] = BWD ? 0u : (uint32_t)a.scales[slot];
  }
}

template <bool BWD, int FM, int G, int NU>
SLIM_DEV void decode_sparse_range(const LayerArgs& a, int s, int64_t rt0, int64_t rt1, _Float16* xs) {
  constexpr int MC = 16 * FM;
  constexpr int SL = 512 * G;              // reduction positions per slice
  constexpr int LDX = SL + 8;
  constexpr int VPR = SL / 8;              // 16-byte activation vectors per row of the slice
  constexpr int XV = MC * VPR / 256;       // ... per thread
  static_assert(!BWD || NU <= 2, "backward blocks stay within one 128-row group: activations carry its scales");
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int S = a.split;
  const int64_t nchunks = a.red / 128;
  const int64_t c0 = (int64_t)s * 4 * G;
  const int64_t red0 = c0 * 128;
  const bool bf16 = a.act_bf16 != 0;
  const int qa = lane >> 4;
  const int64_t cl = c0 + (int64_t)qa * G;      // first chunk (group) of this lane group

  DecodeWords<G> wb[NU > 1 ? 2 : 1];
  const int64_t sgroup = rt0 * 64 / 128;
  // Activations of the slice: wave w stages rows m = w + 4 i (i < MC / 4), each row as G runs of 64
  // lanes x 8 positions (position 8 (lane + 64 j)), so a wave holds whole rows: each row's scaling
  // exponent is a reduction within one wave, with no exchange between waves.
  constexpr int RW = MC / 4;                 // rows per wave
  u32x4_t xv[RW][G], sv[G];
#pragma unroll
  for (int i = 0; i < RW; ++i)
#pragma unroll
    for (int j = 0; j < G; ++j) {
      const int64_t pos = clamp_hi(red0 + 8 * (lane + 64 * j), a.red - 8);
      xv[i][j] = *reinterpret_cast<const u32x4_t*>(a.act + clamp_hi(wave + 4 * i, a.M - 1) * a.red + pos);
    }
  if (BWD)
#pragma unroll
    for (int j = 0; j < G; ++j)
      sv[j] = *reinterpret_cast<const u32x4_t*>(a.scales + sgroup * a.red + clamp_hi(red0 + 8 * (lane + 64 * j), a.red - 8));
  // the first unit's packed words after the activations: loads complete in order, so the staging
  // below waits for the activations only and runs while the words are still in flight
  decode_load_words<BWD, G>(a, rt0, cl, lane, wave, wb[0]);
  // The staged B operand in fp32: the activations, in the backward times the fp16 scales of the
  // block's 128-row group (the product is formed exactly in fp32 and rounded once, below), scaled
  // per row (see act_exponent).
  // (the input type is one uniform choice around the whole staging, not a branch per vector)
  __shared__ float runscale[MC];
  auto stage = [&](auto bfc) {
  constexpr bool kBf16 = decltype(bfc)::value;
#pragma unroll
  for (int i = 0; i < RW; ++i) {
    const int m = wave + 4 * i;
    float xf[G][8];
    uint32_t mx = 0;
#pragma unroll
    for (int j = 0; j < G; ++j) {
      const bool ok = m < a.M && red0 + 8 * (lane + 64 * j) < a.red;
      act8_to_f(xv[i][j], kBf16, xf[j]);
      if (BWD) {
        float sf[8];
        act8_to_f(sv[j], false, sf);
#pragma unroll
        for (int e = 0; e < 8; ++e) xf[j][e] *= sf[e];
      }
#pragma unroll
      for (int e = 0; e < 8; ++e) xf[j][e] = ok ? xf[j][e] : 0.f;
      mx = max(mx, max_abs_bits8(xf[j]));
    }
    const int e = act_exponent(wave_max_u32(mx));
    const float sc = exp2i(e);
    if (lane == 0) runscale[m] = exp2i(-e);
#pragma unroll
    for (int j = 0; j < G; ++j) *reinterpret_cast<h8_t*>(&xs[m * LDX + 8 * (lane + 64 * j)]) = scale8_to_h(xf[j], sc);
  }
  };
  if (bf16) stage(std::true_type{});
  else stage(std::false_type{});
  __syncthreads();
  float unscale[FM];
#pragma unroll
  for (int f = 0; f < FM; ++f) unscale[f] = runscale[16 * f + (lane & 15)];

  const int qb = lane >> 4;
  const int pbase = 128 * G * (qb >> 1) + 8 * (qb & 1);
  // the sparse product of one unit; groups past the reduction (a ragged last slice) are masked,
  // which only a block whose slice runs past the end needs (a uniform choice between two copies)
  auto unit_mfma = [&](const DecodeWords<G>& w, f4_t* acc, auto maskc) {
    constexpr bool kMask = decltype(maskc)::value;
#pragma unroll
    for (int gi = 0; gi < G; ++gi) {
      const bool gok = cl + gi < nchunks;
      const h2_t s2 = splat_h2(w.sw[gi]);
#pragma unroll
      for (int t4 = 0; t4 < 8; ++t4) {
        const uint32_t word = w.cw[2 * gi + (t4 >> 2)][t4 & 3];
        h8_t av = BWD ? dequant_word_int(word) : dequant_word(word, s2);
        if (kMask) av = gok ? av : zero_h8();
        const int idx = (int)w.mw[gi][t4 >> 1];
        const int p0 = pbase + 16 * (8 * gi + t4);
#pragma unroll
        for (int f = 0; f < FM; ++f) {
          const _Float16* xr = xs + (16 * f + (lane & 15)) * LDX + p0;
          acc[f] = smfmac16(av, cat16(*reinterpret_cast<const h8_t*>(xr), *reinterpret_cast<const h8_t*>(xr + 256 * G)),
                            acc[f], idx, t4 & 1);
        }
      }
    }
  };
  const bool ragged = c0 + 4 * G > nchunks;
  f4_t out[NU][FM];
#pragma unroll
  for (int k = 0; k < NU; ++k) {
    if (rt0 + k >= rt1) break;
    // the next unit's words (the last unit reloads itself: loads stay unconditional)
    if (NU > 1) {
      decode_load_words<BWD, G>(a, rt0 + k + 1 < rt1 ? rt0 + k + 1 : rt1 - 1, cl, lane, wave, wb[(k + 1) & 1]);
      __builtin_amdgcn_sched_barrier(0);   // keep them ahead of this unit's work
    }
    f4_t acc[FM];
#pragma unroll
    for (int f = 0; f < FM; ++f) acc[f] = f4_t{0.f, 0.f, 0.f, 0.f};
    if (ragged) unit_mfma(wb[k & 1], acc, std::true_type{});
    else unit_mfma(wb[k & 1], acc, std::false_type{});
#pragma unroll
    for (int f = 0; f < FM; ++f) out[k][f] = acc[f] * unscale[f];   // lane (m + 16 (row / 4)): column m = lane % 16
  }

#pragma unroll
  for (int k = 0; k < NU; ++k) {
    if (rt0 + k >= rt1) break;
    const int64_t rt = rt0 + k;
    if (a.finish) {
      // k_finish sums the split partials (and adds the adapter); the kernel boundary orders them.
      // Lanes of columns past M hold nothing and store nothing.
      float* dst = a.part + ((rt * S + s) * 4 + wave) * (int64_t)(FM * 256);
#pragma unroll
      for (int f = 0; f < FM; ++f)
        if (16 * f + (lane & 15) < a.M) *reinterpret_cast<f4_t*>(dst + f * 256 + 4 * lane) = out[k][f];
      continue;
    }
    // out^T fragment: lane (col + 16 * (row / 4)), element row % 4 -> 4 consecutive rows
    const int64_t rr = rt * 64 + 16 * wave + 4 * (lane >> 4);
    if (rr < a.rows) {
#pragma unroll
      for (int f = 0; f < FM; ++f) {
        const int64_t m = 16 * f + (lane & 15);
        if (m < a.M) *reinterpret_cast<f4_t*>(a.out + m * a.rows + rr) = out[k][f];
      }
    }
  }
}

// ============================================================ small-M: adapter first-product units
// tm[m, j] = sum_red act[m, red] Q[j, red]. Unit = 16 adapter columns x 4 parts of ad_sub slices
// of SLIM_DECODE_AD_SLICE (128) reduction positions: wave w takes part w (more than one slice when
// the reduction is long, so that there are at most about 8 splits), reading both operands straight
// from global memory.
// The four parts are added in LDS in part order, and the last unit of a column block to finish
// sums the units' partials in split order. The partial a unit hands over is one 16 x 16
// fragment per 16 activation rows (1 KB), which keeps the last unit's loads few.
constexpr int kAdSlice = SLIM_DECODE_AD_SLICE;

template <int FM, bool QA>
SLIM_DEV void decode_adapter_unit(const LayerArgs& a, int64_t v, f4_t* red_lds) {
  constexpr int kSteps = kAdSlice / 32;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int SA = a.ad_split;
  const int64_t jb = v / SA;                    // 16-column block
  const int sa = (int)(v - jb * SA);
  const int64_t r0 = ((int64_t)sa * 4 + wave) * a.ad_sub * kAdSlice;
  const bool bf16 = a.act_bf16 != 0;
  const int g = lane >> 4;
  const int64_t jcol = jb * 16 + (lane & 15);
  const int64_t jl = clamp_hi(jcol, a.r - 1);

  f4_t acc[FM];
  uint32_t amx[FM];   // largest |activation| of row 16 f + lane % 16 seen by this wave
#pragma unroll
  for (int f = 0; f < FM; ++f) {
    acc[f] = f4_t{0.f, 0.f, 0.f, 0.f};
    amx[f] = 0u;
  }
  // a.ad_sub consecutive slices of kAdSlice positions (one load round each); in a round at rs, step t
  // of lane group g covers positions rs + 32 t + 8 g .. + 7, so a step's loads of 16 rows read 64
  // contiguous bytes per row. A 4-bit factor row gives one 32-bit word of 8 codes per step; the
  // round lies in one 128-group (one scale).
  const int64_t red8 = a.red / 8, ngk = (a.red + 127) / 128;
  const rsrc_t rq4 = make_rsrc(a.q4, a.r * a.red / 2);
  // (the input type is one uniform choice around the rounds, not a branch per vector)
  auto rounds = [&](auto bfc) {
  constexpr bool kBf16 = decltype(bfc)::value;
  for (int sub = 0; sub < a.ad_sub; ++sub) {
    const int64_t rs = r0 + (int64_t)sub * kAdSlice;
    u32x4_t aq[kSteps][FM], bq[kSteps];
    uint32_t qw[kSteps], qs = 0;
#pragma unroll
    for (int t = 0; t < kSteps; ++t) {
      const int64_t rk = clamp_hi(rs + 32 * t + 8 * g, a.red - 8);
#pragma unroll
      for (int f = 0; f < FM; ++f)
        aq[t][f] = *reinterpret_cast<const u32x4_t*>(a.act + clamp_hi(16 * f + (lane & 15), a.M - 1) * a.red + rk);
      if (QA) qw[t] = __builtin_amdgcn_raw_buffer_load_b32(rq4, (uint32_t)((jl * red8 + rk / 8) * 4), 0, 0);
      else bq[t] = *reinterpret_cast<const u32x4_t*>(a.ad_q + jl * a.red + rk);
    }
    if (QA) qs = a.q4s[jl * ngk + clamp_hi(rs / 128, ngk - 1)];
    // this round's activations of row m = 16 f + lane % 16, scaled per row (see act_exponent): the
    // four lane groups of a row exchange their maxima; the round's product is unscaled in fp32
#pragma unroll
    for (int f = 0; f < FM; ++f) {
      const bool mok = 16 * f + (lane & 15) < a.M;
      float xf[kSteps][8];
      uint32_t mx = 0;
#pragma unroll
      for (int t = 0; t < kSteps; ++t) {
        const bool ok = mok && rs + 32 * t + 8 * g < a.red;
        act8_to_f(aq[t][f], kBf16, xf[t]);
#pragma unroll
        for (int e = 0; e < 8; ++e) xf[t][e] = ok ? xf[t][e] : 0.f;
        mx = max(mx, max_abs_bits8(xf[t]));
      }
      mx = col4_max_u32(mx);
      amx[f] = max(amx[f], mx);
      const int e = act_exponent(mx);
      const float sc = exp2i(e), inv = exp2i(-e);
      // D[j][m] = sum_k Q[j][k] X[m][k] (A = the factor's rows, B = the scaled activations): lane
      // (m + 16 (j / 4)) holds column m, so each lane unscales with its own row's factor
      f4_t racc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int t = 0; t < kSteps; ++t) {
        const bool kok = rs + 32 * t + 8 * g < a.red && jcol < a.r;
        const h8_t qv = QA ? dequant_word(qw[t], splat_h2(qs)) : __builtin_bit_cast(h8_t, bq[t]);
        racc = mfma16(kok ? qv : zero_h8(), scale8_to_h(xf[t], sc), racc);
      }
      acc[f] = acc[f] + racc * inv;
    }
  }
  };
  if (bf16) rounds(std::true_type{});
  else rounds(std::false_type{});
  // the unit's sum: waves 1..3 hand theirs (and their maxima) to wave 0 through LDS
  __shared__ uint32_t mx_lds[3][FM][64];
  if (wave > 0)
#pragma unroll
    for (int f = 0; f < FM; ++f) {
      red_lds[((wave - 1) * FM + f) * 64 + lane] = acc[f];
      mx_lds[wave - 1][f][lane] = amx[f];
    }
  __syncthreads();
  if (wave > 0) return;
#pragma unroll
  for (int w = 0; w < 3; ++w)
#pragma unroll
    for (int f = 0; f < FM; ++f) {
      acc[f] = acc[f] + red_lds[(w * FM + f) * 64 + lane];
      amx[f] = max(amx[f], mx_lds[w][f][lane]);
    }
  if (SA > 1 &&
      !split_reduce_wave<FM>(acc, amx, a.tpart + jb * (int64_t)SA * FM * 272, SA, sa, &a.tcounters[jb]))
    return;
  // amx is now the largest |activation| of the row over the whole reduction, the same in every
  // column block (each block's units cover the whole reduction with the same slices): T is stored
  // in fp16 scaled by that row's exponent, and column block 0 records 2^-e for the finish.
  // D[j][m] fragment: lane (m + 16 (j / 4)) holds ranks 16 jb + 4 g .. + 3 of row m = 16 f + lane % 16
  // (r % 16 == 0, so the four ranks are all in range or all past r)
#pragma unroll
  for (int f = 0; f < FM; ++f) {
    const int64_t m = 16 * f + (lane & 15);
    const int e = act_exponent(amx[f]);
    const f4_t ts = acc[f] * exp2i(e);
    h2_t lo2 = {(_Float16)ts[0], (_Float16)ts[1]}, hi2 = {(_Float16)ts[2], (_Float16)ts[3]};
    if (m < a.M && jb * 16 < a.r)
      *reinterpret_cast<u32x2_t*>(a.tm + m * a.r + jb * 16 + 4 * g) = u32x2_t{bits_of(lo2), bits_of(hi2)};
    if (m < a.M && jb == 0 && g == 0) a.trinv[m] = exp2i(-e);
  }
}

// Blocks [0, jblocks * ad_split) are adapter units (dispatched first: their reduction is the
// longer path); the rest are sparse blocks, block i of them taking slice i % split and row tiles
// [(i / split) NU', + NU') with NU' = a.units (at most NU).
template <bool BWD, int FM, int G, int NU, bool QA>
__global__ void __launch_bounds__(256) k_decode(LayerArgs a) {
  __shared__ __attribute__((aligned(16))) _Float16 xs[16 * FM * (512 * G + 8)];
  static_assert(sizeof(xs) >= 3 * FM * 64 * sizeof(f4_t), "adapter units sum their waves in xs");
  const int64_t nA = a.r > 0 ? a.ad_jblocks * a.ad_split : 0;
  const int64_t b = blockIdx.x;
  if (b < nA) {
    decode_adapter_unit<FM, QA>(a, b, reinterpret_cast<f4_t*>(xs));
    return;
  }
  const int64_t i = b - nA, S = a.split;
  const int64_t rt0 = (i / S) * a.units;
  const int64_t rt1 = rt0 + a.units < a.row_tiles ? rt0 + a.units : a.row_tiles;
  decode_sparse_range<BWD, FM, G, NU>(a, (int)(i % S), rt0, rt1, xs);
}

// ============================================================ small-M: finish
// out[m, row] = sum_s part_s[m, row] + sum_j tm[m, j] P[row, j]. One or two waves (NW) per 16 output
// rows; the split partials are summed in split order (deterministic) and the adapter's second
// product is accumulated on top with 16x16x32 fp16 MFMA; with two waves each takes alternate
// passes of the rank, and wave 0 adds wave 1's sum last. The partials share the MFMA output layout, so each
// lane reads its own four values per split and fragment (lanes of columns past M read nothing).
// The loads of the first adapter pass and of the first eight partials do not depend on each other
// and are all issued before any is used: one memory round trip for the common case (at most
// eight splits, a rank within the waves' first passes).
// Step t of a pass at jbase: lane group g takes ranks jbase + 32 t + 8 g .. + 7 (for both operands).
// A 4-bit P row gives one 32-bit word of 8 codes per step; the scale changes every 4 steps (one
// 128-rank group; jbase is a multiple of 128).
template <int FM, int kSteps, bool QA>
SLIM_DEV void finish_adapter_loads(const LayerArgs& a, int64_t jbase, int64_t lrow, int lane, u32x4_t* aq,
                                   u32x4_t (*bq)[FM], uint32_t* ps) {
  const int g = lane >> 4;
  const rsrc_t rp = make_rsrc(a.p4, a.rows * a.r / 2);
  const int64_t ngr = (a.r + 127) / 128;
#pragma unroll
  for (int t = 0; t < kSteps; ++t) {
    const int64_t jj = clamp_hi(jbase + 32 * t + 8 * g, a.r - 8);
    if (QA) {
      aq[t][0] = __builtin_amdgcn_raw_buffer_load_b32(rp, (uint32_t)((lrow * (a.r / 8) + jj / 8) * 4), 0, 0);
      if (t % 4 == 0) ps[t / 4] = a.p4s[lrow * ngr + clamp_hi((jbase + 32 * t) / 128, ngr - 1)];
    } else {
      // tiled: 8 consecutive ranks of a row stay within one 32 x 16 tile (jj % 16 is 0 or 8)
      const int64_t po = a.p_tiled ? ((lrow >> 5) * (a.r >> 4) + (jj >> 4)) * 512 + (lrow & 31) * 16 + (jj & 15)
                                   : lrow * a.r + jj;
      aq[t] = *reinterpret_cast<const u32x4_t*>(a.ad_p + po);
    }
#pragma unroll
    for (int f = 0; f < FM; ++f)
      bq[t][f] = *reinterpret_cast<const u32x4_t*>(a.tm + clamp_hi(16 * f + (lane & 15), a.M - 1) * a.r + jj);
  }
}

// One rank pass of the second product on the row-scaled fp16 T (D[row][m] = sum_j P[row][j] T[m][j]);
// the caller unscales the sum of all passes.
template <int FM, int kSteps, bool QA>
SLIM_DEV void finish_adapter_mfma(const LayerArgs& a, int64_t jbase, int lane, const u32x4_t* aq,
                                  const u32x4_t (*bq)[FM], const uint32_t* ps, f4_t* adacc) {
  const int g = lane >> 4;
#pragma unroll
  for (int t = 0; t < kSteps; ++t) {
    const bool jok = jbase + 32 * t + 8 * g < a.r;
    const h8_t pv = QA ? dequant_word(aq[t][0], splat_h2(ps[t / 4])) : __builtin_bit_cast(h8_t, aq[t]);
    const h8_t av = jok ? pv : zero_h8();
#pragma unroll
    for (int f = 0; f < FM; ++f) {
      const h8_t bv = (16 * f + (lane & 15) < a.M) ? __builtin_bit_cast(h8_t, bq[t][f]) : zero_h8();
      adacc[f] = mfma16(av, bv, adacc[f]);
    }
  }
}

template <int FM, int NW, bool QA>
__global__ void __launch_bounds__(64 * NW) k_finish(LayerArgs a) {
  constexpr int kSteps = (FM == 1 ? 16 : 8) / NW;   // 32-rank steps per pass of one wave
  static_assert(kSteps % 4 == 0, "whole groups of four steps (4-bit adapter scales)");
  // the wave that sums the split partials: the first, or with four waves the last (which has the
  // fewest rank passes when the rank is not a multiple of four passes)
  constexpr int kPartWave = NW == 4 ? 3 : 0;
  __shared__ f4_t hand[NW > 1 ? NW - 1 : 1][NW > 1 ? FM : 1][64];
  const int lane = threadIdx.x & 63, g = lane >> 4;
  const int h = NW > 1 ? __builtin_amdgcn_readfirstlane((int)threadIdx.x >> 6) : 0;
  const int64_t row0 = (int64_t)blockIdx.x * 16;
  const int64_t lrow = clamp_hi(row0 + (lane & 15), a.rows - 1);
  const int64_t rr = row0 + 4 * g;
  const int64_t rt = row0 / 64;
  const int w16 = (int)((row0 % 64) / 16);
  const int S = a.split;
  const rsrc_t pr = make_rsrc(a.part + (rt * S * 4 + w16) * (int64_t)(FM * 256), ((int64_t)(S - 1) * 4 + 1) * FM * 256 * 4);
  const int64_t jfirst = (int64_t)h * 32 * kSteps;
  u32x4_t aq[kSteps], bq[kSteps][FM];
  uint32_t ps[kSteps / 4];
  float trinv[FM];
  if (a.r > 0) {
    finish_adapter_loads<FM, kSteps, QA>(a, jfirst, lrow, lane, aq, bq, ps);
#pragma unroll
    for (int f = 0; f < FM; ++f) trinv[f] = a.trinv[clamp_hi(16 * f + (lane & 15), a.M - 1)];
  }
  f4_t acc[FM];
#pragma unroll
  for (int f = 0; f < FM; ++f) acc[f] = f4_t{0.f, 0.f, 0.f, 0.f};
  for (int s0 = 0; s0 < (h == kPartWave ? S : 0); s0 += 8) {   // the partials
    f4_t pv[8][FM];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int ss = s0 + j < S ? s0 + j : S - 1;
#pragma unroll
      for (int f = 0; f < FM; ++f) {
        // a lane whose column is past M points past the resource: no memory access, zero returned
        const uint32_t off = 16 * f + (lane & 15) < a.M ? (uint32_t)(((ss * 4 * FM + f) * 256 + 4 * lane) * 4) : 0x80000000u;
        pv[j][f] = __builtin_bit_cast(f4_t, __builtin_amdgcn_raw_buffer_load_b128(pr, off, 0, 0));
      }
    }
#pragma unroll
    for (int j = 0; j < 8; ++j)
      if (s0 + j < S)
#pragma unroll
        for (int f = 0; f < FM; ++f) acc[f] = acc[f] + pv[j][f];
  }
  if (a.r > 0) {
    // wave h takes rank passes h, h + NW, ... of 32 kSteps ranks; D[row][m] sits in lane
    // m + 16 (row / 4), so each lane unscales with its own row's factor
    f4_t adacc[FM];
#pragma unroll
    for (int f = 0; f < FM; ++f) adacc[f] = f4_t{0.f, 0.f, 0.f, 0.f};
    finish_adapter_mfma<FM, kSteps, QA>(a, jfirst, lane, aq, bq, ps, adacc);
    for (int64_t jbase = jfirst + NW * 32 * kSteps; jbase < a.r; jbase += NW * 32 * kSteps) {
      finish_adapter_loads<FM, kSteps, QA>(a, jbase, lrow, lane, aq, bq, ps);
      finish_adapter_mfma<FM, kSteps, QA>(a, jbase, lane, aq, bq, ps, adacc);
    }
#pragma unroll
    for (int f = 0; f < FM; ++f) acc[f] = acc[f] + adacc[f] * trinv[f];
  }
  if (NW > 1) {
    // waves 1 .. NW - 1 hand their sums to wave 0, which adds them in wave order (a fixed order)
    // and stores
    if (h > 0)
#pragma unroll
      for (int f = 0; f < FM; ++f) hand[h - 1][f][lane] = acc[f];
    __syncthreads();
    if (h != 0) return;
#pragma unroll
    for (int w = 0; w < NW - 1; ++w)
#pragma unroll
      for (int f = 0; f < FM; ++f) acc[f] = acc[f] + hand[w][f][lane];
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
// Block = 512 / WR waves over a 512 x TC tile; wave w owns rows [row0 + WR w, +WR) as WR / 32
// fragments of 32 and all columns [m0, m0 + TC) as TC / 32 fragments of 32 (TC = 96 or 128): a
// WR x TC accumulator (in the accumulation registers) on 32x32x32 sparse MFMA. Each dequantised
// weight fragment feeds TC / 32 MFMAs and no weight row is dequantised by two waves; the wider
// tile spends less dequantisation per MFMA, the narrower one gives more tiles to even out the
// last round of blocks (the plan picks per shape). WR = 64 (the launched form) runs two waves per
// SIMD (8 waves, 64 x TC accumulators each), so that one wave's dequantisation, LDS reads and
// waits overlap the other's MFMAs, at twice the B-fragment reads from LDS; WR = 128 runs one (4
// waves, 128 x TC accumulators).
// Per 128-wide reduction chunk, the tile's packed words (codes, index words and scales of its
// 512 rows, in four 128-row groups) and the fp16 activation tile [TC x 128] go straight from
// memory to LDS (direct loads), so no register holds data still in flight: the words into a ring of three stages, two
// chunks ahead; the activations into a ring of three stages, two chunks ahead, at TC = 96, or of
// two stages, one chunk ahead, at TC = 128 (three would not fit in LDS next to the words). A
// chunk's words are read from LDS, and its first step dequantised, during the last step of the
// chunk before. Activation rows in LDS are 256 B with the 16-byte column index XOR-swizzled by
// the row, so B-fragment reads (32 rows at one column) hit distinct banks. The backward also
// brings each 128-row group's scale row into LDS with the activations.
// Each wave loads the words of its own rows; the scales (and in the backward the scale row) of a
// 128-row group are loaded by every wave of the group, so that all waves issue the same loads
// (two waves then write the same bytes).
constexpr int kTR = 512;
template <int TC, int WR> struct TileShape {
  static constexpr int kWaves = kTR / WR;              // waves per block
  static constexpr int kThreads = 64 * kWaves;
  static constexpr int kFn = WR / 32;                  // row fragments per wave
  static constexpr int kFm = TC / 32;                  // column fragments per wave
  static constexpr int kActRows = TC / kWaves;         // activation rows each wave brings in
  static constexpr int kActLoads = kActRows / 4;       // ... four rows per direct load
  static constexpr int kStagesX = TC == 128 ? 2 : 3;   // activation stages
  static constexpr int kAhead = kStagesX - 1;          // chunks of activations in flight ahead
  static_assert(kActRows % 4 == 0, "whole direct loads of four rows");
};
// Direct loads per thread per chunk: activation loads (kActLoads, and in the backward one
// scale-row load) and packed words (WR / 32 code loads, WR / 64 index word loads, and in the
// forward 1 scale load).
// kAhead 2: chunk c issues chunk c + 2's words in its first step and chunk c + 2's activations in
// its second; kAhead 1: chunk c + 1's activations in its first step and chunk c + 2's words in its
// second. The one barrier of chunk c opens its last step, after which the wave reads chunk c + 1's
// words and first B fragments: there chunk c + 1 must have landed, so only the loads chunk c
// issued for chunk c + 2 may still be outstanding (kTop). The prologue issues the loads of chunks
// 0 and 1 in the same order and waits with the same count before a barrier of its own.
template <bool BWD, int TC, int WR> struct TileCounts {
  static constexpr bool kActFirst = TileShape<TC, WR>::kAhead == 1;
  static constexpr int kWords = WR / 32 + WR / 64 + (BWD ? 0 : 1);
  static constexpr int kAct = TileShape<TC, WR>::kActLoads + (BWD ? 1 : 0);
  static constexpr int kTop = kActFirst ? kWords : kAct + kWords;
};

static_assert(vmcnt_wait(40) == 0x8F78u && vmcnt_wait(5) == 0x0F75u && TileCounts<true, 96, 64>::kTop < 64, "s_waitcnt encoding");
static_assert(vmcnt_lgkm0_wait(20) == 0x4074u, "s_waitcnt encoding");


// One chunk's packed words of the tile's four 128-row groups, as the direct loads lay them down
// (lane L of a load at 16 L, or 4 L for 2-byte loads): codes [group][fragment][lane] (16 B: the
// lane's four code words), index words [group][row slot] (16 B: the row's four words; row slot =
// 32 fragment + row in fragment), scales [group][row slot] (fp16 in the low half of a dword). Reads index these
// arrays directly (no pointer casts, and no 8-byte reads the compiler would pair into one
// instruction that has lost track of its address), so that the compiler can tell the stages
// apart and does not wait for every direct load in flight.
template <bool BWD>
struct TileWordsLds {
  u32x4_t cw[4][4][64];
  u32x4_t mw[4][128];
  uint16_t sw[BWD ? 1 : 4][BWD ? 2 : 128];
};
// one chunk's packed words of one lane (FN row fragments), read from LDS
template <int FN>
struct TileWords {
  u32x4_t cw[FN];
  u32x2_t mw[FN];
  uint32_t sw[FN];
};

template <bool BWD, int TC, int WR>
SLIM_DEV void tile_body(const LayerArgs& a) {
  using Sh = TileShape<TC, WR>;
  using Ct = TileCounts<BWD, TC, WR>;
  constexpr int kTC = TC, kFn = Sh::kFn, kFm = Sh::kFm, kStagesX = Sh::kStagesX;
  // one array per stage (the stages of chunk c are c % 3 for the words and c % kStagesX for the
  // activations, constants in the loop unrolled by six), so that reads of one stage are not
  // ordered behind loads still landing in another
  __shared__ __attribute__((aligned(16))) _Float16 xs0[kTC][128], xs1[kTC][128], xs2[kStagesX == 3 ? kTC : 1][128];
  __shared__ __attribute__((aligned(16))) TileWordsLds<BWD> ws0, ws1, ws2;
  __shared__ __attribute__((aligned(16))) _Float16 ss0[BWD ? 4 : 1][512], ss1[BWD ? 4 : 1][512],
      ss2[BWD && kStagesX == 3 ? 4 : 1][512];
  auto xs_at = [&](int stg) -> _Float16(*)[128] { return stg == 0 ? xs0 : (stg == 1 ? xs1 : xs2); };
  auto ws_at = [&](int stg) -> TileWordsLds<BWD>& { return stg == 0 ? ws0 : (stg == 1 ? ws1 : ws2); };
  auto ss_at = [&](int stg) -> _Float16(*)[512] { return stg == 0 ? ss0 : (stg == 1 ? ss1 : ss2); };
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int ha = lane >> 5;
  // the wave's 128-row group and its first fragment there
  const int grp = WR == 128 ? wave : wave >> 1, fbase = WR == 128 ? 0 : 2 * (wave & 1);
  // XCD-aware tile order: block b runs on XCD b % 8 (workgroups are dealt round robin), and XCD x
  // takes positions [x Q, (x + 1) Q) of a tile order that walks bands of kb row tiles column
  // by column. The blocks an XCD runs together then cover a few row tiles x a few column tiles,
  // so they share packed weights and activations in that XCD's L2.
  const int64_t R = a.row_tiles, C = a.col_tiles, T = R * C;
  const int64_t Q = (T + 7) / 8;
  const int64_t pos = (int64_t)(blockIdx.x % 8) * Q + blockIdx.x / 8;
  if (pos >= T) return;
  // bands of 8 row tiles when there are at most 32 row tiles, else 4 (prefill's 22 row tiles:
  // tile kernel 136.6 -> 134.9 us; the 70B layers' 56 were 0.5% slower with 8, all shapes slower
  // with 2)
  const int64_t kb = R <= 32 ? 8 : 4;
  const int64_t band = pos / (kb * C), q = pos - band * kb * C;
  const int64_t rb = R - band * kb < kb ? R - band * kb : kb;   // rows in this band
  const int64_t rt = band * kb + q % rb, ct = q / rb;
  const int64_t row0 = rt * kTR, m0 = ct * kTC;
  const int64_t wrow0 = row0 + WR * wave;
  const int64_t nch = a.red / 128;

  // Addresses. Per-lane offsets are derived inside each chunk from a few base registers (made
  // opaque per chunk) instead of being kept live across the loop. Rows past the matrix (or past
  // M) get offsets at or beyond their resource's extent and read as zero; their results are not
  // stored. The uniform chunk offset only ever moves a valid row within that row.
  // packed words: resources from the first 16-row block of the wave's 128-row group (clamped
  // into the matrix; rows is a multiple of 16). Relative to it, row d of chunk c sits in slot
  // ((d / 16) nch + c) 16 + d % 16; the chunk adds 16 slots, and 32 rows (two blocks) add
  // 32 nch slots, fstep bytes of codes (32 B per slot) and, per 64 rows, of index words (16 B).
  const int64_t grow0 = row0 + 128 * grp;
  const int64_t wblk = (grow0 < a.rows ? grow0 : a.rows - 16) / 16;
  const int64_t nblk = a.rows / 16 - wblk;
  const rsrc_t rc = make_rsrc(a.codes + wblk * nch * 128, nblk * nch * 512);
  const rsrc_t rm = make_rsrc(a.meta + wblk * nch * 64, nblk * nch * 256);
  const rsrc_t rs = make_rsrc(a.scales + wblk * nch * 16, nblk * nch * 32);
  const uint32_t d0 = (uint32_t)(grow0 - 16 * wblk) + 32u * (uint32_t)fbase, snch = 16u * (uint32_t)nch;
  auto rel_slot = [&](uint32_t d) { return (d >> 4) * snch + (d & 15u); };
  const uint32_t fstep = 1024u * (uint32_t)nch;
  const uint32_t co0 = rel_slot(d0 + (uint32_t)(lane & 31)) * 32u + 16u * ha;   // codes: the wave's fragment 0
  const uint32_t mo0 = rel_slot(d0 + (uint32_t)lane) * 16u;                     // index words: the wave's rows 0..63
  const uint32_t so0 = rel_slot(d0 - 32u * (uint32_t)fbase + 2u * (uint32_t)lane) * 2u;   // scales: group rows 2 L, 2 L + 1

  // activation chunk c -> stage c % kStagesX: wave w writes rows R w .. R w + R - 1 (R = kActRows),
  // four per load (lane L: row + L / 16, LDS column slot L % 16 holding column
  // (L % 16) ^ (row % 16)). Load i covers rows R w + 4 i + L / 16; with S = 16 ((L % 16) ^ (L / 16))
  // its byte offset is (R w + L / 16) 2 red + 8 i red + (S ^ 16 ((R w + 4 i) % 16)), as 2 red is a
  // multiple of 256 and S < 256.
  const int lrow = lane >> 4, lslot = lane & 15;
  const int64_t brows = a.M - m0 < kTC ? a.M - m0 : kTC;
  const rsrc_t rx = make_rsrc(a.act16 + m0 * a.red, brows * a.red * 2);    // the block's activation rows
  const uint32_t xo0 = (uint32_t)(Sh::kActRows * wave + lrow) * (uint32_t)a.red * 2u + 16u * (uint32_t)(lslot ^ lrow);
  const uint32_t xstep = 8u * (uint32_t)a.red;
  const rsrc_t rg = make_rsrc(a.scales + (16 * wblk / 128) * a.red, a.red * 2);   // backward: the group's scale row

  auto dma_words = [&](int64_t c, int stg, uint32_t co, uint32_t mo, uint32_t so) {
    const int cc = (int)clamp_hi(c, nch - 1);
    TileWordsLds<BWD>& W = ws_at(stg);
#pragma unroll
    for (int fn = 0; fn < kFn; ++fn)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rc, (lds_ptr_t)&W.cw[grp][fbase + fn][0], 16, co + fn * fstep, 512 * cc, 0, 0);
#pragma unroll
    for (int j = 0; j < kFn / 2; ++j)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rm, (lds_ptr_t)&W.mw[grp][32 * fbase + 64 * j], 16, mo + j * fstep, 256 * cc, 0, 0);
    if (!BWD) __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (lds_ptr_t)&W.sw[grp][0], 4, so, 32 * cc, 0, 0);
  };
  auto dma_act = [&](int64_t c, int stg, uint32_t xo) {
    const int cc = (int)clamp_hi(c, nch - 1);
#pragma unroll
    for (int i = 0; i < Sh::kActLoads; ++i)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rx, (lds_ptr_t)&xs_at(stg)[Sh::kActRows * wave + 4 * i][0], 16,
                                               (xo ^ (16u * ((uint32_t)(Sh::kActRows * wave + 4 * i) & 15u))) + (uint32_t)i * xstep,
                                               256 * cc, 0, 0);
    if (BWD) {
      // the group's scale row s16[n, g] for this chunk (g = the wave's 128-row group), four copies
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rg, (lds_ptr_t)&ss_at(stg)[grp][0], 16, 16u * lslot, 256 * cc, 0, 0);
    }
  };
  auto read_words = [&](int stg, TileWords<kFn>& t) {
    const TileWordsLds<BWD>& W = ws_at(stg);
#pragma unroll
    for (int fn = 0; fn < kFn; ++fn) {
      t.cw[fn] = W.cw[grp][fbase + fn][lane];
      const u32x4_t m4 = W.mw[grp][32 * (fbase + fn) + (lane & 31)];
      t.mw[fn] = ha ? u32x2_t{m4[2], m4[3]} : u32x2_t{m4[0], m4[1]};
      t.sw[fn] = BWD ? 0u : W.sw[grp][32 * (fbase + fn) + (lane & 31)];
    }
  };
  const NibbleConsts nk = nibble_consts_reg();
  auto dequant = [&](const TileWords<kFn>& t, int st, h8_t* av) {
#pragma unroll
    for (int fn = 0; fn < kFn; ++fn)
      av[fn] = BWD ? dequant_word_int(t.cw[fn][st], nk) : dequant_word(t.cw[fn][st], splat_h2(t.sw[fn]), nk);
  };
  // B-fragment reads: fragment fm of step st reads row 32 fm + L % 32 at 16-byte column slots
  // (2 st + L / 32) ^ (L % 16) (low half) and that + 8 (high half); with
  // bo = 256 (L % 32) + 16 ((L % 16) ^ (L / 32)) these are at bytes 8192 fm + (bo ^ 32 st) and
  // 8192 fm + (bo ^ (32 st + 128)) of the stage.
  const uint32_t bo0 = 256u * (uint32_t)(lane & 31) + 16u * (uint32_t)((lane & 15) ^ ha);

  f16_t acc[kFn][kFm];
#pragma unroll
  for (int fn = 0; fn < kFn; ++fn)
#pragma unroll
    for (int fm = 0; fm < kFm; ++fm)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[fn][fm][v] = 0.f;

  // words of chunk c in set c % 3 (read during chunk c - 1); A operands double-buffered by step
  TileWords<kFn> tw[3];
  h8_t aq[2][kFn];
  // B fragment fm of step st from activation stage xstg
  auto read_b = [&](int xstg, int st, int fm, uint32_t bo, h16_t& bv) {
    const char* xsb = reinterpret_cast<const char*>(&xs_at(xstg)[0][0]);
    h8_t lo = *reinterpret_cast<const h8_t*>(xsb + (bo ^ (32u * st)) + 8192 * fm);
    h8_t hi = *reinterpret_cast<const h8_t*>(xsb + (bo ^ (32u * st + 128u)) + 8192 * fm);
    if (BWD) {
      const int c16 = 2 * st + ha;
      lo = mul_h8(lo, *reinterpret_cast<const h8_t*>(&ss_at(xstg)[grp][8 * c16]));
      hi = mul_h8(hi, *reinterpret_cast<const h8_t*>(&ss_at(xstg)[grp][8 * c16 + 64]));
    }
    bv = cat16(lo, hi);
  };
  // one B buffer, refilled fragment by fragment (below)
  h16_t bq[kFm];

  dma_words(0, 0, co0, mo0, so0);
  dma_act(0, 0, xo0);
  dma_words(1, 1, co0, mo0, so0);
  if (!Ct::kActFirst) dma_act(1, 1, xo0);
  // chunk 0 has landed once only chunk 1's loads are outstanding; the other waves brought in
  // part of it. The barrier is issued as a bare instruction: the builtin would also make this
  // wave wait for every direct-to-LDS load in flight, including the ones for the next chunk.
  __builtin_amdgcn_s_waitcnt(vmcnt_lgkm0_wait(Ct::kTop));
  asm volatile("s_barrier" ::: "memory");
  read_words(0, tw[0]);
  dequant(tw[0], 0, aq[0]);
#pragma unroll
  for (int fm = 0; fm < kFm; ++fm) read_b(0, 0, fm, bo0, bq[fm]);

  auto chunk = [&](int64_t c, auto zc, auto xc) {
    constexpr int z = decltype(zc)::value;    // c % 3: word stage and register set
    constexpr int stg = decltype(xc)::value;  // c % kStagesX: activation stage
    // Nothing of the previous chunk is scheduled past this point.
    __builtin_amdgcn_sched_barrier(0);
    // this chunk's copies of the base offsets (opaque, so nothing derived from them is hoisted)
    uint32_t xo = xo0, co = co0, mo = mo0, so = so0, bo = bo0;
    asm volatile("" : "+v"(xo), "+v"(co), "+v"(mo), "+v"(so), "+v"(bo));
    const TileWords<kFn>& cur = tw[z];
    TileWords<kFn>& nxt = tw[(z + 1) % 3];
    // Software pipeline over the four steps. The MFMAs of a step run column fragment by column
    // fragment; once the kFn MFMAs of fragment fm have issued, its registers are refilled with
    // the next step's fragment fm, while the next step's dequantised weights go to the other A
    // buffer. The chunk's one barrier opens its last step: after it the next chunk's words are
    // read and its first step dequantised, and its first B fragments are read during this step's
    // MFMAs (step 0 of a chunk then starts without waiting on LDS).
#pragma unroll
    for (int st = 0; st < 4; ++st) {
      // direct loads into the stages read in chunk c - 1 (chunk c + kAhead's activations, chunk
      // c + 2's words) during steps 0 and 1, one load after each MFMA (issued in a burst at the
      // barrier, the waves' loads would fill the address unit's queue and stall issue)
      if (st == (Ct::kActFirst ? 0 : 1)) dma_act(c + Sh::kAhead, (stg + Sh::kAhead) % kStagesX, xo);
      if (st == (Ct::kActFirst ? 1 : 0)) dma_words(c + 2, (z + 2) % 3, co, mo, so);
      if (st < 3) {
        dequant(cur, st + 1, aq[(st + 1) & 1]);
      } else {
        // chunk c + 1 has landed once only chunk c + 2's loads are outstanding, and this wave's
        // reads of chunk c's activation stage (the last ones, for this step, were issued in the
        // step before) have returned (lgkmcnt 0): after the barrier no wave reads that stage, and
        // the next chunk's direct loads may refill it.
        __builtin_amdgcn_sched_barrier(0);
        __builtin_amdgcn_s_waitcnt(vmcnt_lgkm0_wait(Ct::kTop));
        asm volatile("s_barrier" ::: "memory");
        __builtin_amdgcn_sched_barrier(0);
        read_words((z + 1) % 3, nxt);
        dequant(nxt, 0, aq[0]);
      }
#pragma unroll
      for (int fm = 0; fm < kFm; ++fm) {
#pragma unroll
        for (int fn = 0; fn < kFn; ++fn)
          acc[fn][fm] = smfmac32(aq[st & 1][fn], bq[fm], acc[fn][fm], (int)cur.mw[fn][st >> 1], st & 1);
        if (st < 3) read_b(stg, st + 1, fm, bo, bq[fm]);
        else read_b((stg + 1) % kStagesX, 0, fm, bo, bq[fm]);
      }
      // interleave: each MFMA followed by a share of the VALU work and, in steps 0 and 1, by one
      // direct load; the LDS reads of fragment fm follow its MFMAs (in the last step the next
      // chunk's words are read first)
      const int nvm = st == 0 ? (Ct::kActFirst ? Ct::kAct : Ct::kWords) : st == 1 ? (Ct::kActFirst ? Ct::kWords : Ct::kAct) : 0;
#pragma unroll
      for (int i = 0; i < kFn * kFm; ++i) {
        if (st == 3 && i < 3 * kFn / 2) __builtin_amdgcn_sched_group_barrier(0x0100, 2, 0);   // DS read
        __builtin_amdgcn_sched_group_barrier(0x0008, 1, 0);                          // MFMA
        if (i < nvm) __builtin_amdgcn_sched_group_barrier(0x0020, 1, 0);             // VMEM read
        __builtin_amdgcn_sched_group_barrier(0x0002, 4, 0);                          // VALU
        if (i % kFn == kFn - 1) __builtin_amdgcn_sched_group_barrier(0x0100, 2, 0);   // DS read
      }
    }
  };
  // full groups of six without guards (a load under a branch costs a full wait at the join),
  // then at most five chunks
  using I0 = std::integral_constant<int, 0>;
  using I1 = std::integral_constant<int, 1>;
  using I2 = std::integral_constant<int, 2>;
  using X0 = std::integral_constant<int, 0>;
  using X1 = std::integral_constant<int, 1>;
  using X2 = std::integral_constant<int, kStagesX == 3 ? 2 : 0>;
  using X3 = std::integral_constant<int, kStagesX == 3 ? 0 : 1>;
  using X4 = std::integral_constant<int, kStagesX == 3 ? 1 : 0>;
  using X5 = std::integral_constant<int, kStagesX == 3 ? 2 : 1>;
  int64_t c0 = 0;
  for (; c0 + 6 <= nch; c0 += 6) {
    chunk(c0, I0{}, X0{});
    chunk(c0 + 1, I1{}, X1{});
    chunk(c0 + 2, I2{}, X2{});
    chunk(c0 + 3, I0{}, X3{});
    chunk(c0 + 4, I1{}, X4{});
    chunk(c0 + 5, I2{}, X5{});
  }
  if (c0 < nch) chunk(c0, I0{}, X0{});
  if (c0 + 1 < nch) chunk(c0 + 1, I1{}, X1{});
  if (c0 + 2 < nch) chunk(c0 + 2, I2{}, X2{});
  if (c0 + 3 < nch) chunk(c0 + 3, I0{}, X3{});
  if (c0 + 4 < nch) chunk(c0 + 4, I1{}, X4{});
  // the ring's last loads (repeats of the final chunk) must land before the block's LDS is released
  __builtin_amdgcn_s_waitcnt(0);

  // adapter second product: out^T[row, m] += sum_j P[row, j] tm[m, j], on 32x32x16 fp16 MFMA.
  // Both operands are in 32 x 16 tiles (P re-laid and tm finished by k_adapter_finish, or tm
  // written so by the adapter GEMM): step t (ranks [16 t, 16 t + 16), r a multiple of 16) of one
  // 32-row fragment is 1 KB of contiguous memory, lane (L % 32, L / 32) reading row L % 32, ranks
  // 8 (L / 32) ... + 7. Each wave loads its own rows of P straight into registers, three steps
  // ahead into a ring of four register sets. tm, which every wave needs for all TC columns, comes
  // through LDS: groups of eight steps (kFm x 8 tiles, the size of one activation stage) go to the
  // activation stages in turn by direct loads one group ahead, spread over the waves, and each
  // wave reads its fragments there. Loads past the last step repeat it and are not used;
  // fragments past the tiled extent read zero and their results are not stored.
  if (a.r > 0) {
    const int64_t nj = a.r / 16, ngrp = (nj + 7) / 8;
    const rsrc_t rp = make_rsrc(a.ad_pb, (a.rows + 31) / 32 * 32 * a.r * 2), rt = make_rsrc(a.tm, (a.M + 31) / 32 * 32 * a.r * 2);
    const uint32_t lo16 = 32u * (uint32_t)(lane & 31) + 16u * ha;   // the lane's bytes within a 1 KB tile
    uint32_t po[kFn];
#pragma unroll
    for (int fn = 0; fn < kFn; ++fn) po[fn] = (uint32_t)((wrow0 + 32 * fn) / 32 * nj) * 1024u + lo16;
    // tm tiles of a group per wave: tile q = 8 fm + (step % 8) goes to byte 1024 q of the stage
    constexpr int kTT = kFm * 8 / Sh::kWaves;
    static_assert(kTT * Sh::kWaves == kFm * 8, "tm tiles of a group spread evenly over the waves");
    auto dma_t = [&](int64_t g, int stg) {
      char* dst = reinterpret_cast<char*>(&xs_at(stg)[0][0]);
#pragma unroll
      for (int i = 0; i < kTT; ++i) {
        // the tile row's offset per lane (rows past M lie beyond the resource's extent and read
        // zero), the step's within that row as the uniform offset. Lane L fetches the 16 bytes
        // that lane L of a fragment read needs (lo16) and lays them at 16 L, so the read of a
        // fragment is 1 KB in lane order (a read at lo16 would put lanes L and L + 8 of one
        // 16-lane pass in the same bank).
        const int q = wave + Sh::kWaves * i, fm = q >> 3;
        const int64_t t = clamp_hi(8 * g + (q & 7), nj - 1);
        const uint32_t vo = (uint32_t)((m0 + 32 * fm) / 32 * nj) * 1024u + lo16;
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rt, (lds_ptr_t)(dst + 1024 * q), 16, vo, (int)(t * 1024), 0, 0);
      }
    };
    struct AdRegs { u32x4_t pa[kFn]; };
    AdRegs ar[4];
    auto ad_load = [&](int64_t t, AdRegs& R) {
      const int so = (int)(clamp_hi(t, nj - 1) * 1024);
#pragma unroll
      for (int fn = 0; fn < kFn; ++fn) R.pa[fn] = __builtin_bit_cast(u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(rp, po[fn], so, 0));
    };
    // every wave is done with the ring (its reads returned, its direct loads landed) before the
    // first group overwrites a stage
    asm volatile("s_barrier" ::: "memory");
    dma_t(0, 0);
    ad_load(0, ar[0]);
    ad_load(1, ar[1]);
    ad_load(2, ar[2]);
    // group 0 has landed once only the three steps of P loads issued after it are outstanding
    __builtin_amdgcn_s_waitcnt(vmcnt_wait(3 * kFn));
    asm volatile("s_barrier" ::: "memory");
    // step t = 8 g + tt of group g (stage xstg); group g + 1 was issued at the group's start, after
    // step g 8 + 2's P loads and before step 8 g + 3's
    auto ad_step = [&](int64_t g, auto ttc, int xstg) {
      constexpr int tt = decltype(ttc)::value;
      const int64_t t = 8 * g + tt;
      ad_load(t + 3, ar[(tt + 3) % 4]);
      __builtin_amdgcn_s_waitcnt(vmcnt_wait(3 * kFn + (tt < 3 ? kTT : 0)));
      AdRegs& R = ar[tt % 4];
#pragma unroll
      for (int fn = 0; fn < kFn; ++fn) asm volatile("" : "+v"(R.pa[fn]));
      const char* src = reinterpret_cast<const char*>(&xs_at(xstg)[0][0]);
      h8_t tb[kFm];
#pragma unroll
      for (int fm = 0; fm < kFm; ++fm) tb[fm] = *reinterpret_cast<const h8_t*>(src + 1024 * (8 * fm + tt) + 16 * lane);
      if (t < nj) {
#pragma unroll
        for (int fn = 0; fn < kFn; ++fn)
#pragma unroll
          for (int fm = 0; fm < kFm; ++fm)
            acc[fn][fm] = mfma32(__builtin_bit_cast(h8_t, R.pa[fn]), tb[fm], acc[fn][fm]);
      }
    };
    auto group = [&](int64_t g, int xstg) {
      // the next group into the next stage (read two or three groups ago, before the last
      // barrier); issued also after the last group, whose repeats land in a stage no wave reads
      dma_t(g + 1, (xstg + 1) % kStagesX);
      ad_step(g, std::integral_constant<int, 0>{}, xstg);
      ad_step(g, std::integral_constant<int, 1>{}, xstg);
      ad_step(g, std::integral_constant<int, 2>{}, xstg);
      ad_step(g, std::integral_constant<int, 3>{}, xstg);
      ad_step(g, std::integral_constant<int, 4>{}, xstg);
      ad_step(g, std::integral_constant<int, 5>{}, xstg);
      ad_step(g, std::integral_constant<int, 6>{}, xstg);
      ad_step(g, std::integral_constant<int, 7>{}, xstg);
      // this wave's reads of the stage have returned and the next group has landed (waited for
      // at step 3): after the barrier the stage may be refilled and the next group read
      __builtin_amdgcn_s_waitcnt(vmcnt_lgkm0_wait(3 * kFn));
      asm volatile("s_barrier" ::: "memory");
    };
    int64_t g = 0;
    for (; g + kStagesX <= ngrp; g += kStagesX) {
      group(g, 0);
      group(g + 1, 1);
      if constexpr (kStagesX == 3) group(g + 2, 2);
    }
    for (int xstg = 0; g < ngrp; ++g, ++xstg) group(g, xstg);
    __builtin_amdgcn_s_waitcnt(0);
  }

  // D[i][j] of a 32x32 fragment: lane j + 32 * ((i / 4) % 2), element 4 * (i / 8) + i % 4; column
  // m's activation row was scaled by 2^e (k_rowprep), so its results are multiplied by 2^-e
#pragma unroll
  for (int fm = 0; fm < kFm; ++fm) {
    const int64_t m = m0 + 32 * fm + (lane & 31);
    if (m >= a.M) continue;
    const float inv = a.rowinv ? a.rowinv[m] : 1.0f;
#pragma unroll
    for (int fn = 0; fn < kFn; ++fn)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int64_t rr = wrow0 + 32 * fn + 8 * q + 4 * ha;
        if (rr < a.rows) {
          const f4_t o = {acc[fn][fm][4 * q], acc[fn][fm][4 * q + 1], acc[fn][fm][4 * q + 2], acc[fn][fm][4 * q + 3]};
          *reinterpret_cast<f4_t*>(a.out + m * a.rows + rr) = o * inv;
        }
      }
  }
}

template <bool BWD, int TC, int WR>
__global__ void __launch_bounds__(64 * (kTR / WR)) k_tile(LayerArgs a) {
  tile_body<BWD, TC, WR>(a);
}

// Large-M activation preparation, one block per row m of act [M, red] (bf16 or fp16): the row's
// largest magnitude gives its scaling exponent e (act_exponent); the row times 2^e, rounded to
// fp16, goes to act16 (the copy the adapter GEMM and the tile kernel stream) and 2^-e to
// rowinv[m]. Rows of up to 256 x NR vectors of 8 (NR > 0) stay in registers between the two
// passes; longer rows (NR == 0) are read twice (the second read mostly from L2).
constexpr int kRowRegs = 16;
// With 4-bit adapters the same launch also expands them into the fp16 layouts the adapter GEMM and
// the tile epilogue read (blocks past the M row blocks, one thread per word of 8 codes):
// Q = L^T [r, red] row-major, P = R^T [rows, r] in 32 x 16 tiles.
struct AdapterExpand {
  const uint32_t* q4;
  const uint16_t* q4s;
  uint16_t* q16;
  const uint32_t* p4;
  const uint16_t* p4s;
  uint16_t* p16;
  int64_t r, red, rows, M;
};

SLIM_DEV void expand_adapter_block(const AdapterExpand& d, int64_t b) {
  const int64_t i = b * 256 + threadIdx.x;     // word index: Q words first, then P words
  const int64_t nq = d.r * d.red / 8, np = d.rows * d.r / 8;
  if (i < nq) {
    const int64_t row = i / (d.red / 8), col = (i % (d.red / 8)) * 8;
    const h8_t v = dequant_word(d.q4[i], splat_h2(d.q4s[row * ((d.red + 127) / 128) + col / 128]));
    *reinterpret_cast<h8_t*>(d.q16 + row * d.red + col) = v;
  } else if (i < nq + np) {
    const int64_t w = i - nq, row = w / (d.r / 8), col = (w % (d.r / 8)) * 8;
    const h8_t v = dequant_word(d.p4[w], splat_h2(d.p4s[row * ((d.r + 127) / 128) + col / 128]));
    *reinterpret_cast<h8_t*>(d.p16 + ((row >> 5) * (d.r >> 4) + (col >> 4)) * 512 + (row & 31) * 16 + (col & 15)) = v;
  }
}

template <bool BF16, int NR>
__global__ void __launch_bounds__(256) k_rowprep(const u32x4_t* __restrict__ act, int64_t nv, u32x4_t* __restrict__ act16,
                                                 float* __restrict__ rowinv, AdapterExpand ex) {
  if ((int64_t)blockIdx.x >= ex.M) {
    expand_adapter_block(ex, (int64_t)blockIdx.x - ex.M);
    return;
  }
  constexpr int kR = NR > 0 ? NR : 1;
  __shared__ uint32_t wmax[4];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int64_t row = blockIdx.x;
  const u32x4_t* src = act + row * nv;
  u32x4_t* dst = act16 + row * nv;
  constexpr bool regs = NR > 0;
  u32x4_t v[kR];
  uint32_t mx = 0;
  if (regs) {
#pragma unroll
    for (int i = 0; i < kR; ++i) v[i] = src[clamp_hi(tid + 256 * i, nv - 1)];
#pragma unroll
    for (int i = 0; i < kR; ++i) {
      float f[8];
      act8_to_f(v[i], BF16, f);
      if (tid + 256 * i < nv) mx = max(mx, max_abs_bits8(f));
    }
  } else {
    for (int64_t i = tid; i < nv; i += 256) {
      float f[8];
      act8_to_f(src[i], BF16, f);
      mx = max(mx, max_abs_bits8(f));
    }
  }
  mx = wave_max_u32(mx);
  if (lane == 0) wmax[wave] = mx;
  __syncthreads();
  mx = max(max(wmax[0], wmax[1]), max(wmax[2], wmax[3]));
  const int e = act_exponent(mx);
  const float sc = exp2i(e);
  if (tid == 0) rowinv[row] = exp2i(-e);
  if (regs) {
#pragma unroll
    for (int i = 0; i < kR; ++i) {
      float f[8];
      act8_to_f(v[i], BF16, f);
      if (tid + 256 * i < nv) dst[tid + 256 * i] = __builtin_bit_cast(u32x4_t, scale8_to_h(f, sc));
    }
  } else {
    for (int64_t i = tid; i < nv; i += 256) {
      float f[8];
      act8_to_f(src[i], BF16, f);
      dst[i] = __builtin_bit_cast(u32x4_t, scale8_to_h(f, sc));
    }
  }
}

// Adapter tiles for the tile kernel's epilogue, one launch with two kinds of block:
//  * blocks [0, np): P [rows, r] row-major -> 32 x 16 tiles, element (row, j) at
//    ((row / 32) (r / 16) + j / 16) 512 + (row % 32) 16 + j % 16; one thread per 8 elements
//    (16 B); rows of a last partial 32-row tile are left unwritten (their results are never
//    stored);
//  * blocks [np, ...): when the adapter GEMM split its reduction, tm (fp16, tiled) = the sum of
//    its fp32 split partials in split order; one thread per 8 elements of a row m < M.
__global__ void __launch_bounds__(256) k_adapter_finish(const u32x4_t* __restrict__ P, int64_t rows, int64_t r,
                                                        u32x4_t* __restrict__ Pb, int64_t np,
                                                        const float* __restrict__ part, int split, int64_t M,
                                                        u32x4_t* __restrict__ tm) {
  const int64_t r8 = r / 8;
  if ((int64_t)blockIdx.x < np) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= rows * r8) return;
    const int64_t row = i / r8, k8 = i - row * r8;
    Pb[((row >> 5) * (r >> 4) + (k8 >> 1)) * 64 + (row & 31) * 2 + (k8 & 1)] = P[i];
    return;
  }
  const int64_t i = ((int64_t)blockIdx.x - np) * 256 + threadIdx.x;   // group of 8 in tiled order
  const int64_t total8 = (M + 31) / 32 * 32 * r8;
  if (i >= total8) return;
  // tiled group i: tile i / 64, row in tile (i % 64) / 2 -> m
  const int64_t m = (i / 64) / (r >> 4) * 32 + (i % 64) / 2;
  if (m >= M) return;
  float v[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  for (int s = 0; s < split; ++s) {
    const f4_t* src = reinterpret_cast<const f4_t*>(part + (int64_t)s * total8 * 8 + 8 * i);
    const f4_t a0 = src[0], a1 = src[1];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      v[e] += a0[e];
      v[4 + e] += a1[e];
    }
  }
  h8_t h;
#pragma unroll
  for (int e = 0; e < 8; ++e) h[e] = (_Float16)v[e];
  tm[i] = __builtin_bit_cast(u32x4_t, h);
}

// ------------------------------------------------------------------------------ launch
template <bool BWD, int FM, int G, int NU, bool QA>
void launch_decode(const LayerArgs& a, const SlimPlan& p, hipStream_t s) {
  SlimKernelTimer timer(BWD ? "decode_bwd" : "decode_fwd", s);
  dim3 grid((unsigned)(p.sp_blocks + (a.r > 0 ? p.ad_jblocks * p.ad_split : 0)));
  SLIM_LAUNCH(timer, (k_decode<BWD, FM, G, NU, QA>), grid, dim3(256), s, a);
}

template <bool BWD, int FM, int G, bool QA>
void launch_decode_units(const LayerArgs& a, const SlimPlan& p, hipStream_t s) {
  if (p.dec_units > 1) launch_decode<BWD, FM, G, BWD ? 2 : kDecodeMaxUnits, QA>(a, p, s);
  else launch_decode<BWD, FM, G, 1, QA>(a, p, s);
}

template <int FM, bool QA>
void launch_finish(const LayerArgs& a, bool bwd, hipStream_t s) {
  SlimKernelTimer timer(bwd ? "finish_bwd" : "finish_fwd", s);
  // several waves per 16 rows, splitting the rank, when the rank fills more than one wave's pass
  // and there are few rows (at most 1024 blocks): each wave issues a share of the adapter loads
  // (4096^2 layer at M 16: step 11.7 -> 11.3 us with two). Four waves (one of them summing the
  // split partials) for at most 4096 rows and at most 8 columns, where the adapter pass outweighs
  // the partials (4096^2 layer at M 1: 10.21 -> 10.02 us; at M 16 two waves were as fast). The
  // choice never depends on the adapter's format, so 4-bit and fp16 factors of the same values
  // are summed in the same order.
  // With many rows one wave per 16 rows already fills the CUs.
  const dim3 grid((unsigned)((a.rows + 15) / 16));
  if (FM == 1 && a.r > 16 * 8 && a.rows <= 4096 && a.M <= 8)
    SLIM_LAUNCH(timer, (k_finish<1, 4, QA>), grid, dim3(256), s, a);
  else if (a.r > 16 * (FM == 1 ? 16 : 8) && a.rows <= 16384) SLIM_LAUNCH(timer, (k_finish<FM, 2, QA>), grid, dim3(128), s, a);
  else SLIM_LAUNCH(timer, (k_finish<FM, 1, QA>), grid, dim3(64), s, a);
}

template <bool BWD, bool QA>
void launch_small_m(const LayerArgs& a, const SlimPlan& p, hipStream_t s) {
  if (p.dec_fm == 1) {
    if (p.dec_g == 1) launch_decode_units<BWD, 1, 1, QA>(a, p, s);
    else launch_decode_units<BWD, 1, 2, QA>(a, p, s);
  } else {
    launch_decode_units<BWD, 2, 1, QA>(a, p, s);
  }
}

template <bool BWD>
int launch_layer(const LayerArgs& a, const SlimPlan& p, const uint16_t* act, int act_bf16, char* ws, hipStream_t s) {
  if (p.decode) {
    // 4-bit adapters (forward only) are a template variant, so neither kernel branches around loads
    const bool qa = !BWD && a.q4 != nullptr;
    if (qa) launch_small_m<BWD, true>(a, p, s);
    else launch_small_m<BWD, false>(a, p, s);
    if (hipGetLastError() != hipSuccess) return SLIM_EDEVICE;
    if (a.finish) {
      if (qa) {
        if (p.dec_fm == 1) launch_finish<1, true>(a, BWD, s);
        else launch_finish<2, true>(a, BWD, s);
      } else {
        if (p.dec_fm == 1) launch_finish<1, false>(a, BWD, s);
        else launch_finish<2, false>(a, BWD, s);
      }
      if (hipGetLastError() != hipSuccess) return SLIM_EDEVICE;
    }
    return SLIM_OK;
  }
  if (a.rowinv) {
    // scale each activation row into the fp16 copy the adapter GEMM and the tile kernel stream
    SlimKernelTimer timer("rowprep", s);
    const int64_t nv = a.red / 8;
    AdapterExpand ex{a.q4, a.q4s, const_cast<uint16_t*>(a.ad_q), a.p4, a.p4s, const_cast<uint16_t*>(a.ad_pb),
                     a.r, a.red, a.rows, a.M};
    const int64_t nexp = a.q4 ? (a.r * a.red / 8 + a.rows * a.r / 8 + 255) / 256 : 0;
    const dim3 grid((unsigned)(a.M + nexp));
    u32x4_t* dst = reinterpret_cast<u32x4_t*>(const_cast<uint16_t*>(a.act16));
    const u32x4_t* src = reinterpret_cast<const u32x4_t*>(act);
    float* rinv = const_cast<float*>(a.rowinv);
    const int nr = nv <= 512 ? 2 : nv <= 1024 ? 4 : nv <= 2048 ? 8 : nv <= 256 * kRowRegs ? 16 : 0;
#define SLIM_ROWPREP(B, NR) SLIM_LAUNCH(timer, (k_rowprep<B, NR>), grid, dim3(256), s, src, nv, dst, rinv, ex)
    if (act_bf16) {
      if (nr == 2) SLIM_ROWPREP(true, 2);
      else if (nr == 4) SLIM_ROWPREP(true, 4);
      else if (nr == 8) SLIM_ROWPREP(true, 8);
      else if (nr == 16) SLIM_ROWPREP(true, 16);
      else SLIM_ROWPREP(true, 0);
    } else {
      if (nr == 2) SLIM_ROWPREP(false, 2);
      else if (nr == 4) SLIM_ROWPREP(false, 4);
      else if (nr == 8) SLIM_ROWPREP(false, 8);
      else if (nr == 16) SLIM_ROWPREP(false, 16);
      else SLIM_ROWPREP(false, 0);
    }
#undef SLIM_ROWPREP
    if (hipGetLastError() != hipSuccess) return SLIM_EDEVICE;
  }
  if (a.r > 0) {
    int st = slim_launch_adapter_gemm(a.act16, a.M, a.red, a.ad_q, a.r, p, ws, s);
    if (st != SLIM_OK) return st;
    // the factor needs re-laying only when given row-major (backward); tm needs summing only
    // when the GEMM split its reduction
    const int64_t np = a.p_tiled ? 0 : (a.rows * a.r / 8 + 255) / 256;
    const int64_t nt = p.ad_split > 1 ? ((a.M + 31) / 32 * 32 * a.r / 8 + 255) / 256 : 0;
    if (np + nt > 0) {
      SlimKernelTimer timer("adapter_finish", s);
      SLIM_LAUNCH(timer, k_adapter_finish, dim3((unsigned)(np + nt)), dim3(256), s,
                  reinterpret_cast<const u32x4_t*>(a.ad_p), a.rows, a.r,
                  reinterpret_cast<u32x4_t*>(const_cast<uint16_t*>(a.ad_pb)), np, a.tpart, p.ad_split, a.M,
                  reinterpret_cast<u32x4_t*>(a.tm));
      if (hipGetLastError() != hipSuccess) return SLIM_EDEVICE;
    }
  }
  SlimKernelTimer timer(BWD ? "tile_bwd" : "tile_fwd", s);
  dim3 grid((unsigned)(8 * ((p.sp_row_tiles * p.sp_col_tiles + 7) / 8)));
  // 8 waves of 64 rows (the kernel also builds with 4 of 128, one wave per SIMD, which measured
  // slower on every workload once tm came through LDS)
  if (p.sp_cols_tile == 128) SLIM_LAUNCH(timer, (k_tile<BWD, 128, 64>), grid, dim3(TileShape<128, 64>::kThreads), s, a);
  else SLIM_LAUNCH(timer, (k_tile<BWD, 96, 64>), grid, dim3(TileShape<96, 64>::kThreads), s, a);
  return hipGetLastError() == hipSuccess ? SLIM_OK : SLIM_EDEVICE;
}

LayerArgs make_args(const SlimPlan& p, char* ws, const void* act, int dtype, int64_t M, int64_t rows, int64_t red,
                    const uint8_t* codes, const uint8_t* meta, const uint16_t* scales, const uint16_t* ad_q,
                    const uint16_t* ad_p, bool p_tiled, int64_t r, float* out) {
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
  a.p_tiled = p_tiled;
  a.ad_pb = p.decode ? nullptr : (p_tiled ? ad_p : reinterpret_cast<const uint16_t*>(ws + p.off_pb));
  a.tm = reinterpret_cast<uint16_t*>(ws + p.off_t);
  a.trinv = reinterpret_cast<float*>(ws + p.off_rowinv);
  // large M: the activations are scaled per row into an fp16 copy (p.scaled), except fp16
  // activations of a forward without an adapter, which the tile kernel streams as they are
  a.act16 = p.scaled ? reinterpret_cast<const uint16_t*>(ws + p.off_x16) : a.act;
  a.rowinv = p.scaled ? reinterpret_cast<const float*>(ws + p.off_rowinv) : nullptr;
  a.out = out;
  a.split = p.sp_split;
  a.row_tiles = p.sp_row_tiles;
  a.units = p.dec_units;
  a.col_tiles = p.sp_col_tiles;
  a.ad_split = p.ad_split;
  a.ad_sub = p.ad_sub;
  a.ad_jblocks = p.ad_jblocks;
  a.part = reinterpret_cast<float*>(ws + p.off_ypart);
  a.tpart = reinterpret_cast<float*>(ws + p.off_tpart);
  a.tcounters = reinterpret_cast<uint32_t*>(ws + p.off_counters);
  a.finish = p.decode && (p.sp_split > 1 || r > 0);
  a.q4 = nullptr;
  a.q4s = nullptr;
  a.p4 = nullptr;
  a.p4s = nullptr;
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
  const LayerArgs a = make_args(p, w, X, xdtype, M, N, K, codes, meta, scales, Lt, Rt, true, r, Y);
  return launch_layer<false>(a, p, reinterpret_cast<const uint16_t*>(X), xdtype == SLIM_BF16, w, (hipStream_t)stream);
}

extern "C" int slim_linear_qa(const void* X, int xdtype, int64_t M, int64_t N, int64_t K, const uint8_t* codes,
                              const uint8_t* meta, const uint16_t* scales, const uint8_t* Lq, const uint16_t* Ls,
                              const uint8_t* Rq, const uint16_t* Rs, int64_t r, float* Y, void* ws, size_t ws_bytes,
                              void* stream) {
  SlimPlan p;
  int st = slim_check_linear_qa(X, xdtype, M, N, K, codes, meta, scales, Lq, Ls, Rq, Rs, r, Y, ws, ws_bytes, &p);
  if (st != SLIM_OK) return st;
  char* w = reinterpret_cast<char*>(ws);
  // the fp16 factor pointers are the large-M expansions in the workspace (unused at small M, where the
  // kernels dequantize the 4-bit factors in registers)
  const uint16_t* q16 = reinterpret_cast<const uint16_t*>(w + p.off_q16);
  const uint16_t* p16 = reinterpret_cast<const uint16_t*>(w + p.off_p16);
  LayerArgs a = make_args(p, w, X, xdtype, M, N, K, codes, meta, scales, q16, p16, true, r, Y);
  a.q4 = reinterpret_cast<const uint32_t*>(Lq);
  a.q4s = Ls;
  a.p4 = reinterpret_cast<const uint32_t*>(Rq);
  a.p4s = Rs;
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
  const LayerArgs a = make_args(p, w, dY, dydtype, M, K, N, codesT, metaT, scalesT, R, L, false, r, dX);
  return launch_layer<true>(a, p, reinterpret_cast<const uint16_t*>(dY), dydtype == SLIM_BF16, w, (hipStream_t)stream);
}

// ------------------------------------------------------------------- no-allocation entry point
// slim_linear_noalloc runs slim_linear's kernels on this file-scope array instead of a caller
// workspace. Each device the library runs on holds its own copy until the process ends. Host code
// never passes the array's name to a kernel (on the host it is only a stand-in for the symbol):
// the device address comes from hipGetSymbolAddress, once per device, with that device current.
static __device__ __align__(256) uint8_t scratch[SLIM_NOALLOC_SCRATCH_BYTES];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
char* g_scratch_ptr[kMaxDevices] = {};

__global__ void __launch_bounds__(256) k_zero_u32(uint32_t* __restrict__ p, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i < n) p[i] = 0u;
}

// The current device's scratch address. At its first use on a device the counter region (which
// every call leaves at zero) is cleared by a fill kernel on `s`, ahead of the call's kernels.
int scratch_for_current_device(hipStream_t s, char** out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return SLIM_EDEVICE;
  if (dev < 0 || dev >= kMaxDevices) return SLIM_EUNSUPPORTED;
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || ptr == nullptr) return SLIM_EDEVICE;
    hipLaunchKernelGGL(k_zero_u32, dim3(SLIM_COUNTER_SLOTS / 256), dim3(256), 0, s, reinterpret_cast<uint32_t*>(ptr),
                       (int64_t)SLIM_COUNTER_SLOTS);
    if (hipGetLastError() != hipSuccess) return SLIM_EDEVICE;
    g_scratch_ptr[dev] = reinterpret_cast<char*>(ptr);
  }
  *out = g_scratch_ptr[dev];
  return SLIM_OK;
}
static_assert(SLIM_COUNTER_SLOTS % 256 == 0, "counter region cleared by whole blocks");
}  // namespace

extern "C" int slim_linear_noalloc(const void* X, int xdtype, int64_t M, int64_t N, int64_t K, const uint8_t* codes,
                                   const uint8_t* meta, const uint16_t* scales, const uint16_t* Lt,
                                   const uint16_t* Rt, int64_t r, float* Y, void* stream) {
  // the size checks come first, so a call the scratch cannot hold touches no device
  SlimPlan p;
  int st = slim_make_plan(false, M, N, K, r, &p);
  if (st != SLIM_OK) return st;
  if (p.total > (size_t)SLIM_NOALLOC_SCRATCH_BYTES) return SLIM_EWORKSPACE;
  hipStream_t s = (hipStream_t)stream;
  char* w = nullptr;
  st = scratch_for_current_device(s, &w);
  if (st != SLIM_OK) return st;
  st = slim_check_linear(false, X, xdtype, M, N, K, codes, meta, scales, Lt, Rt, r, Y, w,
                         (size_t)SLIM_NOALLOC_SCRATCH_BYTES, &p);
  if (st != SLIM_OK) return st;
  SlimTimingOff no_events;   // timing would create hip events on first use
  const LayerArgs a = make_args(p, w, X, xdtype, M, N, K, codes, meta, scales, Lt, Rt, true, r, Y);
  return launch_layer<false>(a, p, reinterpret_cast<const uint16_t*>(X), xdtype == SLIM_BF16, w, s);
}
