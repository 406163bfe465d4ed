// sparse_gemm.hip - the 2:4-sparse int4 contraction with the adapter's second product fused
// into the epilogue.
//
//   forward   Y[m, n]  = sum_k X[m, k] Wc[n, k]          + sum_j T[m, j] R[j, n]
//   backward  dX[m, k] = sum_n dY[m, n] W^{R,C}[n, k]    + sum_j U[m, j] L[k, j]
//
// Both are "out[m, row] = sum_red act[m, red] A[row, red] + sum_j tm[m, j] ap(row, j)" with A the
// packed sparse operand (rows = N, red = K forward; rows = K, red = N backward). The packed rows
// feed the sparse MFMA's compressed A operand straight from their code words; activations are
// the dense B operand, staged in LDS as fp16. The accumulator holds out^T tiles (rows x m).
//
// Scales: forward, s16[n, k/128] varies along the output row and is applied while dequantising
// (fp16 product). Backward, the scale s16[n, k/128] varies along the reduction n, so it is folded
// into the activations instead (B'[n, m] = dY[m, n] * s16[n, g], one g per 128-row tile) and
// the codes enter the MFMA as exact integers.
#include "slim_device.h"
#include "slim_launch.h"

namespace {

struct SpArgs {
  const uint32_t* codes;   // [rows, red/16] code words
  const uint32_t* meta;    // [rows, red/32] words = two index half-words
  const uint16_t* scales;  // forward [rows, red/128]; backward scalesT [rows/128, red]
  const uint16_t* act;     // [M, red] activations (bf16 or fp16 bits)
  int act_bf16;
  int64_t M, rows, red;
  int64_t cps;             // 128-wide chunks per split (small-M kernel)
  int split;
  const float* tm;         // [M, r] fp32 adapter intermediate, or null when r == 0
  const uint16_t* ap;      // forward R [r, rows]; backward L [rows, r]
  int64_t r;
  float* out;              // [M, rows]
  float* part;             // split partial tiles
  uint32_t* counters;      // one per output tile
};

// Eight activations at (m, red .. red+7) -> fp16, with the backward's scale fold.
template <bool BWD>
SLIM_DEV h8_t stage8(const SpArgs& a, int64_t m, int64_t red, int64_t sgroup) {
  h8_t h;
#pragma unroll
  for (int e = 0; e < 8; ++e) h[e] = (_Float16)0.0f;
  if (m >= a.M) return h;
  const u32x4_t v = *reinterpret_cast<const u32x4_t*>(a.act + m * a.red + red);
  if (!BWD) return load8_as_h(v, a.act_bf16 != 0);
  const u32x4_t sv = *reinterpret_cast<const u32x4_t*>(a.scales + sgroup * a.red + red);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const float x0 = act_to_f(v[i] & 0xFFFFu, a.act_bf16 != 0), x1 = act_to_f(v[i] >> 16, a.act_bf16 != 0);
    h[2 * i] = (_Float16)(x0 * h_bits_to_f(sv[i] & 0xFFFFu));
    h[2 * i + 1] = (_Float16)(x1 * h_bits_to_f(sv[i] >> 16));
  }
  return h;
}

// Eight fp32 adapter-intermediate values -> fp16.
SLIM_DEV h8_t tm8(const SpArgs& a, int64_t m, int64_t j) {
  h8_t h;
  if (m < a.M && j < a.r) {
    const float4 x = *reinterpret_cast<const float4*>(a.tm + m * a.r + j);
    const float4 y = *reinterpret_cast<const float4*>(a.tm + m * a.r + j + 4);
    h[0] = (_Float16)x.x; h[1] = (_Float16)x.y; h[2] = (_Float16)x.z; h[3] = (_Float16)x.w;
    h[4] = (_Float16)y.x; h[5] = (_Float16)y.y; h[6] = (_Float16)y.z; h[7] = (_Float16)y.w;
  } else {
#pragma unroll
    for (int e = 0; e < 8; ++e) h[e] = (_Float16)0.0f;
  }
  return h;
}

// ================================================================ small-M kernel (M <= 64)
// Block = 4 waves = 64 output rows; each wave owns 16 rows and FM 16-column fragments.
// blockIdx.y splits the reduction; the last block of a row tile sums the partials in order.
template <bool BWD, int FM>
__global__ void __launch_bounds__(256)
k_sparse_small_m(SpArgs a) {
  extern __shared__ __attribute__((aligned(16))) _Float16 xs[];   // [16*FM][ldx]
  __shared__ __attribute__((aligned(16))) _Float16 rt[64][40];     // forward adapter: R^T slab
  __shared__ int last_flag;
  constexpr int MC = 16 * FM;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int64_t row0 = (int64_t)blockIdx.x * 64;
  const int s = blockIdx.y;
  const int64_t c_beg = (int64_t)s * a.cps;
  const int nch = (int)min(a.cps, a.red / 128 - c_beg);
  const int ldx = (int)a.cps * 128 + 8;
  const int64_t red0 = c_beg * 128;

  // stage the activation slice [MC x nch*128] as fp16
  {
    const int vpr = nch * 16;
    const int64_t sgroup = row0 / 128;
    for (int idx = tid; idx < MC * vpr; idx += 256) {
      const int m = idx / vpr, vc = idx - m * vpr;
      *reinterpret_cast<h8_t*>(&xs[m * ldx + 8 * vc]) = stage8<BWD>(a, m, red0 + 8 * vc, sgroup);
    }
  }
  __syncthreads();

  f4_t acc[FM];
#pragma unroll
  for (int f = 0; f < FM; ++f) acc[f] = f4_t{0.f, 0.f, 0.f, 0.f};
  const int64_t arow = row0 + 16 * wave + (lane & 15);
  const int64_t lrow = arow < a.rows ? arow : a.rows - 1;
  const int qa = lane >> 4;
  const uint32_t* cp = a.codes + lrow * (a.red / 16) + c_beg * 8 + 2 * qa;
  const uint32_t* mp = a.meta + lrow * (a.red / 32) + c_beg * 4 + qa;
  const uint16_t* sp = a.scales + lrow * (a.red / 128) + c_beg;

  constexpr int PF = 8;   // chunks whose packed words are loaded ahead
  for (int cb = 0; cb < nch; cb += PF) {
    u32x2_t cw[PF];
    uint32_t mw[PF], sw[PF];
#pragma unroll
    for (int i = 0; i < PF; ++i) {
      if (cb + i < nch) {
        cw[i] = *reinterpret_cast<const u32x2_t*>(cp + 8 * (cb + i));
        mw[i] = mp[4 * (cb + i)];
        sw[i] = BWD ? 0u : (uint32_t)sp[cb + i];
      }
    }
#pragma unroll
    for (int i = 0; i < PF; ++i) {
      if (cb + i < nch) {
        const h2_t s2 = splat_h2(sw[i]);
        const int base = (cb + i) * 128;
#pragma unroll
        for (int st = 0; st < 2; ++st) {
          const h8_t av = BWD ? dequant_word_int(cw[i][st]) : dequant_word(cw[i][st], s2);
          const int off = base + b_chunk_offset<16>(lane, st);
#pragma unroll
          for (int f = 0; f < FM; ++f) {
            const _Float16* xr = xs + (16 * f + (lane & 15)) * ldx + off;
            const h16_t bv = cat16(*reinterpret_cast<const h8_t*>(xr), *reinterpret_cast<const h8_t*>(xr + 64));
            acc[f] = smfmac16(av, bv, acc[f], (int)mw[i], st);
          }
        }
      }
    }
  }

  // split reduction: the last block of this row tile sums the partials in split order
  if (a.split > 1) {
    const int tile = blockIdx.x;
    float* dst = a.part + ((int64_t)s * gridDim.x + tile) * (64 * MC);
#pragma unroll
    for (int f = 0; f < FM; ++f)
#pragma unroll
      for (int v = 0; v < 4; ++v) dst[((wave * FM + f) * 4 + v) * 64 + lane] = acc[f][v];
    __threadfence();
    __syncthreads();
    if (tid == 0) {
      const uint32_t done = atomicAdd(&a.counters[tile], 1u);
      last_flag = (done == (uint32_t)(a.split - 1));
    }
    __syncthreads();
    if (!last_flag) return;
    __threadfence();
#pragma unroll
    for (int f = 0; f < FM; ++f) acc[f] = f4_t{0.f, 0.f, 0.f, 0.f};
    for (int ss = 0; ss < a.split; ++ss) {
      const float* src = a.part + ((int64_t)ss * gridDim.x + tile) * (64 * MC);
#pragma unroll
      for (int f = 0; f < FM; ++f)
#pragma unroll
        for (int v = 0; v < 4; ++v) acc[f][v] += src[((wave * FM + f) * 4 + v) * 64 + lane];
    }
    if (tid == 0) a.counters[tile] = 0u;
  }

  // adapter: out^T[row, m] += sum_j ap(row, j) tm[m, j], 16x16x32 fp16 MFMA over j
  if (a.r > 0) {
    for (int64_t j0 = 0; j0 < a.r; j0 += 32) {
      h8_t av;
      const int64_t jj = j0 + 8 * (lane >> 4);
      if (BWD) {
        u32x4_t v = {0u, 0u, 0u, 0u};
        if (jj < a.r) v = *reinterpret_cast<const u32x4_t*>(a.ap + lrow * a.r + jj);
        av = __builtin_bit_cast(h8_t, v);
      } else {
        __syncthreads();
        {
          const int jr = tid >> 3, nc = tid & 7;   // 32 rows of R x 8 vectors of 8 columns
          const int64_t gj = j0 + jr, gn = row0 + 8 * nc;
          u32x4_t v = {0u, 0u, 0u, 0u};
          if (gj < a.r && gn < a.rows) v = *reinterpret_cast<const u32x4_t*>(a.ap + gj * a.rows + gn);
          const h8_t hv = __builtin_bit_cast(h8_t, v);
#pragma unroll
          for (int e = 0; e < 8; ++e) rt[8 * nc + e][jr] = hv[e];
        }
        __syncthreads();
        av = *reinterpret_cast<const h8_t*>(&rt[16 * wave + (lane & 15)][8 * (lane >> 4)]);
      }
#pragma unroll
      for (int f = 0; f < FM; ++f) {
        const h8_t bv = tm8(a, 16 * f + (lane & 15), jj);
        acc[f] = __builtin_amdgcn_mfma_f32_16x16x32_f16(av, bv, acc[f], 0, 0, 0);
      }
    }
  }

  // D[i][j] of a 16x16 fragment: lane j + 16 * (i / 4), element i % 4 -> 4 consecutive rows
  const int64_t rr = row0 + 16 * wave + 4 * (lane >> 4);
  if (rr < a.rows) {
#pragma unroll
    for (int f = 0; f < FM; ++f) {
      const int64_t m = 16 * f + (lane & 15);
      if (m < a.M) *reinterpret_cast<f4_t*>(a.out + m * a.rows + rr) = acc[f];
    }
  }
}

// ================================================================ tile kernel (large M)
// Block = WN x WM waves; each wave owns 128 rows (4 fragments of 32) x 64 columns (2 of 32),
// on 32x32x32 sparse MFMA. Activations stream through a double-buffered LDS tile of 128
// reduction positions (one quantisation group) per step.
template <bool BWD, int WN, int WM>
__global__ void __launch_bounds__(64 * WN * WM)
k_sparse_tile(SpArgs a) {
  constexpr int NT = 64 * WN * WM;
  constexpr int BR = 128 * WN, BC = 64 * WM;
  constexpr int LDX = 128 + 8;
  constexpr int XV = BC * 16 / NT;          // 16-byte activation vectors per thread per chunk
  __shared__ __attribute__((aligned(16))) _Float16 xs[2][BC][LDX];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wn = wave % WN, wm = wave / WN;
  const int64_t row0 = (int64_t)blockIdx.x * BR, m0 = (int64_t)blockIdx.y * BC;
  const int64_t nch = a.red / 128;
  const int64_t sgroup = row0 / 128;

  auto stage = [&](int64_t c, int buf) {
#pragma unroll
    for (int i = 0; i < XV; ++i) {
      const int idx = tid + NT * i, m = idx >> 4, vc = idx & 15;
      *reinterpret_cast<h8_t*>(&xs[buf][m][8 * vc]) = stage8<BWD>(a, m0 + m, c * 128 + 8 * vc, sgroup);
    }
  };

  f16_t acc[4][2];
#pragma unroll
  for (int fn = 0; fn < 4; ++fn)
#pragma unroll
    for (int fm = 0; fm < 2; ++fm)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[fn][fm][v] = 0.f;

  const uint32_t* cp[4];
  const uint32_t* mp[4];
  const uint16_t* sp[4];
  const int ha = lane >> 5;
#pragma unroll
  for (int fn = 0; fn < 4; ++fn) {
    int64_t arow = row0 + 128 * wn + 32 * fn + (lane & 31);
    if (arow >= a.rows) arow = a.rows - 1;
    cp[fn] = a.codes + arow * (a.red / 16) + 4 * ha;
    mp[fn] = a.meta + arow * (a.red / 32) + 2 * ha;
    sp[fn] = a.scales + arow * (a.red / 128);
  }

  stage(0, 0);
  __syncthreads();
  for (int64_t c = 0; c < nch; ++c) {
    const int buf = (int)(c & 1);
    u32x4_t cw[4];
    u32x2_t mw[4];
    h2_t s2[4];
#pragma unroll
    for (int fn = 0; fn < 4; ++fn) {
      cw[fn] = *reinterpret_cast<const u32x4_t*>(cp[fn] + 8 * c);
      mw[fn] = *reinterpret_cast<const u32x2_t*>(mp[fn] + 4 * c);
      s2[fn] = BWD ? splat_h2(0x3C00u) : splat_h2(sp[fn][c]);
    }
    // activations of the next chunk: global -> registers now, registers -> LDS after the math
    h8_t nx[XV];
    const bool more = c + 1 < nch;
    if (more) {
#pragma unroll
      for (int i = 0; i < XV; ++i) {
        const int idx = tid + NT * i, m = idx >> 4, vc = idx & 15;
        nx[i] = stage8<BWD>(a, m0 + m, (c + 1) * 128 + 8 * vc, sgroup);
      }
    }
#pragma unroll
    for (int st = 0; st < 4; ++st) {
      h8_t av[4];
      h16_t bv[2];
#pragma unroll
      for (int fn = 0; fn < 4; ++fn) av[fn] = BWD ? dequant_word_int(cw[fn][st]) : dequant_word(cw[fn][st], s2[fn]);
      const int off = b_chunk_offset<32>(lane, st);
#pragma unroll
      for (int fm = 0; fm < 2; ++fm) {
        const _Float16* xr = &xs[buf][64 * wm + 32 * fm + (lane & 31)][off];
        bv[fm] = cat16(*reinterpret_cast<const h8_t*>(xr), *reinterpret_cast<const h8_t*>(xr + 64));
      }
#pragma unroll
      for (int fn = 0; fn < 4; ++fn)
#pragma unroll
        for (int fm = 0; fm < 2; ++fm)
          acc[fn][fm] = smfmac32(av[fn], bv[fm], acc[fn][fm], (int)mw[fn][st >> 1], st & 1);
    }
    if (more) {
#pragma unroll
      for (int i = 0; i < XV; ++i) {
        const int idx = tid + NT * i, m = idx >> 4, vc = idx & 15;
        *reinterpret_cast<h8_t*>(&xs[buf ^ 1][m][8 * vc]) = nx[i];
      }
    }
    __syncthreads();
  }

  // adapter: out^T[row, m] += sum_j ap(row, j) tm[m, j] on 32x32x16 fp16 MFMA, 32 j per slab
  if (a.r > 0) {
    _Float16(*at)[40] = reinterpret_cast<_Float16(*)[40]>(&xs[0][0][0]);   // [BR][40]
    _Float16(*ts)[40] = reinterpret_cast<_Float16(*)[40]>(&xs[1][0][0]);   // [BC][40]
    static_assert(BR * 40 <= BC * LDX, "adapter slab must fit in one activation buffer");
    for (int64_t j0 = 0; j0 < a.r; j0 += 32) {
      __syncthreads();
      if (BWD) {   // L [rows, r]: rows contiguous along j
        for (int idx = tid; idx < BR * 4; idx += NT) {
          const int row = idx >> 2, jc = idx & 3;
          const int64_t gr = row0 + row, gj = j0 + 8 * jc;
          u32x4_t v = {0u, 0u, 0u, 0u};
          if (gr < a.rows && gj < a.r) v = *reinterpret_cast<const u32x4_t*>(a.ap + gr * a.r + gj);
          *reinterpret_cast<u32x4_t*>(&at[row][8 * jc]) = v;
        }
      } else {     // R [r, rows]: transpose on the way in
        for (int idx = tid; idx < 32 * (BR / 8); idx += NT) {
          const int jr = idx / (BR / 8), nc = idx % (BR / 8);
          const int64_t gj = j0 + jr, gn = row0 + 8 * nc;
          u32x4_t v = {0u, 0u, 0u, 0u};
          if (gj < a.r && gn < a.rows) v = *reinterpret_cast<const u32x4_t*>(a.ap + gj * a.rows + gn);
          const h8_t hv = __builtin_bit_cast(h8_t, v);
#pragma unroll
          for (int e = 0; e < 8; ++e) at[8 * nc + e][jr] = hv[e];
        }
      }
      for (int idx = tid; idx < BC * 4; idx += NT) {
        const int m = idx >> 2, jc = idx & 3;
        *reinterpret_cast<h8_t*>(&ts[m][8 * jc]) = tm8(a, m0 + m, j0 + 8 * jc);
      }
      __syncthreads();
#pragma unroll
      for (int kk = 0; kk < 32; kk += 16) {
        h8_t av[4], bv[2];
#pragma unroll
        for (int fn = 0; fn < 4; ++fn)
          av[fn] = *reinterpret_cast<const h8_t*>(&at[128 * wn + 32 * fn + (lane & 31)][kk + 8 * ha]);
#pragma unroll
        for (int fm = 0; fm < 2; ++fm)
          bv[fm] = *reinterpret_cast<const h8_t*>(&ts[64 * wm + 32 * fm + (lane & 31)][kk + 8 * ha]);
#pragma unroll
        for (int fn = 0; fn < 4; ++fn)
#pragma unroll
          for (int fm = 0; fm < 2; ++fm)
            acc[fn][fm] = __builtin_amdgcn_mfma_f32_32x32x16_f16(av[fn], bv[fm], acc[fn][fm], 0, 0, 0);
      }
    }
  }

  // D[i][j] of a 32x32 fragment: lane j + 32 * ((i / 4) % 2), element 4 * (i / 8) + i % 4
#pragma unroll
  for (int fm = 0; fm < 2; ++fm) {
    const int64_t m = m0 + 64 * wm + 32 * fm + (lane & 31);
    if (m >= a.M) continue;
#pragma unroll
    for (int fn = 0; fn < 4; ++fn)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int64_t rr = row0 + 128 * wn + 32 * fn + 8 * q + 4 * ha;
        if (rr < a.rows) {
          f4_t o = {acc[fn][fm][4 * q], acc[fn][fm][4 * q + 1], acc[fn][fm][4 * q + 2], acc[fn][fm][4 * q + 3]};
          *reinterpret_cast<f4_t*>(a.out + m * a.rows + rr) = o;
        }
      }
  }
}

template <bool BWD>
int launch_sparse(const SpArgs& a, const SlimPlan& p, hipStream_t s) {
  if (p.decode) {
    dim3 grid((unsigned)p.sp_row_tiles, (unsigned)p.sp_split);
    switch (p.dec_fm) {
      case 1: hipLaunchKernelGGL((k_sparse_small_m<BWD, 1>), grid, dim3(256), p.lds_bytes, s, a); break;
      case 2: hipLaunchKernelGGL((k_sparse_small_m<BWD, 2>), grid, dim3(256), p.lds_bytes, s, a); break;
      default: hipLaunchKernelGGL((k_sparse_small_m<BWD, 4>), grid, dim3(256), p.lds_bytes, s, a); break;
    }
  } else {
    dim3 grid((unsigned)p.sp_row_tiles, (unsigned)p.sp_col_tiles);
    if (BWD)
      hipLaunchKernelGGL((k_sparse_tile<true, 1, 2>), grid, dim3(128), 0, s, a);
    else
      hipLaunchKernelGGL((k_sparse_tile<false, 2, 2>), grid, dim3(256), 0, s, a);
  }
  return hipGetLastError() == hipSuccess ? SLIM_OK : SLIM_EDEVICE;
}

SpArgs make_args(const SlimPlan& p, char* ws, const void* act, int dtype, int64_t M, int64_t rows, int64_t red,
                 const uint8_t* codes, const uint8_t* meta, const uint16_t* scales, const uint16_t* ap, int64_t r,
                 float* out) {
  SpArgs a;
  a.codes = reinterpret_cast<const uint32_t*>(codes);
  a.meta = reinterpret_cast<const uint32_t*>(meta);
  a.scales = scales;
  a.act = reinterpret_cast<const uint16_t*>(act);
  a.act_bf16 = dtype == SLIM_BF16;
  a.M = M;
  a.rows = rows;
  a.red = red;
  a.cps = p.sp_chunks_per_split;
  a.split = p.sp_split;
  a.tm = r > 0 ? reinterpret_cast<const float*>(ws + p.off_t) : nullptr;
  a.ap = ap;
  a.r = r;
  a.out = out;
  a.part = reinterpret_cast<float*>(ws + p.off_ypart);
  a.counters = reinterpret_cast<uint32_t*>(ws + p.off_counters) + p.sp_counter_base;
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
  hipStream_t s = (hipStream_t)stream;
  char* w = reinterpret_cast<char*>(ws);
  if (r > 0) {
    st = slim_launch_adapter_gemm(false, reinterpret_cast<const uint16_t*>(X), xdtype == SLIM_BF16, M, K, L, r, p, w, s);
    if (st != SLIM_OK) return st;
  }
  const SpArgs a = make_args(p, w, X, xdtype, M, N, K, codes, meta, scales, R, r, Y);
  return launch_sparse<false>(a, p, s);
}

extern "C" int slim_linear_bwd_dx(const void* dY, int dydtype, int64_t M, int64_t N, int64_t K,
                                  const uint8_t* codesT, const uint8_t* metaT, const uint16_t* scalesT,
                                  const uint16_t* L, const uint16_t* R, int64_t r, float* dX, void* ws,
                                  size_t ws_bytes, void* stream) {
  SlimPlan p;
  int st = slim_check_linear(true, dY, dydtype, M, N, K, codesT, metaT, scalesT, L, R, r, dX, ws, ws_bytes, &p);
  if (st != SLIM_OK) return st;
  hipStream_t s = (hipStream_t)stream;
  char* w = reinterpret_cast<char*>(ws);
  if (r > 0) {
    st = slim_launch_adapter_gemm(true, reinterpret_cast<const uint16_t*>(dY), dydtype == SLIM_BF16, M, N, R, r, p, w,
                                  s);
    if (st != SLIM_OK) return st;
  }
  const SpArgs a = make_args(p, w, dY, dydtype, M, K, N, codesT, metaT, scalesT, L, r, dX);
  return launch_sparse<true>(a, p, s);
}
