// pack.hip - one-time packing kernels: forward 2:4 + int4 group-128 pack, and the SLoPe
// double-pruned backward pack (2:4 along N of the packed forward weight).
#include "slim_device.h"
#include "slim_host.h"
#include "slim_timing.h"

namespace {

constexpr int kPackThreads = 256;

// One thread per aligned 4-group of one row; the 32 threads of a half-wave cover one
// 128-wide quantisation group (rows hold K/4 groups and K % 128 == 0, so groups never
// straddle half-waves). With `alpha` (one float64 in device memory, SLiM-Quant's per-tensor
// parameter) every group takes it in place of its own absmax.
__global__ void __launch_bounds__(kPackThreads)
k_pack(const float4* __restrict__ W, int64_t total4, int64_t K, uint32_t* __restrict__ codes,
       uint16_t* __restrict__ meta, uint16_t* __restrict__ scales, uint32_t* __restrict__ mask,
       int* __restrict__ status, const double* __restrict__ alpha) {
  const int64_t t = (int64_t)blockIdx.x * kPackThreads + threadIdx.x;
  const bool valid = t < total4;
  float4 v = valid ? W[t] : make_float4(0.f, 0.f, 0.f, 0.f);
  const float w[4] = {v.x, v.y, v.z, v.w};
  float a[4];
  int bad = 0;
#pragma unroll
  for (int p = 0; p < 4; ++p) {
    a[p] = fabsf(w[p]);
    if (!__builtin_isfinite(w[p])) bad = 1;
  }
  // group absmax over the 32 lanes of this half-wave
  float gmax = fmaxf(fmaxf(a[0], a[1]), fmaxf(a[2], a[3]));
#pragma unroll
  for (int off = 16; off >= 1; off >>= 1) gmax = fmaxf(gmax, __shfl_xor(gmax, off, 32));
  // s16 = fp16_RNE(fp32 absmax / 7), IEEE division (alpha rounded to fp32 in its place)
  if (alpha) {
    const double ad = *alpha;
    if (!(ad >= 0.0)) bad |= 2;
    gmax = (float)ad;
  }
  const float s32 = __fdiv_rn(gmax, 7.0f);
  const _Float16 s16 = (_Float16)s32;
  const uint16_t s16bits = __builtin_bit_cast(uint16_t, s16);
  if (!__builtin_isfinite((float)s16)) bad |= 2;
  if (valid && bad) atomicOr(status, bad);

  // top-2 of the four by (|w| desc, position asc)
  int keep[4];
#pragma unroll
  for (int p = 0; p < 4; ++p) {
    int rank = 0;
#pragma unroll
    for (int q = 0; q < 4; ++q)
      if (q != p && (a[q] > a[p] || (a[q] == a[p] && q < p))) ++rank;
    keep[p] = rank < 2;
  }
  int i0 = -1, i1 = -1;
#pragma unroll
  for (int p = 0; p < 4; ++p)
    if (keep[p]) {
      if (i0 < 0) i0 = p;
      else i1 = p;
    }
  const double sd = (double)s16;
  auto code = [&](float x) -> uint32_t {
    if (!(sd > 0.0)) return 8u;
    double q = rint((double)x / sd);
    q = fmin(7.0, fmax(-7.0, q));
    return (uint32_t)((int)q + 8);
  };
  const uint32_t u0 = code(w[i0]);
  const uint32_t u1 = code(w[i1]);
  const int64_t j = t % (K / 4);          // group index inside the row
  const int c = (int)(t & 3);             // group slot inside its 16-position block
  uint32_t cw = (u0 << (4 * c)) | (u1 << (16 + 4 * c));
  uint32_t mw = (uint32_t)(i0 | (i1 << 2)) << (4 * c);
  cw |= __shfl_xor(cw, 1, 64);
  mw |= __shfl_xor(mw, 1, 64);
  cw |= __shfl_xor(cw, 2, 64);
  mw |= __shfl_xor(mw, 2, 64);
  if (!valid) return;
  const int64_t row = t / (K / 4);
  const int64_t slot = packed_slot(row, j >> 5, K / 128);   // word (j >> 2) & 7 of chunk j >> 5
  if (c == 0) {
    codes[8 * slot + ((j >> 2) & 7)] = cw;
    meta[8 * slot + ((j >> 2) & 7)] = (uint16_t)mw;
  }
  if ((j & 31) == 0) scales[slot] = s16bits;
  if (mask) mask[t] = (uint32_t)keep[0] | ((uint32_t)keep[1] << 8) | ((uint32_t)keep[2] << 16) |
                      ((uint32_t)keep[3] << 24);
}

// Backward pack. Block = 256 threads, tile = 64 rows (n) x 64 columns (k).
// Phase 1 decodes the forward pack of the tile into LDS; phase 2 gives each thread one
// column k and one 16-row block, prunes each aligned 4-row group to its top two
// (|Wc| desc, forward-kept desc, row asc) and emits one codesT word and one metaT half-word.
constexpr int kBT = 64;
// Largest forward scale the backward accepts: its large-M path multiplies gradients scaled below
// 2^(kActExp + 1) = 32 by s16 in fp16, which stays below 65504 for s16 < 2048.
constexpr float kBwdScaleLimit = 2048.0f;
static_assert(kActExp == 4, "kBwdScaleLimit assumes row-scaled activations below 32");

__global__ void __launch_bounds__(256)
k_pack_bwd(const uint32_t* __restrict__ codes, const uint16_t* __restrict__ meta,
           const uint16_t* __restrict__ scales, int64_t N, int64_t K, uint32_t* __restrict__ codesT,
           uint16_t* __restrict__ metaT, uint16_t* __restrict__ scalesT, uint8_t* __restrict__ mask_rc,
           int* __restrict__ status) {
  __shared__ uint8_t u_s[kBT][kBT + 4];     // forward code per (row, col), 8 where pruned
  __shared__ uint8_t f_s[kBT][kBT + 4];     // forward-kept bit, later the W^{R,C} support bit
  __shared__ float sc_s[kBT];               // scale of each row for this column tile
  const int tid = threadIdx.x;
  const int64_t k0 = (int64_t)blockIdx.x * kBT;
  const int64_t n0 = (int64_t)blockIdx.y * kBT;
  const int rows = (int)min((int64_t)kBT, N - n0);   // multiple of 16 (N % 16 == 0)

  // phase 1: thread -> (row = tid / 4, 16-column block w = tid % 4)
  {
    const int row = tid >> 2, w = tid & 3;
    if (row < rows) {
      const int64_t n = n0 + row;
      // k0 is a multiple of 64: the tile's four 16-column blocks are words (k0 % 128) / 16 + w
      // of chunk k0 / 128
      const int64_t slot = packed_slot(n, k0 >> 7, K / 128);
      const uint32_t cw = codes[8 * slot + ((k0 & 127) >> 4) + w];
      const uint32_t mw = meta[8 * slot + ((k0 & 127) >> 4) + w];
#pragma unroll
      for (int p = 0; p < 16; ++p) {
        u_s[row][16 * w + p] = 8;
        f_s[row][16 * w + p] = 0;
      }
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const int i0 = (mw >> (4 * c)) & 3, i1 = (mw >> (4 * c + 2)) & 3;
        u_s[row][16 * w + 4 * c + i0] = (cw >> (4 * c)) & 0xF;
        u_s[row][16 * w + 4 * c + i1] = (cw >> (16 + 4 * c)) & 0xF;
        f_s[row][16 * w + 4 * c + i0] = 1;
        f_s[row][16 * w + 4 * c + i1] = 1;
      }
      if (w == 0) {
        sc_s[row] = h_bits_to_f(scales[slot]);
        // the backward's fp16 product of a row-scaled gradient (below 32) and s16 must stay finite
        if (!(sc_s[row] < kBwdScaleLimit)) atomicOr(status, 2);
      }
    }
  }
  __syncthreads();

  // phase 2: thread -> (column col = tid / 4, 16-row block rb = tid % 4)
  uint32_t sel16 = 0;
  const int col = tid >> 2, rb = tid & 3;
  if (16 * rb < rows) {
    uint32_t cw = 0, mw = 0;
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      float av[4];
      int fv[4];
      uint32_t uv[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int row = 16 * rb + 4 * c + i;
        uv[i] = u_s[row][col];
        fv[i] = f_s[row][col];
        av[i] = fabsf((float)((int)uv[i] - 8) * sc_s[row]);   // exact: 3-bit x 11-bit significand
      }
      int keep[4];
#pragma unroll
      for (int p = 0; p < 4; ++p) {
        int rank = 0;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          if (q == p) continue;
          const bool better = av[q] > av[p] || (av[q] == av[p] && (fv[q] > fv[p] || (fv[q] == fv[p] && q < p)));
          if (better) ++rank;
        }
        keep[p] = rank < 2;
      }
      int i0 = -1, i1 = -1;
#pragma unroll
      for (int p = 0; p < 4; ++p)
        if (keep[p]) {
          if (i0 < 0) i0 = p;
          else i1 = p;
        }
      cw |= (uv[i0] << (4 * c)) | (uv[i1] << (16 + 4 * c));
      mw |= (uint32_t)(i0 | (i1 << 2)) << (4 * c);
      sel16 |= (uint32_t)((keep[0] & fv[0]) | ((keep[1] & fv[1]) << 1) | ((keep[2] & fv[2]) << 2) |
                          ((keep[3] & fv[3]) << 3)) << (4 * c);
    }
    // transposed pack: row k, reduction n; n0 is a multiple of 64, so the 16-row block rb is
    // word (n0 % 128) / 16 + rb of chunk n0 / 128
    const int64_t k = k0 + col;
    const int64_t slotT = packed_slot(k, n0 >> 7, N / 128);
    codesT[8 * slotT + ((n0 & 127) >> 4) + rb] = cw;
    metaT[8 * slotT + ((n0 & 127) >> 4) + rb] = (uint16_t)mw;
  }
  if (mask_rc) {
    __syncthreads();
    if (16 * rb < rows) {
#pragma unroll
      for (int i = 0; i < 16; ++i) f_s[16 * rb + i][col] = (sel16 >> i) & 1;
    }
    __syncthreads();
    // write rows of the tile: thread -> (row = tid / 4, 16 bytes at column 16 * (tid % 4))
    const int row = tid >> 2, w = tid & 3;
    if (row < rows) {
      uint32_t v[4];
#pragma unroll
      for (int q = 0; q < 4; ++q)
        v[q] = (uint32_t)f_s[row][16 * w + 4 * q] | ((uint32_t)f_s[row][16 * w + 4 * q + 1] << 8) |
               ((uint32_t)f_s[row][16 * w + 4 * q + 2] << 16) | ((uint32_t)f_s[row][16 * w + 4 * q + 3] << 24);
      uint4* dst = reinterpret_cast<uint4*>(mask_rc + (n0 + row) * K + k0 + 16 * w);
      *dst = make_uint4(v[0], v[1], v[2], v[3]);
    }
  }
  // scalesT: the first column tile of each 128-group copies the tile's row scales
  if ((k0 & 127) == 0 && tid < rows) scalesT[(k0 >> 7) * N + n0 + tid] = scales[packed_slot(n0 + tid, k0 >> 7, K / 128)];
}

// fp16 transpose out[c][r] = in[r][c] of a row-major [R x C] matrix, through a 64 x 64 LDS tile.
__global__ void __launch_bounds__(256)
k_transpose16(const uint16_t* __restrict__ in, int64_t R, int64_t C, uint16_t* __restrict__ out) {
  __shared__ uint16_t t[64][66];
  const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
  const int64_t r0 = (int64_t)blockIdx.y * 64, c0 = (int64_t)blockIdx.x * 64;
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const int rr = ty + 4 * i;
    if (r0 + rr < R && c0 + tx < C) t[rr][tx] = in[(r0 + rr) * C + c0 + tx];
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const int cc = ty + 4 * i;
    if (c0 + cc < C && r0 + tx < R) out[(c0 + cc) * R + r0 + tx] = t[tx][cc];
  }
}

// R [r, N] row-major -> R^T in 32 x 16 tiles: element (n, j) at ((n / 32) (r / 16) + j / 16) 512 +
// (n % 32) 16 + j % 16, rows n >= N of the last tile zero. One thread per output element, in
// output order (a one-time pack: the strided reads do not matter).
__global__ void __launch_bounds__(256) k_tile_rt(const uint16_t* __restrict__ R, int64_t r, int64_t N,
                                                 uint16_t* __restrict__ out) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t total = (N + 31) / 32 * 32 * r;
  if (i >= total) return;
  const int64_t tile = i >> 9, within = i & 511;
  const int64_t tn = tile / (r >> 4), tj = tile - tn * (r >> 4);
  const int64_t n = 32 * tn + (within >> 4), j = 16 * tj + (within & 15);
  out[i] = n < N ? R[j * N + n] : (uint16_t)0;
}

// 4-bit AbsMax pack of one adapter factor laid out as [rows, len] (row-major view of a transposed
// source: element (row, col) is src[col * ld + row]), groups of 128 along len (the last group of a
// row may be shorter). Sixteen consecutive threads share one (row, group): thread i of them codes
// the 8 elements at col = 128 g + 8 i into one 32-bit word (element 2c in nibble c, 2c + 1 in
// nibble c + 4), the group's absmax comes from a 16-lane shuffle, and thread 0 writes the scale.
__global__ void __launch_bounds__(256)
k_pack_adapter_q(const uint16_t* __restrict__ src, int64_t ld, int64_t rows, int64_t len, uint32_t* __restrict__ codes,
                 uint16_t* __restrict__ scales, int* __restrict__ status) {
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t ng = (len + 127) / 128;
  const int64_t pair = t / 16;
  const int i = (int)(t % 16);
  const int64_t row = pair / ng, g = pair % ng;
  const int64_t col0 = 128 * g + 8 * i;
  const bool valid = row < rows && col0 < len;
  float v[8];
  float amax = 0.f;
  int bad = 0;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    v[e] = valid ? h_bits_to_f(src[(col0 + e) * ld + row]) : 0.f;
    if (!__builtin_isfinite(v[e])) bad = 1;
    amax = fmaxf(amax, fabsf(v[e]));
  }
#pragma unroll
  for (int off = 8; off >= 1; off >>= 1) amax = fmaxf(amax, __shfl_xor(amax, off, 16));
  if (valid && bad) atomicOr(status, 1);
  // s16 = fp16_RNE(fp32 absmax / 7), IEEE division; codes against the stored s16 in double precision
  const _Float16 s16 = (_Float16)__fdiv_rn(amax, 7.0f);
  const double sd = (double)(float)s16;
  uint32_t word = 0;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    double q = sd > 0.0 ? rint((double)v[e] / sd) : 0.0;
    q = q < -7.0 ? -7.0 : (q > 7.0 ? 7.0 : q);
    const uint32_t u = (uint32_t)((int)q + 8);
    word |= u << (4 * (e >> 1) + 16 * (e & 1));
  }
  if (!valid) return;
  codes[row * (len / 8) + col0 / 8] = word;
  if (i == 0) scales[row * ng + g] = __builtin_bit_cast(uint16_t, s16);
}

}  // namespace

extern "C" int slim_pack_adapter_q(const uint16_t* L, const uint16_t* R, int64_t K, int64_t N, int64_t r, uint8_t* Lq,
                                   uint16_t* Ls, uint8_t* Rq, uint16_t* Rs, void* stream) {
  if (!L || !R || !Lq || !Ls || !Rq || !Rs) return SLIM_EINVAL;
  if (K < 128 || N < 1 || r < 32 || r % 32 || K % 128 || K >= (int64_t(1) << 31) || N >= (int64_t(1) << 31) ||
      r >= 65536)
    return SLIM_ESHAPE;
  if (!slim_aligned16(L) || !slim_aligned16(R) || !slim_aligned16(Lq) || !slim_aligned16(Ls) || !slim_aligned16(Rq) ||
      !slim_aligned16(Rs))
    return SLIM_EALIGN;
  hipStream_t s = (hipStream_t)stream;
  int* d_status = nullptr;
  if (hipMalloc(&d_status, sizeof(int)) != hipSuccess) return SLIM_EDEVICE;
  int h_status = 0;
  int rc = SLIM_OK;
  do {
    if (hipMemsetAsync(d_status, 0, sizeof(int), s) != hipSuccess) { rc = SLIM_EDEVICE; break; }
    // L^T [r, K]: element (j, k) = L[k * r + j]; R^T [N, r]: element (n, j) = R[j * N + n]
    const int64_t tl = r * ((K + 127) / 128) * 16, tr = N * ((r + 127) / 128) * 16;
    {
      SlimKernelTimer timer("pack_adapter_q", s);
      SLIM_LAUNCH(timer, k_pack_adapter_q, dim3((unsigned)((tl + 255) / 256)), dim3(256), s, L, r, r, K,
                  reinterpret_cast<uint32_t*>(Lq), Ls, d_status);
    }
    {
      SlimKernelTimer timer("pack_adapter_q", s);
      SLIM_LAUNCH(timer, k_pack_adapter_q, dim3((unsigned)((tr + 255) / 256)), dim3(256), s, R, N, N, r,
                  reinterpret_cast<uint32_t*>(Rq), Rs, d_status);
    }
    if (hipGetLastError() != hipSuccess) { rc = SLIM_EDEVICE; break; }
    if (hipMemcpyAsync(&h_status, d_status, sizeof(int), hipMemcpyDeviceToHost, s) != hipSuccess ||
        hipStreamSynchronize(s) != hipSuccess) { rc = SLIM_EDEVICE; break; }
    if (h_status & 1) rc = SLIM_ENONFINITE;
  } while (0);
  (void)hipFree(d_status);
  return rc;
}

extern "C" int slim_pack_adapter(const uint16_t* L, const uint16_t* R, int64_t K, int64_t N, int64_t r, uint16_t* Lt,
                                 uint16_t* Rt, void* stream) {
  if (!L || !R || !Lt || !Rt) return SLIM_EINVAL;
  if (K < 1 || N < 1 || r < 16 || r % 16 || K >= (int64_t(1) << 31) || N >= (int64_t(1) << 31) || r >= 65536)
    return SLIM_ESHAPE;
  if (!slim_aligned16(L) || !slim_aligned16(R) || !slim_aligned16(Lt) || !slim_aligned16(Rt)) return SLIM_EALIGN;
  hipStream_t s = (hipStream_t)stream;
  {
    SlimKernelTimer timer("pack_adapter", s);
    SLIM_LAUNCH(timer, k_transpose16, dim3((unsigned)((r + 63) / 64), (unsigned)((K + 63) / 64)), dim3(256), s, L, K, r,
                Lt);
  }
  {
    SlimKernelTimer timer("pack_adapter", s);
    const int64_t total = (N + 31) / 32 * 32 * r;
    SLIM_LAUNCH(timer, k_tile_rt, dim3((unsigned)((total + 255) / 256)), dim3(256), s, R, r, N, Rt);
  }
  return hipGetLastError() == hipSuccess ? SLIM_OK : SLIM_EDEVICE;
}

namespace {

int pack_forward(const float* W, int64_t N, int64_t K, uint8_t* codes, uint8_t* meta, uint16_t* scales,
                 uint8_t* mask, const double* alpha, void* stream) {
  int st = slim_check_pack(W, N, K, codes, meta, scales, mask);
  if (st != SLIM_OK) return st;
  hipStream_t s = (hipStream_t)stream;
  int* d_status = nullptr;
  if (hipMalloc(&d_status, sizeof(int)) != hipSuccess) return SLIM_EDEVICE;
  int h_status = 0;
  int rc = SLIM_OK;
  const int64_t total4 = N * (K / 4);
  const int64_t blocks = (total4 + kPackThreads - 1) / kPackThreads;
  do {
    if (hipMemsetAsync(d_status, 0, sizeof(int), s) != hipSuccess) { rc = SLIM_EDEVICE; break; }
    {
      SlimKernelTimer timer("pack", s);
      SLIM_LAUNCH(timer, k_pack, dim3((unsigned)blocks), dim3(kPackThreads), s, reinterpret_cast<const float4*>(W),
                  total4, K, reinterpret_cast<uint32_t*>(codes), reinterpret_cast<uint16_t*>(meta), scales,
                  reinterpret_cast<uint32_t*>(mask), d_status, alpha);
    }
    if (hipGetLastError() != hipSuccess) { rc = SLIM_EDEVICE; break; }
    if (hipMemcpyAsync(&h_status, d_status, sizeof(int), hipMemcpyDeviceToHost, s) != hipSuccess ||
        hipStreamSynchronize(s) != hipSuccess) { rc = SLIM_EDEVICE; break; }
    if (h_status & 1) rc = SLIM_ENONFINITE;
    else if (h_status & 2) rc = SLIM_ERANGE;
  } while (0);
  (void)hipFree(d_status);
  return rc;
}

}  // namespace

extern "C" int slim_pack(const float* W, int64_t N, int64_t K, uint8_t* codes, uint8_t* meta,
                         uint16_t* scales, uint8_t* mask, void* stream) {
  return pack_forward(W, N, K, codes, meta, scales, mask, nullptr, stream);
}

extern "C" int slim_pack_alpha(const float* W, int64_t N, int64_t K, const double* alpha, uint8_t* codes,
                               uint8_t* meta, uint16_t* scales, uint8_t* mask, void* stream) {
  if (!alpha) return SLIM_EINVAL;
  if ((uintptr_t)alpha & 7u) return SLIM_EALIGN;
  return pack_forward(W, N, K, codes, meta, scales, mask, alpha, stream);
}

extern "C" int slim_pack_bwd(const uint8_t* codes, const uint8_t* meta, const uint16_t* scales, int64_t N,
                             int64_t K, uint8_t* codesT, uint8_t* metaT, uint16_t* scalesT, uint8_t* mask_rc,
                             void* stream) {
  int st = slim_check_pack_bwd(codes, meta, scales, N, K, codesT, metaT, scalesT, mask_rc);
  if (st != SLIM_OK) return st;
  hipStream_t s = (hipStream_t)stream;
  int* d_status = nullptr;
  if (hipMalloc(&d_status, sizeof(int)) != hipSuccess) return SLIM_EDEVICE;
  int h_status = 0;
  int rc = SLIM_OK;
  do {
    if (hipMemsetAsync(d_status, 0, sizeof(int), s) != hipSuccess) { rc = SLIM_EDEVICE; break; }
    {
      dim3 grid((unsigned)(K / kBT), (unsigned)((N + kBT - 1) / kBT));
      SlimKernelTimer timer("pack_bwd", s);
      SLIM_LAUNCH(timer, k_pack_bwd, grid, dim3(256), s, reinterpret_cast<const uint32_t*>(codes),
                  reinterpret_cast<const uint16_t*>(meta), scales, N, K, reinterpret_cast<uint32_t*>(codesT),
                  reinterpret_cast<uint16_t*>(metaT), scalesT, mask_rc, d_status);
    }
    if (hipGetLastError() != hipSuccess) { rc = SLIM_EDEVICE; break; }
    if (hipMemcpyAsync(&h_status, d_status, sizeof(int), hipMemcpyDeviceToHost, s) != hipSuccess ||
        hipStreamSynchronize(s) != hipSuccess) { rc = SLIM_EDEVICE; break; }
    if (h_status & 2) rc = SLIM_ERANGE;
  } while (0);
  (void)hipFree(d_status);
  return rc;
}
