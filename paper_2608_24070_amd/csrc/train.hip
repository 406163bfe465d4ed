// train.hip - the steps of SLoPe's sparse training step that follow the input gradient, on
// half-precision value packs (SLoPe, Alg. "Accelerated Sparse Pretraining Algorithm for a Linear
// Layer"; appendix "Implementation details"):
//
//   slim_pack16        setup of W^R: 2:4 magnitude mask along K, kept values in fp16
//   slim_pack16_t      W^{R,C} along N for each k (double pruning of the value pack)
//   slim_grad_w        grad W = dY^T X (eq. sparse_backward_weight) at the positions M^R keeps,
//                      compressed to [N, K/2] in the epilogue (prune-and-compress fused)
//   slim_sparse_add    beta A + gamma B on compressed values with one shared pattern
//   slim_update_pack16 the optimizer's new compressed values into the forward pack
//
// Value packs are row-major: vals fp16 [rows, len/2] (group g of a row at 2g, 2g + 1, lower kept
// position first) and meta uint8 [rows, len/8] in the inference pack's index format (half-word b
// covers positions 16b .. 16b + 15; group c of it holds i0 in bits 4c..4c+1, i1 in 4c+2..4c+3).
#include <type_traits>

#include "slim_device.h"
#include "slim_host.h"
#include "slim_timing.h"

namespace {

typedef __bf16 bf8_t __attribute__((ext_vector_type(8)));

// ------------------------------------------------------------------------------- pack16
// One thread per 16 positions (four groups) of a row: top two of each group by (|w| desc,
// position asc), the kept values rounded to fp16 (nearest, ties to even).
__global__ void __launch_bounds__(256)
k_pack16(const float4* __restrict__ W, int64_t n16, u32x4_t* __restrict__ vals, uint16_t* __restrict__ meta,
         u32x4_t* __restrict__ mask, int* __restrict__ status) {
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (t >= n16) return;
  uint32_t mw = 0, mk[4] = {0u, 0u, 0u, 0u};
  uint32_t hv[4];
  int bad = 0;
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    const float4 v = W[4 * t + c];
    const float w[4] = {v.x, v.y, v.z, v.w};
    float a[4];
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      a[p] = fabsf(w[p]);
      if (!__builtin_isfinite(w[p])) bad = 1;
    }
    int i0 = -1, i1 = -1;
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      int rank = 0;
#pragma unroll
      for (int q = 0; q < 4; ++q)
        if (q != p && (a[q] > a[p] || (a[q] == a[p] && q < p))) ++rank;
      if (rank < 2) {
        if (i0 < 0) i0 = p;
        else i1 = p;
        mk[c] |= 1u << (8 * p);
      }
    }
    const h2_t kv = {(_Float16)w[i0], (_Float16)w[i1]};
    hv[c] = bits_of(kv);
    mw |= (uint32_t)(i0 | (i1 << 2)) << (4 * c);
  }
  if (bad) atomicOr(status, 1);
  vals[t] = u32x4_t{hv[0], hv[1], hv[2], hv[3]};
  meta[t] = (uint16_t)mw;
  if (mask) mask[t] = u32x4_t{mk[0], mk[1], mk[2], mk[3]};
}

// ----------------------------------------------------------------------------- pack16_t
// Block = 64 rows (n) x 64 columns (k). Phase 1 expands the value pack of the tile into LDS (fp16
// bits, 0 where M^R drops, and the M^R bit); phase 2 gives each thread one column k and one
// 16-row block, keeps the top two of each aligned 4-row group by (|v| desc, M^R bit desc, n asc)
// and writes 8 values (16 B) of valsT and one metaT half-word.
constexpr int kTT = 64;

__global__ void __launch_bounds__(256)
k_pack16_t(const uint16_t* __restrict__ vals, const uint8_t* __restrict__ meta, int64_t N, int64_t K,
           u32x4_t* __restrict__ valsT, uint16_t* __restrict__ metaT) {
  __shared__ uint16_t v_s[kTT][kTT + 2];
  __shared__ uint8_t f_s[kTT][kTT + 4];
  const int tid = threadIdx.x;
  const int64_t k0 = (int64_t)blockIdx.x * kTT, n0 = (int64_t)blockIdx.y * kTT;
  {
    // thread -> (row tid / 4, 16 columns 16 (tid % 4)): four groups
    const int row = tid >> 2, w = tid & 3;
    const int64_t n = n0 + row;
    const int64_t kc = k0 + 16 * w;                        // first column of the 16
    const uint16_t mw = *reinterpret_cast<const uint16_t*>(meta + n * (K / 8) + kc / 8);
    const u32x4_t v8 = *reinterpret_cast<const u32x4_t*>(vals + n * (K / 2) + kc / 2);
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int i0 = (mw >> (4 * c)) & 3, i1 = (mw >> (4 * c + 2)) & 3;
#pragma unroll
      for (int p = 0; p < 4; ++p) {
        const int col = 16 * w + 4 * c + p;
        const uint32_t pr = v8[c];
        v_s[row][col] = p == i0 ? (uint16_t)(pr & 0xFFFFu) : (p == i1 ? (uint16_t)(pr >> 16) : (uint16_t)0);
        f_s[row][col] = (p == i0 || p == i1) ? 1 : 0;
      }
    }
  }
  __syncthreads();
  // thread -> (column tid % 64, 16-row block tid / 64)
  const int col = tid & 63, blk = tid >> 6;
  uint32_t hv[4], mw = 0;
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    const int r0 = 16 * blk + 4 * c;
    uint32_t mag[4], f[4], bits[4];
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      bits[p] = v_s[r0 + p][col];
      mag[p] = bits[p] & 0x7FFFu;          // fp16 magnitude order (finite values)
      f[p] = f_s[r0 + p][col];
    }
    int i0 = -1, i1 = -1;
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      int rank = 0;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const bool before = mag[q] > mag[p] || (mag[q] == mag[p] && (f[q] > f[p] || (f[q] == f[p] && q < p)));
        if (q != p && before) ++rank;
      }
      if (rank < 2) {
        if (i0 < 0) i0 = p;
        else i1 = p;
      }
    }
    hv[c] = bits[i0] | (bits[i1] << 16);
    mw |= (uint32_t)(i0 | (i1 << 2)) << (4 * c);
  }
  const int64_t k = k0 + col, nb = n0 / 16 + blk;       // 16-row block along n
  valsT[k * (N / 16) + nb] = u32x4_t{hv[0], hv[1], hv[2], hv[3]};
  metaT[k * (N / 16) + nb] = (uint16_t)mw;
}

// ------------------------------------------------------------------------------- grad_w
// D[k][n] = sum_m X[m][k] dY[m][n] (= grad W^T) on 32x32x16 MFMA, fp32 accumulate; tile 256 (k) x
// 256 (n) for 8 waves, two per SIMD: wave (wk, wn) owns k rows 128 wk .. + 127 and n columns
// 64 wn .. + 63 (4 x 2 fragments in the accumulation registers). The tile's operand traffic per
// flop is a quarter of a 128 x 128 tile's (every dY column slab is read by K/256 tiles, every X
// slab by N/256). Both operands are [M, *] row-major, so the reduction runs along their rows: per
// 64-row chunk, each thread loads eight rows of four columns of each (8 B per load; rows past M read
// as zero through the buffer resource) and writes them to LDS transposed, eight reduction positions
// per 16-byte write, into [column][64 + 8] fp16 rows with XOR-swizzled 16-byte slots. Loads run one
// chunk ahead in registers (the SIMD's other wave covers the rest of the latency); LDS has two stages.
// Columns past N or K (a last partial tile) read neighbouring data; D entries of such a column are
// never stored, and no other entry depends on it.
// Epilogue: a fragment row block 8q + 4 (L / 32) .. + 3 of lane L is one aligned 4-group of k for
// column n = L % 32, so the two positions M^R keeps (one metadata nibble) are selected in
// registers and stored as the compressed pair gW[n][2g], gW[n][2g + 1].
constexpr int kGT = 256, kGM = 64, kGLd = kGM + 8, kGThreads = 512;

template <bool BF16>
SLIM_DEV f16_t mfma_acc(u32x4_t a, u32x4_t b, f16_t c) {
  if constexpr (BF16)
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf8_t, a), __builtin_bit_cast(bf8_t, b), c, 0, 0, 0);
  else
    return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(h8_t, a), __builtin_bit_cast(h8_t, b), c, 0, 0, 0);
}

SLIM_DEV float sel4(const f16_t& acc, int base, int i) {
  const float a0 = acc[base], a1 = acc[base + 1], a2 = acc[base + 2], a3 = acc[base + 3];
  return i == 0 ? a0 : (i == 1 ? a1 : (i == 2 ? a2 : a3));
}

struct GradRegs {
  u32x2_t y[8], x[8];   // [row]: four columns of one row
};

template <bool BF16>
__global__ void __launch_bounds__(kGThreads)
k_grad_w(const uint16_t* __restrict__ dY, const uint16_t* __restrict__ X, int64_t M, int64_t N, int64_t K,
         const uint8_t* __restrict__ meta, float* __restrict__ gW) {
  __shared__ __attribute__((aligned(16))) uint16_t xs[2][kGT][kGLd];   // [stage][k][m]
  __shared__ __attribute__((aligned(16))) uint16_t ys[2][kGT][kGLd];   // [stage][n][m]
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wk = wave & 1, wn = wave >> 1, h = lane >> 5;
  // XCD-aware tile order (block b runs on XCD b % 8, which takes positions [x Q, (x + 1) Q) of an
  // order walking bands of four n tiles k tile by k tile), so blocks running together on one XCD
  // share dY and X chunks in its L2
  const int64_t tn = (N + kGT - 1) / kGT, tk = (K + kGT - 1) / kGT, T = tn * tk;
  const int64_t Q = (T + 7) / 8;
  const int64_t pos = (int64_t)(blockIdx.x % 8) * Q + blockIdx.x / 8;
  if (pos >= T) return;
  const int64_t band = pos / (4 * tk), q0 = pos - band * 4 * tk;
  const int64_t nbw = tn - band * 4 < 4 ? tn - band * 4 : 4;
  const int64_t n0 = (band * 4 + q0 % nbw) * kGT, k0 = (q0 / nbw) * kGT;

  // loads: thread -> columns 4 cg .. 4 cg + 3 of the tile (cg = tid % 64) and rows 8 mg .. 8 mg + 7
  // of the chunk (mg = tid / 64, the wave), so that one load instruction of a wave reads one row's
  // 512 contiguous bytes; all of the offset is per lane, so the resource's extent check sees the row
  const int cg = tid & 63, mg = tid >> 6;
  const rsrc_t ry = make_rsrc(dY, M * N * 2), rx = make_rsrc(X, M * K * 2);
  const uint32_t yo = ((uint32_t)(8 * mg) * (uint32_t)N + (uint32_t)(n0 + 4 * cg)) * 2u;
  const uint32_t xo = ((uint32_t)(8 * mg) * (uint32_t)K + (uint32_t)(k0 + 4 * cg)) * 2u;
  const uint32_t ystep = (uint32_t)kGM * (uint32_t)N * 2u, xstep = (uint32_t)kGM * (uint32_t)K * 2u;
  auto load = [&](int64_t c, GradRegs& R) {
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      R.y[j] = __builtin_bit_cast(u32x2_t, __builtin_amdgcn_raw_buffer_load_b64(
                   ry, yo + (uint32_t)c * ystep + (uint32_t)j * (uint32_t)N * 2u, 0, 0));
      R.x[j] = __builtin_bit_cast(u32x2_t, __builtin_amdgcn_raw_buffer_load_b64(
                   rx, xo + (uint32_t)c * xstep + (uint32_t)j * (uint32_t)K * 2u, 0, 0));
    }
  };
  // LDS rows (144 bytes) hold the chunk's 64 reduction positions as eight 16-byte slots and 16
  // bytes of padding; slot s of tile column row r sits at physical slot s ^ ((r / 8) % 8). Eight
  // lanes of a wave's 16-byte transposed writes (rows 4 apart, one slot) and eight of its 16-byte
  // fragment reads (consecutive rows, one slot) then fall in distinct 16-byte bank groups.
  auto slot_of = [](int r, int s) { return s ^ ((r >> 3) & 7); };
  // 8 x 4 transposes of 16-bit elements: column c of the thread's four gets the 8 rows (positions
  // 8 mg .. 8 mg + 7, slot mg) as one 16-byte LDS write
  auto store = [&](const GradRegs& R, int stg) {
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int w = c >> 1, sh = 16 * (c & 1);
      auto pick = [&](const u32x2_t* r, int j) { return (r[j][w] >> sh) & 0xFFFFu; };
      u32x4_t yv, xv;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        yv[i] = pick(R.y, 2 * i) | (pick(R.y, 2 * i + 1) << 16);
        xv[i] = pick(R.x, 2 * i) | (pick(R.x, 2 * i + 1) << 16);
      }
      const int r = 4 * cg + c;
      *reinterpret_cast<u32x4_t*>(&ys[stg][r][8 * slot_of(r, mg)]) = yv;
      *reinterpret_cast<u32x4_t*>(&xs[stg][r][8 * slot_of(r, mg)]) = xv;
    }
  };

  f16_t acc[4][2];
#pragma unroll
  for (int x = 0; x < 4; ++x)
#pragma unroll
    for (int y = 0; y < 2; ++y)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[x][y][v] = 0.f;

  // per step (16 positions) the wave reads 4 A and 2 B fragments, then issues their 8 MFMAs (the
  // SIMD's other wave covers the LDS latency)
  auto compute = [&](int stg) {
#pragma unroll
    for (int st = 0; st < kGM / 16; ++st) {
      u32x4_t af[4], bf[2];
#pragma unroll
      for (int f = 0; f < 4; ++f) {
        const int ra = 128 * wk + 32 * f + (lane & 31);
        af[f] = *reinterpret_cast<const u32x4_t*>(&xs[stg][ra][8 * slot_of(ra, 2 * st + h)]);
      }
#pragma unroll
      for (int f = 0; f < 2; ++f) {
        const int rb = 64 * wn + 32 * f + (lane & 31);
        bf[f] = *reinterpret_cast<const u32x4_t*>(&ys[stg][rb][8 * slot_of(rb, 2 * st + h)]);
      }
#pragma unroll
      for (int x = 0; x < 4; ++x)
#pragma unroll
        for (int y = 0; y < 2; ++y) acc[x][y] = mfma_acc<BF16>(af[x], bf[y], acc[x][y]);
    }
  };

  // chunk c: loads of chunk c + 1 into registers, this chunk's MFMAs from stage c % 2, then the
  // registers into the other stage (last read during chunk c - 1, before the barrier that ended
  // it). Loads past the last chunk address rows past M and read as zero.
  const int64_t nch = (M + kGM - 1) / kGM;
  GradRegs r0;
  load(0, r0);
  store(r0, 0);
  __syncthreads();
  auto chunk = [&](int64_t c, int stg) {
    load(c + 1, r0);
    __builtin_amdgcn_sched_barrier(0);   // issued before this chunk's work, not sunk into it
    compute(stg);
    store(r0, stg ^ 1);
    __syncthreads();
  };
  int64_t c = 0;
  for (; c + 2 <= nch; c += 2) {
    chunk(c, 0);
    chunk(c + 1, 1);
  }
  if (c < nch) chunk(c, 0);

  // D[i][j] of a 32x32 fragment: lane j + 32 ((i / 4) % 2), element 4 (i / 8) + i % 4
#pragma unroll
  for (int y = 0; y < 2; ++y) {
    const int64_t n = n0 + 64 * wn + 32 * y + (lane & 31);
    if (n >= N) continue;
#pragma unroll
    for (int x = 0; x < 4; ++x) {
      const int64_t kb = k0 + 128 * wk + 32 * x;                 // first row of the fragment
      if (kb >= K) continue;
      const int64_t gb = kb / 4;
      const uint32_t md = *reinterpret_cast<const uint32_t*>(meta + n * (K / 8) + gb / 2);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int t = 2 * q + h;                                // group gb + t holds rows 8q + 4h ..
        const uint32_t nib = (md >> (4 * t)) & 0xFu;
        const float v0 = sel4(acc[x][y], 4 * q, (int)(nib & 3u)), v1 = sel4(acc[x][y], 4 * q, (int)(nib >> 2));
        *reinterpret_cast<u32x2_t*>(gW + n * (K / 2) + 2 * (gb + t)) =
            u32x2_t{__builtin_bit_cast(uint32_t, v0), __builtin_bit_cast(uint32_t, v1)};
      }
    }
  }
}

// ------------------------------------------------------------------ sparse add and update
// out = beta A + gamma B elementwise (fp32: beta A rounded, then fused with gamma B); four
// elements per thread.
__global__ void __launch_bounds__(256)
k_sparse_add(const f4_t* __restrict__ A, const u32x2_t* __restrict__ Bv, float beta, float gamma,
             f4_t* __restrict__ out, int64_t n4) {
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (t >= n4) return;
  const f4_t a = A[t];
  const u32x2_t b = Bv[t];
  const float bf[4] = {h_bits_to_f(b[0] & 0xFFFFu), h_bits_to_f(b[0] >> 16), h_bits_to_f(b[1] & 0xFFFFu),
                       h_bits_to_f(b[1] >> 16)};
  f4_t o;
#pragma unroll
  for (int e = 0; e < 4; ++e) o[e] = fmaf(gamma, bf[e], beta * a[e]);
  out[t] = o;
}

// vals = fp16(Wnew) (nearest, ties to even), four elements per thread.
__global__ void __launch_bounds__(256)
k_update16(const f4_t* __restrict__ Wn, u32x2_t* __restrict__ vals, int64_t n4) {
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (t >= n4) return;
  const f4_t w = Wn[t];
  const h2_t lo = {(_Float16)w[0], (_Float16)w[1]}, hi = {(_Float16)w[2], (_Float16)w[3]};
  vals[t] = u32x2_t{bits_of(lo), bits_of(hi)};
}

}  // namespace

extern "C" int slim_pack16(const float* W, int64_t N, int64_t K, uint16_t* vals, uint8_t* meta, uint8_t* mask,
                           void* stream) {
  if (!W || !vals || !meta) return SLIM_EINVAL;
  if (N < 1 || K < 16 || K % 16 || N >= (int64_t(1) << 24) || K >= (int64_t(1) << 24)) return SLIM_ESHAPE;
  if (!slim_aligned16(W) || !slim_aligned16(vals) || !slim_aligned16(meta) || (mask && !slim_aligned16(mask)))
    return SLIM_EALIGN;
  hipStream_t s = (hipStream_t)stream;
  int* d_status = nullptr;
  if (hipMalloc(&d_status, sizeof(int)) != hipSuccess) return SLIM_EDEVICE;
  int h_status = 0, rc = SLIM_OK;
  const int64_t n16 = N * (K / 16);
  do {
    if (hipMemsetAsync(d_status, 0, sizeof(int), s) != hipSuccess) { rc = SLIM_EDEVICE; break; }
    {
      SlimKernelTimer timer("pack16", s);
      SLIM_LAUNCH(timer, k_pack16, dim3((unsigned)((n16 + 255) / 256)), dim3(256), s,
                  reinterpret_cast<const float4*>(W), n16, reinterpret_cast<u32x4_t*>(vals),
                  reinterpret_cast<uint16_t*>(meta), reinterpret_cast<u32x4_t*>(mask), d_status);
    }
    if (hipGetLastError() != hipSuccess) { rc = SLIM_EDEVICE; break; }
    if (hipMemcpyAsync(&h_status, d_status, sizeof(int), hipMemcpyDeviceToHost, s) != hipSuccess ||
        hipStreamSynchronize(s) != hipSuccess) { rc = SLIM_EDEVICE; break; }
    if (h_status & 1) rc = SLIM_ENONFINITE;
  } while (0);
  (void)hipFree(d_status);
  return rc;
}

extern "C" int slim_pack16_t(const uint16_t* vals, const uint8_t* meta, int64_t N, int64_t K, uint16_t* valsT,
                             uint8_t* metaT, void* stream) {
  if (!vals || !meta || !valsT || !metaT) return SLIM_EINVAL;
  if (N < 64 || K < 64 || N % 64 || K % 64 || N >= (int64_t(1) << 24) || K >= (int64_t(1) << 24)) return SLIM_ESHAPE;
  if (!slim_aligned16(vals) || !slim_aligned16(meta) || !slim_aligned16(valsT) || !slim_aligned16(metaT))
    return SLIM_EALIGN;
  hipStream_t s = (hipStream_t)stream;
  SlimKernelTimer timer("pack16_t", s);
  SLIM_LAUNCH(timer, k_pack16_t, dim3((unsigned)(K / kTT), (unsigned)(N / kTT)), dim3(256), s, vals, meta, N, K,
              reinterpret_cast<u32x4_t*>(valsT), reinterpret_cast<uint16_t*>(metaT));
  return hipGetLastError() == hipSuccess ? SLIM_OK : SLIM_EDEVICE;
}

extern "C" int slim_grad_w(const void* dY, const void* X, int dtype, int64_t M, int64_t N, int64_t K,
                           const uint8_t* meta, float* gW, void* stream) {
  if (!dY || !X || !meta || !gW) return SLIM_EINVAL;
  if (dtype != SLIM_F16 && dtype != SLIM_BF16) return SLIM_EDTYPE;
  if (M < 1 || N < 128 || K < 128 || N % 128 || K % 128) return SLIM_ESHAPE;
  // per-lane byte offsets are 32-bit: the operands must stay below 4 GiB
  if (M * N * 2 >= (int64_t(1) << 32) || M * K * 2 >= (int64_t(1) << 32) || N >= (int64_t(1) << 24) ||
      K >= (int64_t(1) << 24))
    return SLIM_EUNSUPPORTED;
  if (!slim_aligned16(dY) || !slim_aligned16(X) || !slim_aligned16(meta) || !slim_aligned16(gW)) return SLIM_EALIGN;
  hipStream_t s = (hipStream_t)stream;
  const int64_t T = ((N + kGT - 1) / kGT) * ((K + kGT - 1) / kGT);
  const dim3 grid((unsigned)(8 * ((T + 7) / 8)));
  SlimKernelTimer timer("grad_w", s);
  if (dtype == SLIM_BF16)
    SLIM_LAUNCH(timer, k_grad_w<true>, grid, dim3(kGThreads), s, reinterpret_cast<const uint16_t*>(dY),
                reinterpret_cast<const uint16_t*>(X), M, N, K, meta, gW);
  else
    SLIM_LAUNCH(timer, k_grad_w<false>, grid, dim3(kGThreads), s, reinterpret_cast<const uint16_t*>(dY),
                reinterpret_cast<const uint16_t*>(X), M, N, K, meta, gW);
  return hipGetLastError() == hipSuccess ? SLIM_OK : SLIM_EDEVICE;
}

extern "C" int slim_sparse_add(const float* A, const uint16_t* B, float beta, float gamma, float* out, int64_t count,
                               void* stream) {
  if (!A || !B || !out) return SLIM_EINVAL;
  if (count < 0 || count % 8) return SLIM_ESHAPE;
  if (!slim_aligned16(A) || !slim_aligned16(B) || !slim_aligned16(out)) return SLIM_EALIGN;
  if (count == 0) return SLIM_OK;
  hipStream_t s = (hipStream_t)stream;
  const int64_t n4 = count / 4;
  SlimKernelTimer timer("sparse_add", s);
  SLIM_LAUNCH(timer, k_sparse_add, dim3((unsigned)((n4 + 255) / 256)), dim3(256), s,
              reinterpret_cast<const f4_t*>(A), reinterpret_cast<const u32x2_t*>(B), beta, gamma,
              reinterpret_cast<f4_t*>(out), n4);
  return hipGetLastError() == hipSuccess ? SLIM_OK : SLIM_EDEVICE;
}

extern "C" int slim_update_pack16(const float* Wnew, int64_t count, uint16_t* vals, void* stream) {
  if (!Wnew || !vals) return SLIM_EINVAL;
  if (count < 0 || count % 8) return SLIM_ESHAPE;
  if (!slim_aligned16(Wnew) || !slim_aligned16(vals)) return SLIM_EALIGN;
  if (count == 0) return SLIM_OK;
  hipStream_t s = (hipStream_t)stream;
  const int64_t n4 = count / 4;
  SlimKernelTimer timer("update16", s);
  SLIM_LAUNCH(timer, k_update16, dim3((unsigned)((n4 + 255) / 256)), dim3(256), s,
              reinterpret_cast<const f4_t*>(Wnew), reinterpret_cast<u32x2_t*>(vals), n4);
  return hipGetLastError() == hipSuccess ? SLIM_OK : SLIM_EDEVICE;
}
