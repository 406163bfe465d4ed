// hybrid.hip - PATCH's hybrid dense / 2:4 tile layer (PATCH chapter, "Efficient deployment of
// PATCH"; appendix "STOICC Integration"): a weight whose 128 x 128 tiles are either dense fp16 or
// 2:4-sparse fp16, multiplied in one GEMM, Y = X Wp^T.
//
//   k_hybrid_pack    one thread per 16 positions of a row: the tile's payload, dense (fp16 values)
//                    or compressed (the two largest of each group of four as fp16, lower position
//                    first, and one index half-word per 16 positions), at the offset the host
//                    computed from the tile map
//   k_hybrid_gemm    128 x 128 output tiles of Y^T (rows n, columns m); a chunk of 128 along K is
//                    one weight tile, dense (v_mfma_f32_32x32x16_f16) or sparse
//                    (v_smfmac_f32_32x32x32_f16, half the MFMA issue for the same K); both write
//                    the same 32 x 32 accumulator layout, so a tile row may mix them freely
//   k_hybrid_reduce  the split partials of small-M calls, summed in split order
#include <new>

#include "slim_device.h"
#include "slim_host.h"
#include "slim_timing.h"

namespace {

constexpr int kHT = 128;                        // weight tile edge
constexpr int kHDense = kHT * kHT * 2;          // bytes of a dense tile
constexpr int kHSparse = kHT * kHT + kHT * kHT / 8;
constexpr uint64_t kHSparseBit = 1ull << 63;
constexpr int kHThreads = 256;

// ------------------------------------------------------------------------------------- pack
__global__ void __launch_bounds__(kHThreads)
k_hybrid_pack(const float* __restrict__ W, int64_t N, int64_t K, const uint64_t* __restrict__ info,
              uint8_t* __restrict__ payload, int* __restrict__ status) {
  const int64_t t = (int64_t)blockIdx.x * kHThreads + threadIdx.x;
  const int64_t per_row = K / 16;
  if (t >= N * per_row) return;
  const int64_t n = t / per_row, j = t % per_row;
  const int64_t tk = (16 * j) / kHT, tkn = K / kHT;
  const uint64_t ti = info[(n / kHT) * tkn + tk];
  const uint64_t off = ti & ~kHSparseBit;
  const int r = (int)(n % kHT), kk = (int)((16 * j) % kHT);
  const float4* src = reinterpret_cast<const float4*>(W + n * K + 16 * j);
  float w[16];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const float4 v = src[q];
    w[4 * q] = v.x;
    w[4 * q + 1] = v.y;
    w[4 * q + 2] = v.z;
    w[4 * q + 3] = v.w;
  }
  int bad = 0;
#pragma unroll
  for (int p = 0; p < 16; ++p)
    if (!__builtin_isfinite(w[p])) bad = 1;
  if (bad) atomicOr(status, 1);
  if (!(ti & kHSparseBit)) {
    h8_t lo, hi;
#pragma unroll
    for (int p = 0; p < 8; ++p) {
      lo[p] = (_Float16)w[p];
      hi[p] = (_Float16)w[8 + p];
    }
    u32x4_t* dst = reinterpret_cast<u32x4_t*>(payload + off + (uint64_t)r * 256 + 2 * kk);
    dst[0] = __builtin_bit_cast(u32x4_t, lo);
    dst[1] = __builtin_bit_cast(u32x4_t, hi);
    return;
  }
  h8_t vals;
  uint32_t half = 0;
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    float a[4];
#pragma unroll
    for (int p = 0; p < 4; ++p) a[p] = fabsf(w[4 * c + p]);
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
      }
    }
    vals[2 * c] = (_Float16)w[4 * c + i0];
    vals[2 * c + 1] = (_Float16)w[4 * c + i1];
    half |= (uint32_t)(i0 | (i1 << 2)) << (4 * c);
  }
  *reinterpret_cast<u32x4_t*>(payload + off + (uint64_t)r * 128 + kk) = __builtin_bit_cast(u32x4_t, vals);
  *reinterpret_cast<uint16_t*>(payload + off + kHT * kHT + (uint64_t)r * 16 + 2 * (kk / 16)) = (uint16_t)half;
}

// ------------------------------------------------------------------------------------- GEMM
// LDS row of the X chunk: 128 fp16 = 16 slots of 16 bytes, slot s of row m at s ^ (m % 8), so that
// the B-operand reads of 8 consecutive rows at one slot fall in distinct banks.
__device__ __forceinline__ int xs_off(int row, int slot) { return row * 256 + ((slot ^ (row & 7)) << 4); }

struct HybridArgs {
  const uint16_t* X;
  const uint64_t* info;
  const uint8_t* payload;
  float* out;          // Y [M, N] (one split) or partials [split][M][N]
  int64_t M, N, K;
  int chunks_per_split;
};

// Operands of one chunk for one wave: 16 x 16 bytes of values (dense: 8 steps x 2 row fragments;
// sparse: 4 steps x 2 fragments) and, for a sparse chunk, each fragment's four index half-words of
// this lane's group (8 bytes).
struct ChunkRegs {
  u32x4_t a[16];
  u32x2_t m[2];
  bool sparse;
};

// One block per CU: the next chunk's operands (weights in registers, X on its way to LDS) are held
// while the current chunk's MFMAs run, next to the 64 accumulators.
__global__ void __launch_bounds__(kHThreads, 1)
k_hybrid_gemm(HybridArgs g) {
  __shared__ __attribute__((aligned(16))) uint8_t xs[2][kHT * 256];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wn = wave >> 1, wm = wave & 1;
  const int l32 = lane & 31, h = lane >> 5;
  const int64_t tn = blockIdx.x, n0 = tn * kHT, m0 = (int64_t)blockIdx.y * kHT;
  const int64_t chunks = g.K / kHT;
  const int64_t c_begin = (int64_t)blockIdx.z * g.chunks_per_split;
  const int64_t c_end = c_begin + g.chunks_per_split < chunks ? c_begin + g.chunks_per_split : chunks;

  // X chunk staging: 8 pieces of 16 bytes per thread
  auto load_x = [&](int64_t c, u32x4_t (&v)[8]) {
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int p = tid + kHThreads * i, row = p >> 4, slot = p & 15;
      const int64_t m = m0 + row;
      v[i] = m < g.M ? *reinterpret_cast<const u32x4_t*>(g.X + m * g.K + c * kHT + 8 * slot) : u32x4_t{0, 0, 0, 0};
    }
  };
  auto store_x = [&](int stg, const u32x4_t (&v)[8]) {
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int p = tid + kHThreads * i, row = p >> 4, slot = p & 15;
      *reinterpret_cast<u32x4_t*>(&xs[stg][xs_off(row, slot)]) = v[i];
    }
  };
  // this wave's weight operands of chunk c
  auto load_w = [&](int64_t c, ChunkRegs& w) {
    const uint64_t ti = g.info[tn * chunks + c];
    const uint8_t* base = g.payload + (ti & ~kHSparseBit);
    w.sparse = (ti & kHSparseBit) != 0;
    if (!w.sparse) {
#pragma unroll
      for (int fn = 0; fn < 2; ++fn) {
        const int r = 64 * wn + 32 * fn + l32;
#pragma unroll
        for (int s = 0; s < 8; ++s)
          w.a[8 * fn + s] = *reinterpret_cast<const u32x4_t*>(base + r * 256 + 32 * s + 16 * h);
      }
    } else {
#pragma unroll
      for (int fn = 0; fn < 2; ++fn) {
        const int r = 64 * wn + 32 * fn + l32;
#pragma unroll
        for (int s = 0; s < 4; ++s)
          w.a[4 * fn + s] = *reinterpret_cast<const u32x4_t*>(base + r * 128 + 64 * h + 16 * s);
        // half-words 4 h .. 4 h + 3 of the row: lane group h covers positions 64 h .. 64 h + 63
        w.m[fn] = *reinterpret_cast<const u32x2_t*>(base + kHT * kHT + r * 16 + 8 * h);
      }
    }
  };

  f16_t acc[2][2];
#pragma unroll
  for (int fn = 0; fn < 2; ++fn)
#pragma unroll
    for (int fm = 0; fm < 2; ++fm)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[fn][fm][e] = 0.f;

  auto compute = [&](int stg, const ChunkRegs& w) {
    const uint8_t* x = xs[stg];
    if (!w.sparse) {
#pragma unroll
      for (int s = 0; s < 8; ++s) {
        h8_t b[2];
#pragma unroll
        for (int fm = 0; fm < 2; ++fm)
          b[fm] = __builtin_bit_cast(h8_t, *reinterpret_cast<const u32x4_t*>(&x[xs_off(64 * wm + 32 * fm + l32, 2 * s + h)]));
#pragma unroll
        for (int fn = 0; fn < 2; ++fn) {
          const h8_t a = __builtin_bit_cast(h8_t, w.a[8 * fn + s]);
#pragma unroll
          for (int fm = 0; fm < 2; ++fm) acc[fn][fm] = mfma32(a, b[fm], acc[fn][fm]);
        }
      }
    } else {
#pragma unroll
      for (int s = 0; s < 4; ++s) {
        h16_t b[2];
#pragma unroll
        for (int fm = 0; fm < 2; ++fm) {
          const int row = 64 * wm + 32 * fm + l32;
          const h8_t lo = __builtin_bit_cast(h8_t, *reinterpret_cast<const u32x4_t*>(&x[xs_off(row, 2 * s + h)]));
          const h8_t hi = __builtin_bit_cast(h8_t, *reinterpret_cast<const u32x4_t*>(&x[xs_off(row, 8 + 2 * s + h)]));
          b[fm] = cat16(lo, hi);
        }
#pragma unroll
        for (int fn = 0; fn < 2; ++fn) {
          const h8_t a = __builtin_bit_cast(h8_t, w.a[4 * fn + s]);
          const uint32_t word = w.m[fn][s >> 1];
          const int idx = (int)((s & 1) ? (word >> 16) : (word & 0xFFFFu));
#pragma unroll
          for (int fm = 0; fm < 2; ++fm) acc[fn][fm] = smfmac32(a, b[fm], acc[fn][fm], idx, 0);
        }
      }
    }
  };

  if (c_begin < c_end) {
    u32x4_t xv[8];
    ChunkRegs wc, wnx;
    load_x(c_begin, xv);
    load_w(c_begin, wc);
    store_x(0, xv);
    __syncthreads();
    int stg = 0;
    for (int64_t c = c_begin; c < c_end; ++c) {
      const bool more = c + 1 < c_end;
      if (more) {
        load_x(c + 1, xv);
        load_w(c + 1, wnx);
      }
      compute(stg, wc);
      if (more) store_x(stg ^ 1, xv);
      __syncthreads();
      stg ^= 1;
      if (more) wc = wnx;
    }
  }

  // D[i][j] of a 32x32 fragment: lane j + 32 ((i / 4) % 2), element 4 (i / 8) + i % 4
  float* out = g.out + (int64_t)blockIdx.z * g.M * g.N;
#pragma unroll
  for (int fm = 0; fm < 2; ++fm) {
    const int64_t m = m0 + 64 * wm + 32 * fm + l32;
    if (m >= g.M) continue;
#pragma unroll
    for (int fn = 0; fn < 2; ++fn)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int64_t nn = n0 + 64 * wn + 32 * fn + 8 * q + 4 * h;
        const f4_t o = {acc[fn][fm][4 * q], acc[fn][fm][4 * q + 1], acc[fn][fm][4 * q + 2], acc[fn][fm][4 * q + 3]};
        *reinterpret_cast<f4_t*>(out + m * g.N + nn) = o;
      }
  }
}

__global__ void __launch_bounds__(kHThreads)
k_hybrid_reduce(const float* __restrict__ part, int splits, int64_t count4, float* __restrict__ Y) {
  const int64_t i = (int64_t)blockIdx.x * kHThreads + threadIdx.x;
  if (i >= count4) return;
  const f4_t* p = reinterpret_cast<const f4_t*>(part);
  f4_t s = p[i];
  for (int z = 1; z < splits; ++z) s += p[(int64_t)z * count4 + i];
  reinterpret_cast<f4_t*>(Y)[i] = s;
}

struct HybridPlan {
  int64_t tiles, splits, chunks_per_split;
  size_t ws;
};

HybridPlan hybrid_plan(int64_t M, int64_t N, int64_t K) {
  HybridPlan p{};
  const int64_t chunks = K / kHT;
  p.tiles = (N / kHT) * ((M + kHT - 1) / kHT);
  int64_t s = 1;
  if (p.tiles < 256) s = (512 + p.tiles - 1) / p.tiles;          // at least ~512 blocks
  if (s > chunks) s = chunks;
  p.chunks_per_split = (chunks + s - 1) / s;
  p.splits = (chunks + p.chunks_per_split - 1) / p.chunks_per_split;
  p.ws = p.splits > 1 ? (size_t)p.splits * M * N * sizeof(float) : 0;
  return p;
}

}  // namespace

extern "C" int slim_hybrid_layout(const uint8_t* kinds, int64_t N, int64_t K, uint64_t* tile_info,
                                  size_t* payload_bytes) {
  if (!kinds || !payload_bytes) return SLIM_EINVAL;
  if (N < kHT || K < kHT || N % kHT || K % kHT) return SLIM_ESHAPE;
  const int64_t tiles = (N / kHT) * (K / kHT);
  uint64_t off = 0;
  for (int64_t t = 0; t < tiles; ++t) {
    if (kinds[t] > 1) return SLIM_EINVAL;
    if (tile_info) tile_info[t] = off | (kinds[t] ? kHSparseBit : 0);
    off += kinds[t] ? kHSparse : kHDense;
  }
  *payload_bytes = (size_t)off;
  return SLIM_OK;
}

extern "C" int slim_pack_hybrid(const float* W, int64_t N, int64_t K, const uint8_t* kinds, uint64_t* tile_info,
                                uint8_t* payload, size_t payload_bytes, void* stream) {
  if (!W || !kinds || !tile_info || !payload) return SLIM_EINVAL;
  size_t need = 0;
  int st = slim_hybrid_layout(kinds, N, K, nullptr, &need);
  if (st != SLIM_OK) return st;
  if (payload_bytes < need) return SLIM_EWORKSPACE;
  if (!slim_aligned16(W) || !slim_aligned16(payload) || !slim_aligned16(tile_info)) return SLIM_EALIGN;
  const int64_t tiles = (N / kHT) * (K / kHT);
  uint64_t* h_info = new (std::nothrow) uint64_t[tiles];
  if (!h_info) return SLIM_EDEVICE;
  slim_hybrid_layout(kinds, N, K, h_info, &need);
  hipStream_t s = (hipStream_t)stream;
  int* d_status = nullptr;
  int rc = SLIM_OK, h_status = 0;
  if (hipMalloc(&d_status, sizeof(int)) != hipSuccess) {
    delete[] h_info;
    return SLIM_EDEVICE;
  }
  do {
    if (hipMemcpyAsync(tile_info, h_info, tiles * sizeof(uint64_t), hipMemcpyHostToDevice, s) != hipSuccess ||
        hipMemsetAsync(d_status, 0, sizeof(int), s) != hipSuccess) {
      rc = SLIM_EDEVICE;
      break;
    }
    const int64_t threads = N * (K / 16);
    {
      SlimKernelTimer timer("hybrid_pack", s);
      SLIM_LAUNCH(timer, k_hybrid_pack, dim3((unsigned)((threads + kHThreads - 1) / kHThreads)), dim3(kHThreads), s, W,
                  N, K, (const uint64_t*)tile_info, payload, d_status);
    }
    if (hipGetLastError() != hipSuccess ||
        hipMemcpyAsync(&h_status, d_status, sizeof(int), hipMemcpyDeviceToHost, s) != hipSuccess ||
        hipStreamSynchronize(s) != hipSuccess) {
      rc = SLIM_EDEVICE;
      break;
    }
    if (h_status & 1) rc = SLIM_ENONFINITE;
  } while (0);
  (void)hipFree(d_status);
  delete[] h_info;
  return rc;
}

extern "C" int slim_linear_hybrid_workspace(int64_t M, int64_t N, int64_t K, size_t* bytes) {
  if (!bytes) return SLIM_EINVAL;
  if (M < 1 || N < kHT || K < kHT || N % kHT || K % kHT) return SLIM_ESHAPE;
  *bytes = hybrid_plan(M, N, K).ws;
  return SLIM_OK;
}

extern "C" int slim_linear_hybrid(const void* X, int64_t M, int64_t N, int64_t K, const uint64_t* tile_info,
                                  const uint8_t* payload, float* Y, void* ws, size_t ws_bytes, void* stream) {
  if (!X || !tile_info || !payload || !Y) return SLIM_EINVAL;
  if (M < 1 || N < kHT || K < kHT || N % kHT || K % kHT) return SLIM_ESHAPE;
  if (M * K >= ((int64_t)1 << 40) || M * N >= ((int64_t)1 << 40) || (M + kHT) / kHT >= 65536) return SLIM_EUNSUPPORTED;
  if (!slim_aligned16(X) || !slim_aligned16(payload) || !slim_aligned16(Y) || ((uintptr_t)tile_info & 7u))
    return SLIM_EALIGN;
  const HybridPlan p = hybrid_plan(M, N, K);
  if (p.splits > 1 && (!ws || ws_bytes < p.ws)) return SLIM_EWORKSPACE;
  if (p.splits > 1 && !slim_aligned16(ws)) return SLIM_EALIGN;
  hipStream_t s = (hipStream_t)stream;
  HybridArgs a{static_cast<const uint16_t*>(X), tile_info, payload, p.splits > 1 ? static_cast<float*>(ws) : Y,
               M, N, K, (int)p.chunks_per_split};
  {
    SlimKernelTimer timer("hybrid_gemm", s);
    SLIM_LAUNCH(timer, k_hybrid_gemm, dim3((unsigned)(N / kHT), (unsigned)((M + kHT - 1) / kHT), (unsigned)p.splits),
                dim3(kHThreads), s, a);
  }
  if (p.splits > 1) {
    const int64_t count4 = M * N / 4;
    SlimKernelTimer timer("hybrid_reduce", s);
    SLIM_LAUNCH(timer, k_hybrid_reduce, dim3((unsigned)((count4 + kHThreads - 1) / kHThreads)), dim3(kHThreads), s,
                (const float*)static_cast<float*>(ws), (int)p.splits, count4, Y);
  }
  return hipGetLastError() == hipSuccess ? SLIM_OK : SLIM_EDEVICE;
}
