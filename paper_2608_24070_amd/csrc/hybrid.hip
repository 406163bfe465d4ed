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
constexpr int kHRing = 3;
constexpr int kHMaxChunks = 256;               // K <= 32768

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
  // the tile's half (positions 0..63 or 64..127): 128 rows x 64 bytes of values, then 128 rows x
  // 8 bytes of index words
  const uint64_t hb = off + (uint64_t)(kHSparse / 2) * (uint64_t)(kk >> 6);
  const int kh = kk & 63;
  *reinterpret_cast<u32x4_t*>(payload + hb + (uint64_t)r * 64 + kh) = __builtin_bit_cast(u32x4_t, vals);
  *reinterpret_cast<uint16_t*>(payload + hb + 8192 + (uint64_t)r * 8 + 2 * (kh / 16)) = (uint16_t)half;
}

// ------------------------------------------------------------------------------------- GEMM
// A block computes 256 rows (two weight-tile rows) x 128 columns with 8 waves of 64 x 64; each
// 128-row half has its own tile kind per chunk. Ring stages hold 64 positions of K (half a weight
// tile) of both tile rows and of the 128 activation rows, 48 KiB per stage, three stages, two
// ahead: everything reaches LDS by direct loads (buffer_load ... lds, 16 bytes per lane), so no
// register holds data in flight. Waves 0-3 load tile row 0's weights and waves 4-7 tile row 1's:
// 4 loads per wave for a dense half-tile, 2 for a 2:4 one (+1 in the group's first wave, the
// index words); every wave loads 2 of the activations. The wait before stage s lets the loads of
// stage s + 1 be in flight, a count known from its kinds (a switch over the three possible
// immediates). LDS layouts (16-byte slots XOR-swizzled so that a wave's reads of one slot over
// consecutive rows hit distinct banks), per tile row at 16384 tr:
//   dense weights  row r (0..127): 128 bytes, slot s at s ^ (r % 8)
//   2:4 weights    values: row r 64 bytes, slot s at s ^ ((r / 4) % 2); index words at 8192 + 8 r
//   activations    (at 32768) row m (0..127): 128 bytes, slot s at s ^ (m % 8)
constexpr int kHStageK = 64;
constexpr int kHRows = 256;                   // output rows per block
constexpr int kHGemmThreads = 512;
struct HybridStage {
  uint8_t a[32768];
  uint8_t x[16384];
};

struct HybridArgs {
  const uint16_t* X;
  const uint64_t* info;
  const uint8_t* payload;
  float* out;          // Y [M, N] (one split) or partials [split][M][N]
  int64_t M, N, K;
  int64_t payload_bytes;
  int chunks_per_split;
};

// One block per CU: 144 KiB of ring.
__global__ void __launch_bounds__(kHGemmThreads, 1)
k_hybrid_gemm(HybridArgs g) {
  // one variable per stage, selected by compile-time indices
  __shared__ __attribute__((aligned(16))) HybridStage st0, st1, st2;
  // the block's tile-info words (two tile rows), read once before any direct load: afterwards an
  // info word comes from LDS into scalar registers, where the loads' offsets must be
  __shared__ uint64_t infos[2][kHMaxChunks];
  auto ring = [&](auto zc) -> HybridStage& {
    constexpr int z = decltype(zc)::value;
    if constexpr (z == 0) return st0;
    else if constexpr (z == 1) return st1;
    else return st2;
  };
  // the wave index in a scalar register: load counts and waits are wave-uniform branches
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wn = wave >> 1, wm = wave & 1;       // rows 64 wn .. + 63 of the block, columns 64 wm ..
  const int tr = wn >> 1;                        // the wave's tile row (for compute)
  const int lt = wave >> 2, lw = wave & 3;       // the tile row this wave loads, and its rank there
  const int l32 = lane & 31, h = lane >> 5;
  const int64_t n0 = (int64_t)blockIdx.x * kHRows, m0 = (int64_t)blockIdx.y * kHT;
  const int64_t chunks = g.K / kHT;
  const int64_t c_begin = (int64_t)blockIdx.z * g.chunks_per_split;
  const int64_t c_end = c_begin + g.chunks_per_split < chunks ? c_begin + g.chunks_per_split : chunks;
  const int64_t s_begin = 2 * c_begin, s_end = 2 * c_end;
  const int64_t tn0 = n0 / kHT;
  // a last block of a 128-row remainder (N % 256 == 128) loads and computes tile row 0 twice; the
  // second copy's rows lie past N and are never stored
  const int64_t tn1 = tn0 + 1 < g.N / kHT ? tn0 + 1 : tn0;
  for (int64_t c = c_begin + tid; c < c_end; c += kHGemmThreads) {
    infos[0][c - c_begin] = g.info[tn0 * chunks + c];
    infos[1][c - c_begin] = g.info[tn1 * chunks + c];
  }
  __syncthreads();

  const rsrc_t rw = make_rsrc(g.payload, g.payload_bytes);
  const int64_t xrows = g.M - m0 < kHT ? g.M - m0 : kHT;
  const rsrc_t rx = make_rsrc(g.X + m0 * g.K, xrows * g.K * 2);     // rows past M read as zero
  // per-lane source offsets of the wave's loads
  uint32_t ad[4], as[2], xo[2];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int p = 4 * lw + i, row = 8 * p + (lane >> 3), phys = lane & 7;
    ad[i] = (uint32_t)row * 256u + 16u * (uint32_t)(phys ^ (row & 7));
  }
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int p = 2 * lw + i, row = 16 * p + (lane >> 2), phys = lane & 3;
    as[i] = (uint32_t)row * 64u + 16u * (uint32_t)(phys ^ ((row >> 2) & 1));
    const int px = 2 * wave + i, rx_row = 8 * px + (lane >> 3), pxs = lane & 7;
    xo[i] = (uint32_t)rx_row * (uint32_t)g.K * 2u + 16u * (uint32_t)(pxs ^ (rx_row & 7));
  }
  const uint32_t ami = 8192u + 16u * (uint32_t)lane;     // the half's index words, 16 bytes per lane

  auto kind_of = [&](int t, int64_t s) -> uint64_t {
    const uint64_t v = infos[t][(s >> 1) - c_begin];
    const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
    const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(v >> 32));
    return ((uint64_t)hi << 32) | lo;
  };
  auto clamp_s = [&](int64_t s) -> int64_t { return s < s_end ? s : s_end - 1; };   // past the end: a dead slot
  // loads this wave issues for stage s
  auto loads_of = [&](int64_t s) -> int {
    return 2 + ((kind_of(lt, clamp_s(s)) & kHSparseBit) ? (lw == 0 ? 3 : 2) : 4);
  };
  auto issue = [&](int64_t s, auto zc) {
    const int64_t sc = clamp_s(s);
    const uint64_t ti = kind_of(lt, sc);
    const uint32_t toff = (uint32_t)(ti & ~kHSparseBit), half = (uint32_t)(sc & 1);
    HybridStage& S = ring(zc);
    uint8_t* A = &S.a[16384 * lt];
    if (!(ti & kHSparseBit)) {
#pragma unroll
      for (int i = 0; i < 4; ++i)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rw, (lds_ptr_t)&A[(4 * lw + i) * 1024], 16, ad[i] + 128u * half, toff,
                                                 0, 0);
    } else {
      const uint32_t soff = toff + (uint32_t)(kHSparse / 2) * half;
#pragma unroll
      for (int i = 0; i < 2; ++i)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rw, (lds_ptr_t)&A[(2 * lw + i) * 1024], 16, as[i], soff, 0, 0);
      if (lw == 0) __builtin_amdgcn_raw_ptr_buffer_load_lds(rw, (lds_ptr_t)&A[8192], 16, ami, soff, 0, 0);
    }
#pragma unroll
    for (int i = 0; i < 2; ++i)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rx, (lds_ptr_t)&S.x[(2 * wave + i) * 1024], 16, xo[i],
                                               (uint32_t)(sc * kHStageK * 2), 0, 0);
  };

  f16_t acc[2][2];
#pragma unroll
  for (int fn = 0; fn < 2; ++fn)
#pragma unroll
    for (int fm = 0; fm < 2; ++fm)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[fn][fm][e] = 0.f;

  // The compute phase reads LDS with ds_read instructions written out, and waits for them itself:
  // the compiler cannot tell which ring slot a direct load writes, so for reads it can see it would
  // wait for every direct load in flight, the next stage's included. Each wait names the registers
  // it completes, so no instruction using them is scheduled before it.
  auto rd16 = [](uint32_t addr) -> u32x4_t {
    u32x4_t v;
    asm volatile("ds_read_b128 %0, %1" : "=v"(v) : "v"(addr));
    return v;
  };
  auto rd_u16 = [](uint32_t addr) -> uint32_t {
    uint32_t v;
    asm volatile("ds_read_u16 %0, %1" : "=v"(v) : "v"(addr));
    return v;
  };
  struct DenseOps {
    u32x4_t a[2], b[2];
  };
  struct SparseOps {
    u32x4_t a[2], b[4];
    uint32_t i[2];
  };
  auto wait_dense = [](DenseOps& o) {
    asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(o.a[0]), "+v"(o.a[1]), "+v"(o.b[0]), "+v"(o.b[1]));
  };
  auto wait_sparse = [](SparseOps& o) {
    asm volatile("s_waitcnt lgkmcnt(0)"
                 : "+v"(o.a[0]), "+v"(o.a[1]), "+v"(o.b[0]), "+v"(o.b[1]), "+v"(o.b[2]), "+v"(o.b[3]), "+v"(o.i[0]),
                   "+v"(o.i[1]));
  };
  // per-lane LDS byte offsets inside a stage (rows of this lane's fragments)
  uint32_t ra_d[2], ra_s[2], ri_s[2], rx_[2];
  int rsw[2], xsw[2], rsw_s[2];
#pragma unroll
  for (int f = 0; f < 2; ++f) {
    const int r = 64 * (wn & 1) + 32 * f + l32, m = 64 * wm + 32 * f + l32;   // r: row within the tile row
    ra_d[f] = 16384u * (uint32_t)tr + (uint32_t)r * 128u;
    ra_s[f] = 16384u * (uint32_t)tr + (uint32_t)r * 64u;
    ri_s[f] = 16384u * (uint32_t)tr + 8192u + (uint32_t)r * 8u;
    rx_[f] = 32768u + (uint32_t)m * 128u;
    rsw[f] = r & 7;
    rsw_s[f] = (r >> 2) & 1;
    xsw[f] = m & 7;
  }

  auto compute = [&](auto zc, bool sparse) {
    const uint32_t base = (uint32_t)(uintptr_t)(lds_ptr_t)&ring(zc).a[0];   // the stage (a, then x)
    if (!sparse) {
      auto read = [&](int t, DenseOps& o) {
#pragma unroll
        for (int f = 0; f < 2; ++f) {
          o.a[f] = rd16(base + ra_d[f] + ((uint32_t)((2 * t + h) ^ rsw[f]) << 4));
          o.b[f] = rd16(base + rx_[f] + ((uint32_t)((2 * t + h) ^ xsw[f]) << 4));
        }
      };
      DenseOps o[2];
      read(0, o[0]);
      wait_dense(o[0]);
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        if (t < 3) read(t + 1, o[(t + 1) & 1]);
        const DenseOps& c = o[t & 1];
#pragma unroll
        for (int fn = 0; fn < 2; ++fn)
#pragma unroll
          for (int fm = 0; fm < 2; ++fm)
            acc[fn][fm] = mfma32(__builtin_bit_cast(h8_t, c.a[fn]), __builtin_bit_cast(h8_t, c.b[fm]), acc[fn][fm]);
        if (t < 3) wait_dense(o[(t + 1) & 1]);
      }
    } else {
      auto read = [&](int t, SparseOps& o) {
#pragma unroll
        for (int f = 0; f < 2; ++f) {
          // lane group h holds the 16 positions 32 t + 16 h .. + 15 of its row
          o.a[f] = rd16(base + ra_s[f] + ((uint32_t)((2 * t + h) ^ rsw_s[f]) << 4));
          o.i[f] = rd_u16(base + ri_s[f] + 2u * (uint32_t)(2 * t + h));
          o.b[2 * f] = rd16(base + rx_[f] + ((uint32_t)((4 * t + h) ^ xsw[f]) << 4));
          o.b[2 * f + 1] = rd16(base + rx_[f] + ((uint32_t)((4 * t + 2 + h) ^ xsw[f]) << 4));
        }
      };
      SparseOps o[2];
      read(0, o[0]);
      wait_sparse(o[0]);
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        if (t < 1) read(t + 1, o[1]);
        const SparseOps& c = o[t & 1];
#pragma unroll
        for (int fn = 0; fn < 2; ++fn)
#pragma unroll
          for (int fm = 0; fm < 2; ++fm)
            acc[fn][fm] = smfmac32(__builtin_bit_cast(h8_t, c.a[fn]),
                                   cat16(__builtin_bit_cast(h8_t, c.b[2 * fm]), __builtin_bit_cast(h8_t, c.b[2 * fm + 1])),
                                   acc[fn][fm], (int)c.i[fn], 0);
        if (t < 1) wait_sparse(o[1]);
      }
    }
  };

  // stage s in slot z: the wave's loads of stage s have landed once only those of s + 1 are
  // outstanding; the barrier then makes every wave's loads visible and ends every read of the slot
  // that stage s + 2 refills
  auto wait_ahead = [&](int n) {
    switch (n) {
      case 4: __builtin_amdgcn_s_waitcnt(vmcnt_lgkm0_wait(4)); break;
      case 5: __builtin_amdgcn_s_waitcnt(vmcnt_lgkm0_wait(5)); break;
      default: __builtin_amdgcn_s_waitcnt(vmcnt_lgkm0_wait(6)); break;
    }
  };
  auto step = [&](int64_t s, auto zc) {
    constexpr int z = decltype(zc)::value;
    const int ahead = loads_of(s + 1);
    __builtin_amdgcn_sched_barrier(0);
    wait_ahead(ahead);
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
    issue(s + 2, std::integral_constant<int, (z + 2) % kHRing>{});
    compute(zc, (kind_of(tr, s) & kHSparseBit) != 0);
  };

  if (s_begin < s_end) {
    issue(s_begin, std::integral_constant<int, 0>{});
    issue(s_begin + 1, std::integral_constant<int, 1>{});
    for (int64_t s = s_begin; s < s_end; s += kHRing) {
      step(s, std::integral_constant<int, 0>{});
      if (s + 1 < s_end) step(s + 1, std::integral_constant<int, 1>{});
      if (s + 2 < s_end) step(s + 2, std::integral_constant<int, 2>{});
    }
    // no direct load may still be writing LDS when the workgroup ends
    __builtin_amdgcn_s_waitcnt(0);
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
        if (nn >= g.N) continue;
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
  p.tiles = ((N + kHRows - 1) / kHRows) * ((M + kHT - 1) / kHT);
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
                                  const uint8_t* payload, size_t payload_bytes, float* Y, void* ws, size_t ws_bytes,
                                  void* stream) {
  if (!X || !tile_info || !payload || !Y) return SLIM_EINVAL;
  if (M < 1 || N < kHT || K < kHT || N % kHT || K % kHT) return SLIM_ESHAPE;
  // 32-bit buffer offsets: the payload and 128 activation rows stay below 4 GiB
  if (payload_bytes >= ((size_t)1 << 32) || (size_t)kHT * K * 2 >= ((size_t)1 << 32) || K / kHT > kHMaxChunks)
    return SLIM_EUNSUPPORTED;
  if (M * K >= ((int64_t)1 << 40) || M * N >= ((int64_t)1 << 40) || (M + kHT) / kHT >= 65536) return SLIM_EUNSUPPORTED;
  if (!slim_aligned16(X) || !slim_aligned16(payload) || !slim_aligned16(Y) || ((uintptr_t)tile_info & 7u))
    return SLIM_EALIGN;
  const HybridPlan p = hybrid_plan(M, N, K);
  if (p.splits > 1 && (!ws || ws_bytes < p.ws)) return SLIM_EWORKSPACE;
  if (p.splits > 1 && !slim_aligned16(ws)) return SLIM_EALIGN;
  hipStream_t s = (hipStream_t)stream;
  HybridArgs a{static_cast<const uint16_t*>(X), tile_info, payload, p.splits > 1 ? static_cast<float*>(ws) : Y,
               M, N, K, (int64_t)payload_bytes, (int)p.chunks_per_split};
  {
    SlimKernelTimer timer("hybrid_gemm", s);
    SLIM_LAUNCH(timer, k_hybrid_gemm, dim3((unsigned)((N + kHRows - 1) / kHRows), (unsigned)((M + kHT - 1) / kHT),
                                           (unsigned)p.splits),
                dim3(kHGemmThreads), s, a);
  }
  if (p.splits > 1) {
    const int64_t count4 = M * N / 4;
    SlimKernelTimer timer("hybrid_reduce", s);
    SLIM_LAUNCH(timer, k_hybrid_reduce, dim3((unsigned)((count4 + kHThreads - 1) / kHThreads)), dim3(kHThreads), s,
                (const float*)static_cast<float*>(ws), (int)p.splits, count4, Y);
  }
  return hipGetLastError() == hipSuccess ? SLIM_OK : SLIM_EDEVICE;
}
