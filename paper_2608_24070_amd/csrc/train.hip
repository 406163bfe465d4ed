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
// Block = 128 rows (n) x 128 columns (k). Phase 1 expands the value pack of the tile into LDS (fp16
// bits, 0 where M^R drops, and the M^R bit), each thread 16 columns of four rows with 16-byte LDS
// writes; phase 2 gives each thread a 16-row block nb and a column k, keeps the top two of each
// aligned 4-row group by (|v| desc, M^R bit desc, n asc) and writes 8 values (16 B) of valsT and
// one metaT half-word. A tile row is one whole 128-byte line of the value pack, and the eight
// 16-row blocks of one column go to eight consecutive threads, so every load and store moves whole
// lines. LDS columns are XOR-swizzled by the 16-row block (values by 8 nb, flags by 16 nb), so the
// phase-2 reads of one wave fall in distinct banks. A last partial tile (64 rows or 64 columns) is
// loaded from clamped addresses and stores only its own part.
constexpr int kTTn = 128, kTTk = 128;

__global__ void __launch_bounds__(256)
k_pack16_t(const uint16_t* __restrict__ vals, const uint8_t* __restrict__ meta, int64_t N, int64_t K,
           u32x4_t* __restrict__ valsT, uint16_t* __restrict__ metaT) {
  __shared__ __attribute__((aligned(16))) uint16_t v_s[kTTn][kTTk];
  __shared__ __attribute__((aligned(16))) uint8_t f_s[kTTn][kTTk];
  const int tid = threadIdx.x;
  const int64_t k0 = (int64_t)blockIdx.x * kTTk, n0 = (int64_t)blockIdx.y * kTTn;
  const int rows = N - n0 < kTTn ? (int)(N - n0) : kTTn;   // 64 or 128
  const int cols = K - k0 < kTTk ? (int)(K - k0) : kTTk;   // 64 or 128
  // every load first, then the LDS writes; thread -> (row tid / 8 + 32 j, 16 columns 16 (tid % 8))
  const int w = tid & 7;
  const int64_t kc = k0 + (16 * w < cols ? 16 * w : 0);    // first column of the thread's 16
  uint16_t mws[4];
  u32x4_t v8s[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int row = (tid >> 3) + 32 * j;
    const int64_t n = n0 + (row < rows ? row : rows - 1);
    mws[j] = *reinterpret_cast<const uint16_t*>(meta + n * (K / 8) + kc / 8);
    v8s[j] = *reinterpret_cast<const u32x4_t*>(vals + n * (K / 2) + kc / 2);
  }
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int row = (tid >> 3) + 32 * j;
    const int nb = (row >> 4) & 7;
    uint32_t vd[8], fd[4];
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const uint32_t i0 = (mws[j] >> (4 * c)) & 3u, i1 = (mws[j] >> (4 * c + 2)) & 3u;
      const uint32_t pr = v8s[j][c], lo = pr & 0xFFFFu, hi = pr >> 16;
      uint32_t e[4];
#pragma unroll
      for (int p = 0; p < 4; ++p) e[p] = (uint32_t)p == i0 ? lo : ((uint32_t)p == i1 ? hi : 0u);
      vd[2 * c] = e[0] | (e[1] << 16);
      vd[2 * c + 1] = e[2] | (e[3] << 16);
      fd[c] = (1u << (8 * i0)) | (1u << (8 * i1));
    }
    if (row < rows && 16 * w < cols) {
      *reinterpret_cast<u32x4_t*>(&v_s[row][(16 * w) ^ (8 * nb)]) = u32x4_t{vd[0], vd[1], vd[2], vd[3]};
      *reinterpret_cast<u32x4_t*>(&v_s[row][(16 * w + 8) ^ (8 * nb)]) = u32x4_t{vd[4], vd[5], vd[6], vd[7]};
      *reinterpret_cast<u32x4_t*>(&f_s[row][(16 * w) ^ (16 * nb)]) = u32x4_t{fd[0], fd[1], fd[2], fd[3]};
    }
  }
  __syncthreads();
  // thread -> (16-row block tid % 8, column tid / 8 + 32 j)
  const int blk = tid & 7;
  if (16 * blk >= rows) return;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int col = (tid >> 3) + 32 * j;
    if (col >= cols) break;
    uint32_t hv[4], mw = 0;
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int r0 = 16 * blk + 4 * c;
      // key: fp16 magnitude (finite values order as their bit patterns), then the M^R bit, then
      // the lower row; distinct within a group, so q comes before p exactly when key[q] > key[p]
      uint32_t key[4], bits[4];
#pragma unroll
      for (int p = 0; p < 4; ++p) {
        bits[p] = v_s[r0 + p][col ^ (8 * blk)];
        key[p] = ((bits[p] & 0x7FFFu) << 3) | ((uint32_t)f_s[r0 + p][col ^ (16 * blk)] << 2) | (uint32_t)(3 - p);
      }
      // keep[p]: fewer than two entries come before p; exactly two are kept, so the first kept is
      // among 0..2 and the last among 1..3 (selects, no branches)
      bool keep[4];
#pragma unroll
      for (int p = 0; p < 4; ++p) {
        uint32_t rank = 0;
#pragma unroll
        for (int q = 0; q < 4; ++q)
          if (q != p) rank += key[q] > key[p] ? 1u : 0u;
        keep[p] = rank < 2;
      }
      const uint32_t i0 = keep[0] ? 0u : (keep[1] ? 1u : 2u), i1 = keep[3] ? 3u : (keep[2] ? 2u : 1u);
      const uint32_t b0 = keep[0] ? bits[0] : (keep[1] ? bits[1] : bits[2]);
      const uint32_t b1 = keep[3] ? bits[3] : (keep[2] ? bits[2] : bits[1]);
      hv[c] = b0 | (b1 << 16);
      mw |= (i0 | (i1 << 2)) << (4 * c);
    }
    const int64_t k = k0 + col, nb = n0 / 16 + blk;       // 16-row block along n
    valsT[k * (N / 16) + nb] = u32x4_t{hv[0], hv[1], hv[2], hv[3]};
    metaT[k * (N / 16) + nb] = (uint16_t)mw;
  }
}

// ------------------------------------------------------------------------------- grad_w
// D[k][n] = sum_m X[m][k] dY[m][n] (= grad W^T) on 32x32x16 MFMA, fp32 accumulate; tile 256 (k) x
// 256 (n) for 8 waves, two per SIMD: wave (wk, wn) owns k rows 128 wk .. + 127 and n columns
// 64 wn .. + 63 (4 x 2 fragments). The tile's operand traffic per flop is half a 128 x 128 tile's
// (every dY column slab is read by K/256 tiles, every X slab by N/256).
// Both operands are [M, *] row-major and the reduction runs along their rows, so the MFMA operands
// (eight consecutive reduction positions of one column per lane) are columns of the stored tiles.
// The tiles go to LDS as they are, by direct loads (buffer_load ... lds, 16 bytes per lane): per
// 32-row chunk 16 KiB of X and 16 KiB of dY, a ring of four stages three ahead, no register holding
// data in flight. The operands are read back transposed with ds_read_b64_tr_b16: in each group of 16
// lanes, lane 16 G + 4 a + b receives element b of the 8-byte rows addressed by lanes
// 16 G + a + 4 i (i = 0..3). Lane q of group G addresses row m0 + 8 (G / 2) + q / 4 (+ 4 for the
// second read) at column c0 + 16 (G % 2) + 4 (q % 4), so lane l gets the eight reduction positions
// 8 (l / 32) .. + 7 of column c0 + l % 32: the MFMA's operand layout.
// LDS rows are 512 bytes; 32-byte pieces are XOR-swizzled by 2 (row % 4) so that the four rows one
// group reads at once fall in distinct banks.
// Columns past N or K (a last partial tile) read neighbouring data; D entries of such a column are
// never stored, and no other entry depends on it.
// Epilogue: a fragment row block 8q + 4 (L / 32) .. + 3 of lane L is one aligned 4-group of k for
// column n = L % 32, so the two positions M^R keeps (one metadata nibble) are selected in
// registers and stored as the compressed pair gW[n][2g], gW[n][2g + 1].
constexpr int kGT = 256, kGM = 32, kGThreads = 512, kGRing = 4;

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

// byte offset of 16-bit column c of row r in a swizzled 512-byte LDS row
SLIM_DEV uint32_t gw_off(int r, int c) {
  return (uint32_t)r * 512u + ((uint32_t)(((c >> 4) ^ (2 * (r & 3))) << 5)) + (uint32_t)((c & 15) * 2);
}

template <bool BF16>
__global__ void __launch_bounds__(kGThreads)
k_grad_w(const uint16_t* __restrict__ dY, const uint16_t* __restrict__ X, int64_t M, int64_t N, int64_t K,
         const uint8_t* __restrict__ meta, float* __restrict__ gW) {
  // the ring: X chunks [m][k] in slots of 16 KiB at 0, dY chunks [m][n] at 64 KiB (512-byte rows);
  // every offset a read adds to its lane's address then fits the 16-bit immediate of a DS read
  constexpr uint32_t kSlot = kGM * kGT * 2, kYBase = kGRing * kSlot;
  __shared__ __attribute__((aligned(16))) uint8_t lds[2 * kGRing * kSlot];
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

  // direct loads: each wave loads two 1 KiB pieces (rows 2 p, 2 p + 1, p = 2 wave + i) of X and of
  // dY per chunk; lane L writes LDS bytes 16 L of the piece, i.e. row 2 p + L / 32 at physical
  // 16-byte slot L % 32, which holds logical slot (L % 32) ^ (4 (row % 4)) (the 32-byte XOR above)
  const rsrc_t ry = make_rsrc(dY, M * N * 2), rx = make_rsrc(X, M * K * 2);
  uint32_t xo[2], yo[2];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int p = 2 * wave + i, row = 2 * p + (lane >> 5), ls = (lane & 31) ^ (4 * (row & 3));
    xo[i] = ((uint32_t)row * (uint32_t)K + (uint32_t)(k0 + 8 * ls)) * 2u;
    yo[i] = ((uint32_t)row * (uint32_t)N + (uint32_t)(n0 + 8 * ls)) * 2u;
  }
  const uint32_t xstep = (uint32_t)kGM * (uint32_t)K * 2u, ystep = (uint32_t)kGM * (uint32_t)N * 2u;
  const int64_t nch = (M + kGM - 1) / kGM;
  auto issue = [&](int64_t c, auto zc) {
    const uint32_t cc = (uint32_t)(c < nch ? c : nch - 1);      // past the end: reload into a dead slot
    constexpr uint32_t z = decltype(zc)::value;
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const uint32_t o = z * kSlot + (uint32_t)(2 * wave + i) * 1024u;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rx, (lds_ptr_t)&lds[o], 16, xo[i], cc * xstep, 0, 0);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(ry, (lds_ptr_t)&lds[kYBase + o], 16, yo[i], cc * ystep, 0, 0);
    }
  };

  f16_t acc[4][2];
#pragma unroll
  for (int x = 0; x < 4; ++x)
#pragma unroll
    for (int y = 0; y < 2; ++y)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[x][y][v] = 0.f;

  // transposed operand reads, written out (the compiler cannot tell ring slots apart for direct
  // loads and would wait for every one in flight); each wait names the registers it completes
  auto rd_tr = [](uint32_t addr, auto oc) -> u32x2_t {
    u32x2_t v;
    asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2" : "=v"(v) : "v"(addr), "i"(decltype(oc)::value));
    return v;
  };
  // per-lane part of the read addresses: row 8 (G / 2) + q / 4 and column 16 (G % 2) + 4 (q % 4)
  const int G = lane >> 4, q = lane & 15;
  const int rr = 8 * (G >> 1) + (q >> 2), cr = 16 * (G & 1) + 4 * (q & 3);
  const uint32_t lb = (uint32_t)(uintptr_t)(lds_ptr_t)&lds[0];
  uint32_t ax[4][2], by[2][2];           // [fragment][read]: addresses in slot 0, for step 0
#pragma unroll
  for (int j = 0; j < 2; ++j) {
#pragma unroll
    for (int f = 0; f < 4; ++f) ax[f][j] = lb + gw_off(rr + 4 * j, 128 * wk + 32 * f + cr);
#pragma unroll
    for (int f = 0; f < 2; ++f) by[f][j] = lb + kYBase + gw_off(rr + 4 * j, 64 * wn + 32 * f + cr);
  }
  // operands of one 16-row step: X fragments [4][2 reads], dY fragments [2][2 reads]
  struct Frags {
    u32x2_t a[4][2], b[2][2];
  };
  auto read = [&](Frags& F, auto zc, auto stc) {    // step st (0, 1) of the chunk in slot z
    using off = std::integral_constant<uint32_t, decltype(zc)::value * kSlot + decltype(stc)::value * 16u * 512u>;
#pragma unroll
    for (int j = 0; j < 2; ++j) {
#pragma unroll
      for (int f = 0; f < 4; ++f) F.a[f][j] = rd_tr(ax[f][j], off{});
#pragma unroll
      for (int f = 0; f < 2; ++f) F.b[f][j] = rd_tr(by[f][j], off{});
    }
  };
  auto landed = [](Frags& F) {
    asm volatile("s_waitcnt lgkmcnt(0)"
                 : "+v"(F.a[0][0]), "+v"(F.a[0][1]), "+v"(F.a[1][0]), "+v"(F.a[1][1]), "+v"(F.a[2][0]),
                   "+v"(F.a[2][1]), "+v"(F.a[3][0]), "+v"(F.a[3][1]), "+v"(F.b[0][0]), "+v"(F.b[0][1]),
                   "+v"(F.b[1][0]), "+v"(F.b[1][1]));
  };
  // MFMAs I0 .. I1 - 1 of the step in F (i = 2 x + y); with RD the twelve reads of the step N
  // (slot z, step st) are spread over them, two before each of the first six, so that no wave
  // sends a burst of reads and the last ones have an MFMA or two to land
  auto mma_rng = [&](const Frags& F, Frags& N, auto zc, auto stc, auto i0c, auto i1c, auto rdc) {
    using off = std::integral_constant<uint32_t, decltype(zc)::value * kSlot + decltype(stc)::value * 16u * 512u>;
    constexpr int I0 = decltype(i0c)::value, I1 = decltype(i1c)::value, n = I1 - I0;
    constexpr int m = n > 7 ? 6 : (n > 1 ? n - 1 : 1);
#pragma unroll
    for (int i = I0; i < I1; ++i) {
      const int x = i >> 1, y = i & 1, k = i - I0;
      if (decltype(rdc)::value && k < m) {
#pragma unroll
        for (int r = 12 * k / m; r < 12 * (k + 1) / m; ++r) {
          if (r < 8) N.a[r >> 1][r & 1] = rd_tr(ax[r >> 1][r & 1], off{});
          else N.b[(r - 8) >> 1][(r - 8) & 1] = rd_tr(by[(r - 8) >> 1][(r - 8) & 1], off{});
        }
      }
      __builtin_amdgcn_sched_barrier(0);
      const u32x4_t av = {F.a[x][0][0], F.a[x][0][1], F.a[x][1][0], F.a[x][1][1]};
      const u32x4_t bv = {F.b[y][0][0], F.b[y][0][1], F.b[y][1][0], F.b[y][1][1]};
      acc[x][y] = mfma_acc<BF16>(av, bv, acc[x][y]);
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  using I_0 = std::integral_constant<int, 0>;
  using I_1 = std::integral_constant<int, 1>;
  using I_8 = std::integral_constant<int, 8>;

  // Software pipeline over chunks: the operands of the next step are read while the MFMAs of the
  // current one run, and the barrier sits between a chunk's two steps, so no wave starts a chunk
  // waiting for LDS. Chunk c + 1 has landed for this wave once only the loads of c + 2 and c + 3
  // are outstanding (8); the barrier then makes every wave's loads of c + 1 visible and ends every
  // read of chunk c, whose slot chunk c + 4 refills (after one MFMA, so that the SIMD has work
  // while the loads issue). After the last chunk the same steps read a slot refilled with a copy
  // of the last chunk (loads past the end repeat it) and use none of it.
  Frags A, B;
  auto step = [&](int64_t c, auto zc) {
    constexpr int z = decltype(zc)::value;
    using zn = std::integral_constant<int, (z + 1) % kGRing>;
    mma_rng(A, B, zc, I_1{}, I_0{}, I_8{}, std::true_type{});
    landed(B);
    __builtin_amdgcn_s_waitcnt(vmcnt_lgkm0_wait(8));
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
    mma_rng(B, A, zn{}, I_0{}, I_0{}, I_1{}, std::false_type{});
    issue(c + 4, zc);
    mma_rng(B, A, zn{}, I_0{}, I_1{}, I_8{}, std::true_type{});
    landed(A);
  };
  issue(0, std::integral_constant<int, 0>{});
  issue(1, std::integral_constant<int, 1>{});
  issue(2, std::integral_constant<int, 2>{});
  __builtin_amdgcn_s_waitcnt(vmcnt_lgkm0_wait(8));
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_sched_barrier(0);
  issue(3, std::integral_constant<int, 3>{});
  read(A, std::integral_constant<int, 0>{}, std::integral_constant<int, 0>{});
  landed(A);
  for (int64_t c = 0; c < nch; c += kGRing) {
    step(c, std::integral_constant<int, 0>{});
    if (c + 1 < nch) step(c + 1, std::integral_constant<int, 1>{});
    if (c + 2 < nch) step(c + 2, std::integral_constant<int, 2>{});
    if (c + 3 < nch) step(c + 3, std::integral_constant<int, 3>{});
  }
  // no direct load may still be writing LDS when the workgroup ends
  __builtin_amdgcn_s_waitcnt(0);

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
      for (int q4 = 0; q4 < 4; ++q4) {
        const int t = 2 * q4 + h;                               // group gb + t holds rows 8 q4 + 4h ..
        const uint32_t nib = (md >> (4 * t)) & 0xFu;
        const float v0 = sel4(acc[x][y], 4 * q4, (int)(nib & 3u)), v1 = sel4(acc[x][y], 4 * q4, (int)(nib >> 2));
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
  SLIM_LAUNCH(timer, k_pack16_t, dim3((unsigned)((K + kTTk - 1) / kTTk), (unsigned)((N + kTTn - 1) / kTTn)), dim3(256),
              s, vals, meta, N, K,
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
