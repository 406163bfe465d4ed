// lora.hip - SLiM-LoRA on the GPU: saliency-based low-rank adapters from the compression error
// (SLiM chapter, "SLiM-LoRA low-rank adapters": eq. lora_wanda_objective_function, eq. lora_svd,
// Alg. lora).
//
// With x the per-channel mean input magnitude shifted by its minimum and
// S = diag(x) (W^C - W)^T [K x N], the adapters are L = -diag(1/x) U_r Sigma_r^(1/2) and
// R = Sigma_r^(1/2) V_r^T from the r largest singular triplets of S. The singular vectors of the
// smaller side come from the eigenvectors of the Gram matrix G = A A^T (float64), where A is S
// (K <= N, left vectors) or S^T (N < K, right vectors), d = min(K, N); the other side follows
// from one more product with A.
//
// The eigensolver is two-sided block Jacobi. Indices are cut into blocks of 32; each round pairs
// the blocks by the round-robin (circle) schedule, and every pair's 64 x 64 diagonal block of G gets
// one cyclic Jacobi sweep in LDS (k_lora_pair_solve, its own round-robin over 64 indices: running
// the inner problem to convergence instead costs about six times as much per round and saves at most
// one outer sweep);
// the round then applies the pairs' rotations to G (G <- J^T G J, tile by tile, k_lora_apply_g)
// and accumulates them in V (V <- V J, k_lora_apply_v). Sweeps of nb - 1 rounds repeat until the
// off-diagonal norm of G falls below 1e-13 of its Frobenius norm (or stalls at rounding level).
// The eigenvalues are then G's diagonal; the r largest are picked by rank (ties to the lower index).
#include <math.h>

#include "slim_device.h"
#include "slim_host.h"
#include "slim_timing.h"

namespace {

constexpr int kLB = 32;              // Jacobi block
constexpr int kLP = 2 * kLB;         // pair size
constexpr int kLT = 256;             // threads of the tiled kernels
constexpr int kLPad = kLP + 1;       // LDS row pitch (doubles) of 64 x 64 tiles
constexpr int kLInnerSweeps = 1;
constexpr int kLMaxSweeps = 40;
constexpr int kLCalibRows = 256;     // calibration rows per partial sum
constexpr int kLOffBlocks = 512;

__device__ __forceinline__ int rr_slot(int i, int t, int n) { return i == 0 ? 0 : 1 + ((i - 1 + t) % (n - 1)); }

// index of row/column i (0..63) of pair p in round t of nb blocks
__device__ __forceinline__ int64_t pair_index(int p, int t, int nb, int i) {
  const int blk = i < kLB ? rr_slot(p, t, nb) : rr_slot(nb - 1 - p, t, nb);
  return (int64_t)blk * kLB + (i & (kLB - 1));
}

// 64 x 64 tiles between a dp-pitch matrix and LDS. Tile row r is matrix row row_of(r); the tile's
// columns are two runs of 32 contiguous doubles (a pair's two blocks), at c0 (tile columns 0..31)
// and c1 (32..63). Thread e of a 16-byte piece: run e / 16 (row run / 2, half run % 2), doubles
// 2 (e % 16) and 2 (e % 16) + 1 of it; eight pieces per thread. All loads are issued before the
// first LDS write: a loop that stored each element as its load arrived waited for every load in
// turn.
template <typename RowOf>
__device__ __forceinline__ void tile_load(const double* __restrict__ M, int64_t dp, RowOf row_of, int64_t c0,
                                          int64_t c1, double (*s)[kLPad]) {
  double2 v[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int e = threadIdx.x + kLT * i, run = e >> 4, q = e & 15;
    v[i] = *reinterpret_cast<const double2*>(M + row_of(run >> 1) * dp + ((run & 1) ? c1 : c0) + 2 * q);
  }
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int e = threadIdx.x + kLT * i, run = e >> 4, q = e & 15, r = run >> 1, c = 32 * (run & 1) + 2 * q;
    s[r][c] = v[i].x;
    s[r][c + 1] = v[i].y;
  }
}
// the same tile stored back; TRANS stores s transposed (matrix row row_of(r), column c <- s[c][r])
template <bool TRANS, typename RowOf>
__device__ __forceinline__ void tile_store(double* __restrict__ M, int64_t dp, RowOf row_of, int64_t c0, int64_t c1,
                                           const double (*s)[kLPad]) {
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int e = threadIdx.x + kLT * i, run = e >> 4, q = e & 15, r = run >> 1, c = 32 * (run & 1) + 2 * q;
    double2 w;
    w.x = TRANS ? s[c][r] : s[r][c];
    w.y = TRANS ? s[c + 1][r] : s[r][c + 1];
    *reinterpret_cast<double2*>(M + row_of(r) * dp + ((run & 1) ? c1 : c0) + 2 * q) = w;
  }
}
// the two column runs of pair p in round t
__device__ __forceinline__ int64_t pair_run(int p, int t, int nb, int h) {
  return (int64_t)rr_slot(h ? nb - 1 - p : p, t, nb) * kLB;
}

// ---------------------------------------------------------------- calibration statistic
// part[c][k] = sum over rows c*kLCalibRows .. +kLCalibRows-1 of |X[row][k]| (float64)
__global__ void __launch_bounds__(kLT)
k_lora_calib(const uint16_t* __restrict__ X, int bf16, int64_t B, int64_t K, double* __restrict__ part) {
  const int64_t k = (int64_t)blockIdx.x * kLT + threadIdx.x;
  if (k >= K) return;
  const int64_t r0 = (int64_t)blockIdx.y * kLCalibRows;
  const int64_t r1 = r0 + kLCalibRows < B ? r0 + kLCalibRows : B;
  double s = 0.0;
  for (int64_t i = r0; i < r1; ++i) {
    const uint16_t b = X[i * K + k];
    const float v = bf16 ? __uint_as_float((uint32_t)b << 16) : (float)__builtin_bit_cast(_Float16, b);
    s += (double)fabsf(v);
  }
  part[blockIdx.y * K + k] = s;
}

// x_k = mean_k + min_j mean_j; status bit 2 if some x_k is zero (one block)
__global__ void __launch_bounds__(1024)
k_lora_calib_final(const double* __restrict__ part, int64_t chunks, int64_t B, int64_t K, double* __restrict__ x,
                   int* __restrict__ status) {
  __shared__ double red[16];
  double mn = INFINITY;
  for (int64_t k = threadIdx.x; k < K; k += 1024) {
    double s = 0.0;
    for (int64_t c = 0; c < chunks; ++c) s += part[c * K + k];
    const double m = s / (double)B;
    x[k] = m;
    mn = fmin(mn, m);
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) mn = fmin(mn, __shfl_xor(mn, off, 64));
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = mn;
  __syncthreads();
  double m = red[0];
  for (int w = 1; w < 16; ++w) m = fmin(m, red[w]);
  int bad = 0;
  for (int64_t k = threadIdx.x; k < K; k += 1024) {
    const double v = x[k] + m;
    x[k] = v;
    if (!(v > 0.0)) bad = 1;
  }
  if (bad) atomicOr(status, 2);
}

// ---------------------------------------------------------------- saliency-weighted error
// Wc[n][k] of the blocked forward pack (exact in float64), 0 where the mask drops it.
__device__ __forceinline__ double pack_value(const uint32_t* __restrict__ codes, const uint16_t* __restrict__ meta,
                                             const uint16_t* __restrict__ scales, int64_t n, int64_t k, int64_t K) {
  const int64_t slot = packed_slot(n, k >> 7, K >> 7);
  const int w = (int)((k & 127) >> 4);
  const uint32_t cw = codes[8 * slot + w];
  const uint32_t mw = meta[8 * slot + w];
  const int c = (int)((k & 15) >> 2), pos = (int)(k & 3);
  const int i0 = (mw >> (4 * c)) & 3, i1 = (mw >> (4 * c + 2)) & 3;
  int u;
  if (pos == i0) u = (cw >> (4 * c)) & 15;
  else if (pos == i1) u = (cw >> (16 + 4 * c)) & 15;
  else return 0.0;
  const double s = (double)__builtin_bit_cast(_Float16, scales[slot]);
  return (double)(u - 8) * s;
}

// A = S [K x N] (left: A[k][n]) or S^T [N x K] (right: A[n][k]), with
// S[k][n] = x_k (Wc[n][k] - W[n][k]). 64 x 64 tiles of (n, k); the left form is written transposed
// through LDS so that both the reads of W and the writes of A are along contiguous rows.
__global__ void __launch_bounds__(kLT)
k_lora_error(const float* __restrict__ W, const uint32_t* __restrict__ codes, const uint16_t* __restrict__ meta,
             const uint16_t* __restrict__ scales, int64_t N, int64_t K, const double* __restrict__ x, int left,
             double* __restrict__ A) {
  __shared__ double t[64][65];
  const int64_t n0 = (int64_t)blockIdx.y * 64, k0 = (int64_t)blockIdx.x * 64;
  for (int e = threadIdx.x; e < 64 * 64; e += kLT) {
    const int i = e >> 6, j = e & 63;                 // i: n offset, j: k offset
    const int64_t n = n0 + i, k = k0 + j;
    double v = 0.0;
    if (n < N && k < K) v = x[k] * (pack_value(codes, meta, scales, n, k, K) - (double)W[n * K + k]);
    if (left) t[i][j] = v;
    else if (n < N && k < K) A[n * K + k] = v;
  }
  if (!left) return;
  __syncthreads();
  for (int e = threadIdx.x; e < 64 * 64; e += kLT) {
    const int j = e >> 6, i = e & 63;                 // A[k][n]: rows k, contiguous n
    const int64_t n = n0 + i, k = k0 + j;
    if (n < N && k < K) A[k * N + n] = t[i][j];
  }
}

// ---------------------------------------------------------------- Gram matrix
// G = A A^T over rows 0..d-1 of A [d x D] (rows d..dp-1 are zero); 64 x 64 tiles with ti <= tj,
// the mirror written from the same tile.
__global__ void __launch_bounds__(kLT)
k_lora_gram(const double* __restrict__ A, int64_t D, int64_t d, int64_t dp, double* __restrict__ G) {
  const int ti = blockIdx.y, tj = blockIdx.x;
  if (ti > tj) return;
  __shared__ double as[64][33], bs[64][33];
  const int tr = threadIdx.x >> 4, tc = threadIdx.x & 15;     // 4 x 4 outputs per thread
  double acc[4][4] = {};
  const int64_t i0 = (int64_t)ti * 64, j0 = (int64_t)tj * 64;
  for (int64_t t0 = 0; t0 < D; t0 += 32) {
    for (int e = threadIdx.x; e < 64 * 32; e += kLT) {
      const int r = e >> 5, c = e & 31;
      const int64_t t = t0 + c;
      as[r][c] = (i0 + r < d && t < D) ? A[(i0 + r) * D + t] : 0.0;
      bs[r][c] = (j0 + r < d && t < D) ? A[(j0 + r) * D + t] : 0.0;
    }
    __syncthreads();
#pragma unroll 4
    for (int c = 0; c < 32; ++c) {
      double a[4], b[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        a[u] = as[4 * tr + u][c];
        b[u] = bs[4 * tc + u][c];
      }
#pragma unroll
      for (int u = 0; u < 4; ++u)
#pragma unroll
        for (int v = 0; v < 4; ++v) acc[u][v] = fma(a[u], b[v], acc[u][v]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int u = 0; u < 4; ++u)
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int64_t i = i0 + 4 * tr + u, j = j0 + 4 * tc + v;
      G[i * dp + j] = acc[u][v];
      if (ti != tj) G[j * dp + i] = acc[u][v];
    }
}

__global__ void __launch_bounds__(kLT) k_lora_eye(double* __restrict__ V, int64_t dp) {
  const int64_t e = (int64_t)blockIdx.x * kLT + threadIdx.x;
  if (e >= dp * dp) return;
  V[e] = (e / dp == e % dp) ? 1.0 : 0.0;
}

// ---------------------------------------------------------------- block Jacobi
// Off-diagonal and diagonal sums of squares of G, per block (fixed grid, fixed order).
__global__ void __launch_bounds__(kLT)
k_lora_offnorm(const double* __restrict__ G, int64_t dp, double* __restrict__ part) {
  double off = 0.0, dia = 0.0;
  const int64_t tot = dp * dp;
  for (int64_t e = (int64_t)blockIdx.x * kLT + threadIdx.x; e < tot; e += (int64_t)gridDim.x * kLT) {
    const double v = G[e];
    if (e / dp == e % dp) dia += v * v;
    else off += v * v;
  }
  __shared__ double ro[kLT / 64], rd[kLT / 64];
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    off += __shfl_xor(off, o, 64);
    dia += __shfl_xor(dia, o, 64);
  }
  if ((threadIdx.x & 63) == 0) {
    ro[threadIdx.x >> 6] = off;
    rd[threadIdx.x >> 6] = dia;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    double so = 0.0, sd = 0.0;
    for (int w = 0; w < kLT / 64; ++w) {
      so += ro[w];
      sd += rd[w];
    }
    part[2 * blockIdx.x] = so;
    part[2 * blockIdx.x + 1] = sd;
  }
}

__global__ void __launch_bounds__(64) k_lora_offnorm_final(const double* __restrict__ part, int nparts,
                                                           double* __restrict__ out) {
  if (threadIdx.x != 0) return;
  double so = 0.0, sd = 0.0;
  for (int b = 0; b < nparts; ++b) {
    so += part[2 * b];
    sd += part[2 * b + 1];
  }
  out[0] = so;
  out[1] = sd;
}

// Jacobi rotation zeroing a[p][q] of a symmetric 2 x 2 problem: returns false when a_pq is
// negligible (no rotation).
__device__ __forceinline__ bool rotation(double app, double aqq, double apq, double& c, double& s) {
  if (fabs(apq) <= 1e-300 || fabs(apq) <= 1e-17 * sqrt(fabs(app * aqq))) {
    c = 1.0;
    s = 0.0;
    return false;
  }
  const double th = (aqq - app) / (2.0 * apq);
  double t;
  if (fabs(th) >= 1e150) t = 1.0 / (2.0 * th);
  else t = (th >= 0.0 ? 1.0 : -1.0) / (fabs(th) + sqrt(th * th + 1.0));
  c = 1.0 / sqrt(t * t + 1.0);
  s = t * c;
  return true;
}

// One block per pair of round t: kLInnerSweeps cyclic Jacobi sweeps over G's 64 x 64 block of the
// pair (fewer if a sweep rotates nothing); its accumulated rotation J (64 x 64, row-major) goes to
// Jout[pair].
__global__ void __launch_bounds__(kLT)
k_lora_pair_solve(const double* __restrict__ G, int64_t dp, int nb, int t, double* __restrict__ Jout) {
  __shared__ double a[kLP][kLPad], j[kLP][kLPad];
  __shared__ double cc[kLB], ss[kLB];
  __shared__ int pp[kLB], qq[kLB];
  __shared__ int rotated;
  const int pr = blockIdx.x;
  tile_load(G, dp, [&](int r) { return pair_index(pr, t, nb, r); }, pair_run(pr, t, nb, 0), pair_run(pr, t, nb, 1), a);
  for (int e = threadIdx.x; e < kLP * kLP; e += kLT) {
    const int r = e >> 6, c = e & 63;
    j[r][c] = r == c ? 1.0 : 0.0;
  }
  __syncthreads();
  for (int sw = 0; sw < kLInnerSweeps; ++sw) {
    if (threadIdx.x == 0) rotated = 0;
    __syncthreads();
    for (int u = 0; u < kLP - 1; ++u) {
      // the step's 32 rotations, and their index pairs for the updates below (computed once here:
      // the round-robin slot is a remainder, costly per element)
      if (threadIdx.x < kLB) {
        const int p = rr_slot(threadIdx.x, u, kLP), q = rr_slot(kLP - 1 - threadIdx.x, u, kLP);
        double c, s;
        if (rotation(a[p][p], a[q][q], a[p][q], c, s)) rotated = 1;
        cc[threadIdx.x] = c;
        ss[threadIdx.x] = s;
        pp[threadIdx.x] = p;
        qq[threadIdx.x] = q;
      }
      __syncthreads();
      // A <- J^T A J in one pass: the rotations are disjoint index pairs, so every element of A lies
      // in exactly one 2 x 2 block (rows p1, q1 of rotation w1, columns p2, q2 of rotation w2), which
      // becomes R1^T block R2 from its own four values; thread: rotation w1 = tid / 8 and w2 =
      // tid % 8 + 8 i (i < 4). J <- J R by columns: thread row tid % 64, rotations w = tid / 64 + 4 i
      // (i < 8). Every LDS read of a phase is issued before its arithmetic.
      {
        const int w1 = threadIdx.x >> 3;
        const int p1 = pp[w1], q1 = qq[w1];
        const double c1 = cc[w1], s1 = ss[w1];
        int p2[4], q2[4];
        double c2[4], s2[4], b00[4], b01[4], b10[4], b11[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int w2 = (threadIdx.x & 7) + 8 * i;
          p2[i] = pp[w2];
          q2[i] = qq[w2];
          c2[i] = cc[w2];
          s2[i] = ss[w2];
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          b00[i] = a[p1][p2[i]];
          b01[i] = a[p1][q2[i]];
          b10[i] = a[q1][p2[i]];
          b11[i] = a[q1][q2[i]];
        }
        const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
        int pw[8], qw[8];
        double cw[8], sw[8], jp[8], jq[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          pw[i] = pp[wv + 4 * i];
          qw[i] = qq[wv + 4 * i];
          cw[i] = cc[wv + 4 * i];
          sw[i] = ss[wv + 4 * i];
        }
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          jp[i] = j[lane][pw[i]];
          jq[i] = j[lane][qw[i]];
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          // rows: (R1^T B) with R1 = [[c1, s1], [-s1, c1]] acting as p' = c p - s q, q' = s p + c q
          const double r00 = c1 * b00[i] - s1 * b10[i], r01 = c1 * b01[i] - s1 * b11[i];
          const double r10 = s1 * b00[i] + c1 * b10[i], r11 = s1 * b01[i] + c1 * b11[i];
          // then columns, the same rotation form with rotation w2
          a[p1][p2[i]] = c2[i] * r00 - s2[i] * r01;
          a[p1][q2[i]] = s2[i] * r00 + c2[i] * r01;
          a[q1][p2[i]] = c2[i] * r10 - s2[i] * r11;
          a[q1][q2[i]] = s2[i] * r10 + c2[i] * r11;
        }
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          j[lane][pw[i]] = cw[i] * jp[i] - sw[i] * jq[i];
          j[lane][qw[i]] = sw[i] * jp[i] + cw[i] * jq[i];
        }
      }
      __syncthreads();
    }
    const bool stop = rotated == 0;
    __syncthreads();
    if (stop) break;
  }
  double* out = Jout + (int64_t)pr * kLP * kLP;
  for (int e = threadIdx.x; e < kLP * kLP; e += kLT) out[e] = j[e >> 6][e & 63];
}

// 64 x 64 products, out[r][c] = sum_k L(r, k) R(k, c), on v_mfma_f64_16x16x4_f64: wave w computes
// rows 32 (w / 2) .. + 31 and columns 32 (w % 2) .. + 31 as 2 x 2 tiles of 16 x 16, 16 steps of 4
// along k. Operand layouts (from an in-bounds probe of the instruction): A[i][k] in lane i + 16 k,
// B[k][j] in lane j + 16 k, one double each; D[i][j] in lane j + 16 (i % 4), element i / 4. A
// lane reads 2 doubles from LDS per step for 4 instructions of 1024 multiply-adds (the
// thread-tiled VALU product read 8 per 16 multiply-adds).
typedef double d4_t __attribute__((ext_vector_type(4)));
// A rotation J (64 x 64, row-major, in global memory; a round's J are 2 MB and stay in L2) as the
// operand fragments of tile_mma_j, loaded into registers at once: f[s][t] = J[4 s + k][base + 16 t + i]
// for lane i + 16 k. With base = the wave's column start this is the B operand J; with the row
// start, the A operand J^T.
__device__ __forceinline__ void j_frags(const double* __restrict__ J, int base, double f[kLP / 4][2]) {
  const int lane = threadIdx.x & 63, i = lane & 15, kk = lane >> 4;
#pragma unroll
  for (int s = 0; s < kLP / 4; ++s)
#pragma unroll
    for (int t = 0; t < 2; ++t) f[s][t] = J[(4 * s + kk) * kLP + base + 16 * t + i];
}
// the product with one operand in registers (j_frags, f): L = m (LDS) times R = J, or (JL)
// L = J^T times R = m (LDS)
template <bool JL>
__device__ __forceinline__ void tile_mma_j(const double (*m)[kLPad], const double f[kLP / 4][2], d4_t acc[2][2]) {
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63, i = lane & 15, kk = lane >> 4;
  const int r0 = 32 * (w >> 1), c0 = 32 * (w & 1);
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b) acc[a][b] = d4_t{0.0, 0.0, 0.0, 0.0};
#pragma unroll
  for (int s = 0; s < kLP / 4; ++s) {
    const int k = 4 * s + kk;
    double x[2], y[2];
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      x[t] = JL ? f[s][t] : m[r0 + 16 * t + i][k];
      y[t] = JL ? m[k][c0 + 16 * t + i] : f[s][t];
    }
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
      for (int b = 0; b < 2; ++b) acc[a][b] = __builtin_amdgcn_mfma_f64_16x16x4f64(x[a], y[b], acc[a][b], 0, 0, 0);
  }
}
// the product's 64 x 64 result (tile_mma_j's layout) into s
__device__ __forceinline__ void tile_put(const d4_t acc[2][2], double (*s)[kLPad]) {
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int r0 = 32 * (w >> 1), c0 = 32 * (w & 1);
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int e = 0; e < 4; ++e) s[r0 + 16 * a + 4 * e + (lane >> 4)][c0 + 16 * b + (lane & 15)] = acc[a][b][e];
}

// G[pair a rows, pair c cols] <- J_a^T G[..] J_c for a <= c; the mirror block from the same result.
__global__ void __launch_bounds__(kLT)
k_lora_apply_g(double* __restrict__ G, int64_t dp, int nb, int t, const double* __restrict__ J) {
  const int pa = blockIdx.y, pc = blockIdx.x;
  if (pa > pc) return;
  // only the G tile lives in LDS (two blocks share a CU, so one's loads overlap the other's MFMAs);
  // the rotations come straight from L2 into registers, with the tile's loads
  __shared__ double g[kLP][kLPad];
  const int w = threadIdx.x >> 6;
  const double* Ja = J + (int64_t)pa * kLP * kLP;
  const double* Jc = J + (int64_t)pc * kLP * kLP;
  auto rows_a = [&](int r) { return pair_index(pa, t, nb, r); };
  auto rows_c = [&](int r) { return pair_index(pc, t, nb, r); };
  double fc[kLP / 4][2], fa[kLP / 4][2];
  j_frags(Jc, 32 * (w & 1), fc);
  j_frags(Ja, 32 * (w >> 1), fa);
  tile_load(G, dp, rows_a, pair_run(pc, t, nb, 0), pair_run(pc, t, nb, 1), g);
  __syncthreads();
  d4_t acc[2][2];
  tile_mma_j<false>(g, fc, acc);        // T = G J_c
  __syncthreads();
  tile_put(acc, g);
  __syncthreads();
  tile_mma_j<true>(g, fa, acc);         // J_a^T T
  __syncthreads();
  tile_put(acc, g);
  __syncthreads();
  tile_store<false>(G, dp, rows_a, pair_run(pc, t, nb, 0), pair_run(pc, t, nb, 1), g);
  if (pa != pc) tile_store<true>(G, dp, rows_c, pair_run(pa, t, nb, 0), pair_run(pa, t, nb, 1), g);
}

// V[row block, pair a cols] <- V[..] J_a
__global__ void __launch_bounds__(kLT)
k_lora_apply_v(double* __restrict__ V, int64_t dp, int nb, int t, const double* __restrict__ J) {
  const int pa = blockIdx.x;
  const int64_t r0 = (int64_t)blockIdx.y * kLP;
  __shared__ double v[kLP][kLPad];
  const int w = threadIdx.x >> 6;
  const double* Ja = J + (int64_t)pa * kLP * kLP;
  auto rows = [&](int r) { return r0 + r; };
  double fa[kLP / 4][2];
  j_frags(Ja, 32 * (w & 1), fa);
  tile_load(V, dp, rows, pair_run(pa, t, nb, 0), pair_run(pa, t, nb, 1), v);
  __syncthreads();
  d4_t acc[2][2];
  tile_mma_j<false>(v, fa, acc);        // V J_a
  __syncthreads();
  tile_put(acc, v);
  __syncthreads();
  tile_store<false>(V, dp, rows, pair_run(pa, t, nb, 0), pair_run(pa, t, nb, 1), v);
}

// ---------------------------------------------------------------- selection and adapters
// sel[rank] = i for the r largest diagonal entries of G (i < d; equal values: lower index first)
__global__ void __launch_bounds__(kLT)
k_lora_select(const double* __restrict__ G, int64_t dp, int64_t d, int64_t r, int* __restrict__ sel,
              double* __restrict__ lam) {
  const int64_t i = (int64_t)blockIdx.x * kLT + threadIdx.x;
  if (i >= d) return;
  const double li = G[i * dp + i];
  int64_t rank = 0;
  for (int64_t j = 0; j < d; ++j) {
    const double lj = G[j * dp + j];
    rank += (lj > li || (lj == li && j < i)) ? 1 : 0;
  }
  if (rank < r) {
    sel[rank] = (int)i;
    lam[rank] = li;
  }
}

// Vsel[k][c] = V[k][sel[c]] for k < d
__global__ void __launch_bounds__(kLT)
k_lora_gather(const double* __restrict__ V, int64_t dp, int64_t d, const int* __restrict__ sel, int64_t r,
              double* __restrict__ Vsel) {
  const int64_t e = (int64_t)blockIdx.x * kLT + threadIdx.x;
  if (e >= d * r) return;
  const int64_t k = e / r, c = e % r;
  Vsel[e] = V[k * dp + sel[c]];
}

// C[m][n] = sum_t P[t][m] Q[t][n]; P [T x M], Q [T x Nn] row-major, C [M x Nn]; 64 x 64 tiles
__global__ void __launch_bounds__(kLT)
k_lora_tgemm(const double* __restrict__ P, const double* __restrict__ Q, int64_t T, int64_t M, int64_t Nn,
             double* __restrict__ C) {
  __shared__ double ps[32][kLPad], qs[32][kLPad];
  const int64_t m0 = (int64_t)blockIdx.y * 64, n0 = (int64_t)blockIdx.x * 64;
  const int tr = threadIdx.x >> 4, tc = threadIdx.x & 15;
  double acc[4][4] = {};
  for (int64_t t0 = 0; t0 < T; t0 += 32) {
    for (int e = threadIdx.x; e < 32 * 64; e += kLT) {
      const int r = e >> 6, c = e & 63;
      const int64_t t = t0 + r;
      ps[r][c] = (t < T && m0 + c < M) ? P[t * M + m0 + c] : 0.0;
      qs[r][c] = (t < T && n0 + c < Nn) ? Q[t * Nn + n0 + c] : 0.0;
    }
    __syncthreads();
#pragma unroll 4
    for (int k = 0; k < 32; ++k) {
      double x[4], y[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        x[u] = ps[k][4 * tr + u];
        y[u] = qs[k][4 * tc + u];
      }
#pragma unroll
      for (int u = 0; u < 4; ++u)
#pragma unroll
        for (int v = 0; v < 4; ++v) acc[u][v] = fma(x[u], y[v], acc[u][v]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int u = 0; u < 4; ++u)
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int64_t m = m0 + 4 * tr + u, n = n0 + 4 * tc + v;
      if (m < M && n < Nn) C[m * Nn + n] = acc[u][v];
    }
}

// One block per component c: scale by sigma^(+-1/2) and -1/x, fix the sign (largest-magnitude entry
// of R's row positive, the first on equal magnitudes), write L [K x r] and R [r x N] in fp32.
// left: R row from C [r x N], L column from Vsel [K x r]; right: R row from Vsel [N x r], L column
// from C [K x r].
__global__ void __launch_bounds__(kLT)
k_lora_finalize(const double* __restrict__ lam, const double* __restrict__ Vsel, const double* __restrict__ C,
                const double* __restrict__ x, int64_t N, int64_t K, int64_t r, int left, float* __restrict__ L,
                float* __restrict__ R, double* __restrict__ sigma) {
  const int64_t c = blockIdx.x;
  const double sg = sqrt(fmax(lam[c], 0.0));
  const double sq = sqrt(sg);
  const double rs = sg > 0.0 ? 1.0 / sq : 0.0;       // sigma^(-1/2), zero for a null component
  auto rval = [&](int64_t n) -> double { return left ? C[c * N + n] * rs : Vsel[n * r + c] * sq; };
  auto lval = [&](int64_t k) -> double {
    const double v = left ? Vsel[k * r + c] * sq : C[k * r + c] * rs;
    return -(v / x[k]);
  };
  // argmax |R[c][n]|, first index on ties
  double best = -1.0;
  int64_t bi = 0;
  for (int64_t n = threadIdx.x; n < N; n += kLT) {
    const double v = fabs(rval(n));
    if (v > best) {
      best = v;
      bi = n;
    }
  }
  __shared__ double bv[kLT];
  __shared__ int64_t bx[kLT];
  bv[threadIdx.x] = best;
  bx[threadIdx.x] = bi;
  __syncthreads();
  for (int h = kLT / 2; h >= 1; h >>= 1) {
    if (threadIdx.x < h) {
      const double v2 = bv[threadIdx.x + h];
      const int64_t i2 = bx[threadIdx.x + h];
      if (v2 > bv[threadIdx.x] || (v2 == bv[threadIdx.x] && i2 < bx[threadIdx.x])) {
        bv[threadIdx.x] = v2;
        bx[threadIdx.x] = i2;
      }
    }
    __syncthreads();
  }
  const double sign = rval(bx[0]) < 0.0 ? -1.0 : 1.0;
  for (int64_t n = threadIdx.x; n < N; n += kLT) R[c * N + n] = (float)(sign * rval(n));
  for (int64_t k = threadIdx.x; k < K; k += kLT) L[k * r + c] = (float)(sign * lval(k));
  if (sigma && threadIdx.x == 0) sigma[c] = sg;
}

struct LoraPlan {
  int64_t d, D, dp, nb, chunks;
  bool left;
  size_t off_A, off_G, off_V, off_J, off_part, off_x, off_off, off_sel, off_lam, off_vsel, off_C, off_status, total;
};

inline size_t align256(size_t v) { return (v + 255) & ~(size_t)255; }

LoraPlan lora_plan(int64_t N, int64_t K, int64_t B, int64_t r) {
  LoraPlan p{};
  p.left = K <= N;
  p.d = p.left ? K : N;
  p.D = p.left ? N : K;
  p.dp = (p.d + kLP - 1) / kLP * kLP;
  p.nb = p.dp / kLB;
  p.chunks = (B + kLCalibRows - 1) / kLCalibRows;
  size_t o = 0;
  auto take = [&](size_t bytes) {
    const size_t at = o;
    o = align256(o + bytes);
    return at;
  };
  p.off_A = take(sizeof(double) * (size_t)p.d * p.D);
  p.off_G = take(sizeof(double) * (size_t)p.dp * p.dp);
  p.off_V = take(sizeof(double) * (size_t)p.dp * p.dp);
  p.off_J = take(sizeof(double) * (size_t)(p.nb / 2) * kLP * kLP);
  p.off_part = take(sizeof(double) * (size_t)(p.chunks * K > 2 * kLOffBlocks ? p.chunks * K : 2 * kLOffBlocks));
  p.off_x = take(sizeof(double) * (size_t)K);
  p.off_off = take(sizeof(double) * 2);
  p.off_sel = take(sizeof(int) * (size_t)(r > 0 ? r : 1));
  p.off_lam = take(sizeof(double) * (size_t)(r > 0 ? r : 1));
  p.off_vsel = take(sizeof(double) * (size_t)p.d * (r > 0 ? r : 1));
  p.off_C = take(sizeof(double) * (size_t)(r > 0 ? r : 1) * (N > K ? N : K));
  p.off_status = take(sizeof(int));
  p.total = o;
  return p;
}

}  // namespace

extern "C" int slim_lora_workspace(int64_t N, int64_t K, int64_t B, int64_t r, size_t* bytes) {
  if (!bytes) return SLIM_EINVAL;
  if (N < 16 || K < 128 || B < 1 || r < 0 || r > (N < K ? N : K)) return SLIM_ESHAPE;
  *bytes = lora_plan(N, K, B, r).total;
  return SLIM_OK;
}

extern "C" int slim_lora(const float* W, int64_t N, int64_t K, const uint8_t* codes, const uint8_t* meta,
                         const uint16_t* scales, const void* X, int xdtype, int64_t B, int64_t r, float* L, float* R,
                         double* sigma, int* sweeps, void* ws, size_t ws_bytes, void* stream) {
  if (!W || !codes || !meta || !scales || !X || !ws) return SLIM_EINVAL;
  if (r > 0 && (!L || !R)) return SLIM_EINVAL;
  if (xdtype != SLIM_F16 && xdtype != SLIM_BF16) return SLIM_EDTYPE;
  if (N < 16 || N % 16 || K < 128 || K % 128 || B < 1 || r < 0 || r > (N < K ? N : K)) return SLIM_ESHAPE;
  if (N * K >= ((int64_t)1 << 34) || B * K >= ((int64_t)1 << 40)) return SLIM_EUNSUPPORTED;
  if (!slim_aligned16(W) || !slim_aligned16(codes) || !slim_aligned16(meta) || !slim_aligned16(scales) ||
      !slim_aligned16(X) || !slim_aligned16(ws))
    return SLIM_EALIGN;
  const LoraPlan p = lora_plan(N, K, B, r);
  if (ws_bytes < p.total) return SLIM_EWORKSPACE;
  hipStream_t s = (hipStream_t)stream;
  char* base = static_cast<char*>(ws);
  double* A = reinterpret_cast<double*>(base + p.off_A);
  double* G = reinterpret_cast<double*>(base + p.off_G);
  double* V = reinterpret_cast<double*>(base + p.off_V);
  double* J = reinterpret_cast<double*>(base + p.off_J);
  double* part = reinterpret_cast<double*>(base + p.off_part);
  double* x = reinterpret_cast<double*>(base + p.off_x);
  double* offs = reinterpret_cast<double*>(base + p.off_off);
  int* sel = reinterpret_cast<int*>(base + p.off_sel);
  double* lam = reinterpret_cast<double*>(base + p.off_lam);
  double* vsel = reinterpret_cast<double*>(base + p.off_vsel);
  double* C = reinterpret_cast<double*>(base + p.off_C);
  int* status = reinterpret_cast<int*>(base + p.off_status);
  const uint32_t* codes32 = reinterpret_cast<const uint32_t*>(codes);
  const uint16_t* meta16 = reinterpret_cast<const uint16_t*>(meta);
  if (sweeps) *sweeps = 0;

  auto sync_status = [&](int* h) -> int {
    if (hipGetLastError() != hipSuccess) return SLIM_EDEVICE;
    if (hipMemcpyAsync(h, status, sizeof(int), hipMemcpyDeviceToHost, s) != hipSuccess ||
        hipStreamSynchronize(s) != hipSuccess)
      return SLIM_EDEVICE;
    return SLIM_OK;
  };
  // status word: cleared by a copy from the host (the call is synchronous anyway)
  const int zero = 0;
  if (hipMemcpyAsync(status, &zero, sizeof(int), hipMemcpyHostToDevice, s) != hipSuccess) return SLIM_EDEVICE;
  {
    SlimKernelTimer timer("lora_calib", s);
    SLIM_LAUNCH(timer, k_lora_calib, dim3((unsigned)((K + kLT - 1) / kLT), (unsigned)p.chunks), dim3(kLT), s,
                static_cast<const uint16_t*>(X), xdtype == SLIM_BF16 ? 1 : 0, B, K, part);
  }
  {
    SlimKernelTimer timer("lora_calib_final", s);
    SLIM_LAUNCH(timer, k_lora_calib_final, dim3(1), dim3(1024), s, (const double*)part, p.chunks, B, K, x, status);
  }
  int h_status = 0;
  int rc = sync_status(&h_status);
  if (rc != SLIM_OK) return rc;
  if (h_status & 2) return SLIM_ERANGE;
  if (r == 0) return SLIM_OK;
  {
    SlimKernelTimer timer("lora_error", s);
    SLIM_LAUNCH(timer, k_lora_error, dim3((unsigned)((K + 63) / 64), (unsigned)((N + 63) / 64)), dim3(kLT), s, W,
                codes32, meta16, scales, N, K, (const double*)x, p.left ? 1 : 0, A);
  }
  {
    SlimKernelTimer timer("lora_gram", s);
    const unsigned tiles = (unsigned)(p.dp / 64);
    SLIM_LAUNCH(timer, k_lora_gram, dim3(tiles, tiles), dim3(kLT), s, (const double*)A, p.D, p.d, p.dp, G);
  }
  {
    SlimKernelTimer timer("lora_eye", s);
    SLIM_LAUNCH(timer, k_lora_eye, dim3((unsigned)((p.dp * p.dp + kLT - 1) / kLT)), dim3(kLT), s, V, p.dp);
  }
  const int nb = (int)p.nb, npair = nb / 2;
  double prev = INFINITY;
  int done_sweeps = 0;
  bool converged = false;
  for (int sw = 0; sw <= kLMaxSweeps; ++sw) {
    {
      SlimKernelTimer timer("lora_offnorm", s);
      SLIM_LAUNCH(timer, k_lora_offnorm, dim3(kLOffBlocks), dim3(kLT), s, (const double*)G, p.dp, part);
    }
    {
      SlimKernelTimer timer("lora_offnorm_final", s);
      SLIM_LAUNCH(timer, k_lora_offnorm_final, dim3(1), dim3(64), s, (const double*)part, kLOffBlocks, offs);
    }
    double h_off[2];
    if (hipGetLastError() != hipSuccess ||
        hipMemcpyAsync(h_off, offs, sizeof(h_off), hipMemcpyDeviceToHost, s) != hipSuccess ||
        hipStreamSynchronize(s) != hipSuccess)
      return SLIM_EDEVICE;
    const double off = sqrt(h_off[0]), fro = sqrt(h_off[0] + h_off[1]);
    if (!(fro < INFINITY)) return SLIM_ENONFINITE;     // NaN or Inf in W or in the calibration input
    // converged, or stalled at rounding level
    if (!(off > 1e-13 * fro) || (off <= 1e-11 * fro && off > 0.25 * prev)) {
      converged = true;
      break;
    }
    if (sw == kLMaxSweeps) break;
    prev = off;
    ++done_sweeps;
    for (int t = 0; t < nb - 1; ++t) {
      {
        SlimKernelTimer timer("lora_pair_solve", s);
        SLIM_LAUNCH(timer, k_lora_pair_solve, dim3((unsigned)npair), dim3(kLT), s, (const double*)G, p.dp, nb, t, J);
      }
      {
        SlimKernelTimer timer("lora_apply_g", s);
        SLIM_LAUNCH(timer, k_lora_apply_g, dim3((unsigned)npair, (unsigned)npair), dim3(kLT), s, G, p.dp, nb, t,
                    (const double*)J);
      }
      {
        SlimKernelTimer timer("lora_apply_v", s);
        SLIM_LAUNCH(timer, k_lora_apply_v, dim3((unsigned)npair, (unsigned)(p.dp / kLP)), dim3(kLT), s, V, p.dp, nb, t,
                    (const double*)J);
      }
    }
  }
  if (sweeps) *sweeps = done_sweeps;
  if (!converged) return SLIM_EUNSUPPORTED;
  {
    SlimKernelTimer timer("lora_select", s);
    SLIM_LAUNCH(timer, k_lora_select, dim3((unsigned)((p.d + kLT - 1) / kLT)), dim3(kLT), s, (const double*)G, p.dp,
                p.d, r, sel, lam);
  }
  {
    SlimKernelTimer timer("lora_gather", s);
    SLIM_LAUNCH(timer, k_lora_gather, dim3((unsigned)((p.d * r + kLT - 1) / kLT)), dim3(kLT), s, (const double*)V,
                p.dp, p.d, (const int*)sel, r, vsel);
  }
  {
    SlimKernelTimer timer("lora_tgemm", s);
    if (p.left)   // C [r x N] = Vsel^T A, Vsel [K x r], A [K x N]
      SLIM_LAUNCH(timer, k_lora_tgemm, dim3((unsigned)((N + 63) / 64), (unsigned)((r + 63) / 64)), dim3(kLT), s,
                  (const double*)vsel, (const double*)A, K, r, N, C);
    else          // C [K x r] = A^T Vsel, A [N x K], Vsel [N x r]
      SLIM_LAUNCH(timer, k_lora_tgemm, dim3((unsigned)((r + 63) / 64), (unsigned)((K + 63) / 64)), dim3(kLT), s,
                  (const double*)A, (const double*)vsel, N, K, r, C);
  }
  {
    SlimKernelTimer timer("lora_finalize", s);
    SLIM_LAUNCH(timer, k_lora_finalize, dim3((unsigned)r), dim3(kLT), s, (const double*)lam, (const double*)vsel,
                (const double*)C, (const double*)x, N, K, r, p.left ? 1 : 0, L, R, sigma);
  }
  rc = sync_status(&h_status);
  return rc;
}
