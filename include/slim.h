/*
 * slim.h - C ABI of libslim: the SLiM compressed linear layer on AMD Instinct MI355X (gfx950).
 *
 * The layer (thesis "Compression Trinity", SLiM chapter, section "Quantized sparse plus
 * low-rank approximation of LLMs"; SLoPe chapter, eq. sparse_plus_low_rank) is
 *
 *     Y = X * Wc^T + (X * L) * R,      Wc = dequant(Q(M (.) W))
 *
 * where M keeps two of every four consecutive weights along the reduction dimension K,
 * Q is symmetric AbsMax 4-bit quantisation per group of 128 weights of a row, and L*R is
 * a rank-r adapter kept as a parallel dense path. SLoPe's double-pruned input gradient
 * (SLoPe chapter, "Double-pruned Backward Pass", eq. sparse_backward_input) is
 *
 *     dX = dY * W^{R,C} + (dY * R^T) * L^T,
 *
 * where W^{R,C} is Wc pruned 2:4 a second time along N, so that the backward contraction is
 * sparse along its own reduction dimension too.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * Shapes: W is [N x K] (N output features, K input features), X is [M x K], Y is [M x N],
 * L is [K x r], R is [r x N], dY is [M x N], dX is [M x K]. Activations, outputs and the
 * adapter factors as given are dense row-major with no padding between rows; the packed
 * weights and the forward's adapter factors use the layouts below.
 *
 * Pointers: every array argument is a DEVICE pointer unless the comment says "host". The
 * caller allocates and owns every buffer, including workspace. The library never frees
 * anything and never keeps a pointer after a call returns.
 *
 * Alignment: device arrays must be 16-byte aligned.
 *
 * Streams: `stream` is a hipStream_t cast to void* (NULL = the null stream). Work is
 * enqueued on it; slim_linear and slim_linear_bwd_dx return without synchronising, and a
 * kernel fault shows up at the caller's next synchronisation of that stream.
 *
 * Errors: every entry point returns an slim_status. Argument checks run on the host before
 * anything is enqueued; when a check fails nothing is launched and the outputs are not
 * touched. No C++ exception crosses the ABI.
 *
 * Packed format (all multi-byte words little-endian)
 * --------------------------------------------------
 * Words. Per row and 16 consecutive reduction positions (four aligned 2:4 groups, g = 0..3):
 *   one code word (uint32): nibble g = u of group g's lower kept position, nibble g + 4 = u of
 *     its higher kept position, where u = q + 8 and q in [-7, 7] is the signed code;
 *   one index half-word (uint16): nibble g = i0 | i1 << 2, the kept offsets i0 < i1 (0..3).
 * Per row and 128 consecutive reduction positions (one quantisation group): one fp16 scale
 *   s16 = fp16_RNE(fp32(max |w| of the group) / 7).
 * The value of kept weight (n, k) is (u - 8) * s16[n, k / 128]; every other weight is zero.
 *
 * Layout. Rows are kept in blocks of 16 and the reduction in chunks of 128 (nch = reduction
 * length / 128). Row n, chunk c owns slot ((n / 16) * nch + c) * 16 + n % 16, which holds its 8
 * code words at bytes 32 slot .. 32 slot + 31 of `codes`, its 8 index half-words at bytes
 * 16 slot .. 16 slot + 15 of `meta` and its scale at element `slot` of `scales`:
 *   codes  uint8 [rows/16][nch][16][32], meta uint8 [rows/16][nch][16][16], scales fp16 [rows/16][nch][16].
 * One chunk of a 16-row block is thus contiguous (512 B of codes, 256 B of index words, 32 B of
 * scales). The forward pack has rows n and reduction k; the backward pack (codesT, metaT) has
 * rows k and reduction n, and its scales are scalesT fp16 [K/128][N] = s16[n, k/128].
 * 3.125 bits per dense weight (0.390625 bytes).
 *
 * Precision
 * ---------
 * Products accumulate in fp32 and Y / dX are fp32. Operands reach the matrix cores in fp16:
 *   - dequantised forward weights (u - 8) * s16, rounded to fp16 once;
 *   - activations (X, dY): each row of activations is multiplied by a power of two 2^e chosen
 *     so that its largest magnitude lies in [16, 32), rounded to fp16, and the fp32 results are
 *     multiplied by 2^-e (both exact), so bf16 inputs of any magnitude keep fp16's relative
 *     precision. At M <= 32 the exponent is chosen per slice of the reduction that one block
 *     or wave stages (at most 1024 positions); at M > 32 per whole row;
 *   - backward: the scale s16[n, k/128] multiplies the (row-scaled) gradient, and the product is
 *     rounded to fp16 once; the codes enter as exact small integers;
 *   - adapter: the first product (X L, or dY R^T) accumulates in fp32. At M <= 32 it stays fp32
 *     and is row-scaled into fp16 for the second product per pass of at most 512 ranks; at
 *     M > 32 it is formed from the row-scaled activations and stored in fp16, so its entries
 *     must stay below 65504 after that scaling: |T[m, j]| < 2^11 max_k |X[m, k]| (true when
 *     sum_k |L[k, j]| < 2^11).
 * Deterministic: identical inputs give identical bits.
 */
#ifndef SLIM_H
#define SLIM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SLIM_ABI_VERSION 2

typedef enum {
  SLIM_OK = 0,
  SLIM_EINVAL = 1,        /* a required pointer is NULL, or an argument is out of range */
  SLIM_ESHAPE = 2,        /* a size breaks a divisibility or range rule */
  SLIM_EDTYPE = 3,        /* unsupported dtype code */
  SLIM_EALIGN = 4,        /* a device array is not 16-byte aligned */
  SLIM_ENONFINITE = 5,    /* W holds a NaN or an infinity */
  SLIM_EWORKSPACE = 6,    /* workspace missing or smaller than the query returned */
  SLIM_EDEVICE = 7,       /* a HIP runtime call or a kernel launch failed */
  SLIM_EUNSUPPORTED = 8,  /* valid but not supported by this library (e.g. no gfx950 device) */
  SLIM_ERANGE = 9         /* a group scale the packed format or the backward cannot represent */
} slim_status;

/* Element types. Activations (X, dY) are SLIM_F16 or SLIM_BF16; Y and dX are always SLIM_F32. */
typedef enum { SLIM_F16 = 0, SLIM_BF16 = 1, SLIM_F32 = 2 } slim_dtype;

/* Human-readable name of a status code (static string, never NULL). */
const char* slim_status_string(int status);

/* SLIM_ABI_VERSION of the built library. */
int slim_abi_version(void);

/*
 * slim_pack - one-time forward pack of a dense fp32 weight.
 * Thesis: 2:4 magnitude pruning along the reduction dimension (SLoPe "Double-pruned Backward
 * Pass"; background "Sparse Tensor Core Acceleration"); symmetric AbsMax quantisation
 * (SLiM preliminaries, eq. symmetric_quantization) with groups of 128 (SLiM setup).
 *
 *   W       fp32 [N, K], device.
 *   N, K    N >= 16 and N % 16 == 0; K >= 128 and K % 128 == 0.
 *   codes   out, uint8 [N/16][K/128][16][32]; meta out, uint8 [N/16][K/128][16][16];
 *   scales  out, uint16 [N/16][K/128][16]. The packed layout keeps rows in blocks of 16 and K in
 *           chunks of 128: row n, chunk c (positions 128c .. 128c+127) owns slot
 *           ((n/16) * (K/128) + c) * 16 + n%16, holding 8 code words (uint32, little-endian;
 *           word i covers positions 16i .. 16i+15 of the chunk: the kept codes, as q + 8, of
 *           its four 2:4 groups, the first kept of group g in nibble g, the second in nibble
 *           g+4), 8 index
 *           half-words (uint16; nibble g = i0 | i1 << 2, the kept positions of group g) and one
 *           fp16 scale (the chunk is one quantisation group). The blocks keep one chunk of 16
 *           rows contiguous (512 B of codes, 256 B of indices, 32 B of scales).
 *   mask    out, optional (NULL to skip): uint8 [N, K], 1 where the weight is kept.
 * Mask rule: in each aligned group of four along K, keep the two largest |w|; on equal
 * magnitude the lower position wins (-0 and +0 are equal). Codes: q = clamp(rint(w / s16), -7, 7)
 * with the division done in double precision and ties rounded to even; q = 0 when s16 == 0.
 * Returns SLIM_ENONFINITE if W holds a NaN/Inf and SLIM_ERANGE if a scale overflows fp16; the
 * outputs are then unspecified. This call synchronises `stream` (it reads back a status word)
 * and allocates 4 bytes of device memory for that word for the duration of the call.
 */
int slim_pack(const float* W, int64_t N, int64_t K, uint8_t* codes, uint8_t* meta,
              uint16_t* scales, uint8_t* mask, void* stream);

/*
 * slim_pack_bwd - one-time backward pack: prune the packed forward weight a second time,
 * 2:4 along N, for the transposed contraction of the input gradient.
 * Thesis: SLoPe "Double-pruned Backward Pass" (W^{R,C}, eq. sparse_backward_input; Lemma
 * sparsity_ratio gives the extra zeros, 9.375% for 2:4).
 *
 *   codes, meta, scales   a forward pack of an [N, K] weight (from slim_pack), device.
 *   N, K                  N >= 128 and N % 128 == 0; K % 128 == 0.
 *   codesT  out, uint8 [K/16][N/128][16][32]; metaT out, uint8 [K/16][N/128][16][16]: the packed
 *           layout of slim_pack with rows k and reduction n (W^{R,C} transposed, pruned 2:4
 *           along n). scalesT out, uint16 [K/128, N]: s16[n, k/128] by 128-group of k.
 *   mask_rc out, optional (NULL to skip): uint8 [N, K], 1 on the support of W^{R,C}.
 * Rule: for each column k and aligned group of four rows, keep two slots ranked by
 * (|Wc| descending, forward-kept descending, row ascending). A kept slot carries its forward
 * code (8, i.e. zero, if the forward mask had dropped it).
 * Returns SLIM_ERANGE if a forward scale is 2048 or more (a group max |w| of about 14336): the
 * M > 32 backward forms dY * s16 in fp16 from row-scaled gradients below 32, which would overflow.
 * The outputs are then unspecified. This call synchronises `stream` (it reads back a status word)
 * and allocates 4 bytes of device memory for that word for the duration of the call.
 */
int slim_pack_bwd(const uint8_t* codes, const uint8_t* meta, const uint16_t* scales, int64_t N,
                  int64_t K, uint8_t* codesT, uint8_t* metaT, uint16_t* scalesT, uint8_t* mask_rc,
                  void* stream);

/*
 * slim_pack_adapter - one-time layout of the adapter factors for slim_linear.
 * Thesis: the rank-r adapter W ~ W^C + L R (SLiM "SLiM-LoRA low-rank adapters"); like the weight
 * pack (set up once, multiply many times), this runs once per layer. The forward reads L along
 * K for each rank (X L) and R along the rank for each output row (T R), so it takes L^T
 * row-major and R^T in tiles of 32 rows x 16 ranks; re-laying them inside every slim_linear call
 * would add a launch and 4 r (K + N) bytes of traffic per call. The backward
 * (slim_linear_bwd_dx) reads L and R as given.
 *
 *   L    fp16 [K, r], device.     R    fp16 [r, N], device.
 *   K, N >= 1; r >= 16, r % 16 == 0.
 *   Lt   out, fp16 [r, K] = L^T, row-major.
 *   Rt   out, fp16 R^T in 32 x 16 tiles: ceil(N/32) * 32 * r elements, element (n, j) of R^T at
 *        ((n / 32) * (r / 16) + j / 16) * 512 + (n % 32) * 16 + j % 16; rows n >= N of the last
 *        tile are zero. One tile is 1 KiB of contiguous memory, the unit the kernels load.
 * Asynchronous on `stream`; a pure data movement (bit-exact).
 */
int slim_pack_adapter(const uint16_t* L, const uint16_t* R, int64_t K, int64_t N, int64_t r, uint16_t* Lt,
                      uint16_t* Rt, void* stream);

/*
 * slim_pack_adapter_q - one-time 4-bit pack of the adapter factors for slim_linear_qa.
 * Thesis: SLiM "Low-rank adapter quantization" (SLiM-LoRA^Q): AbsMax group quantization of the
 * adapters with groups of 128 elements, which cuts their bytes about 4x. The groups run along each
 * factor's input dimension: L^T [r, K] by rows j along K (the reduction of X L) and R^T [N, r] by
 * rows n along r (the reduction of T R); a row's last group holds r % 128 elements when 128 does
 * not divide r. Scale and codes follow the weights' rules: s16 = fp16_RNE(fp32(max |a|) / 7),
 * q = clamp(rint(a / s16), -7, 7) (double-precision division, ties to even; 0 when s16 == 0).
 *
 *   L    fp16 [K, r], device.     R    fp16 [r, N], device.
 *   K % 128 == 0, N >= 1, r >= 32 and r % 32 == 0.
 *   Lq   out, uint8 [r, K/2]: row j holds the codes u = q + 8 of L[:, j], 8 consecutive elements
 *        per little-endian 32-bit word, element 2c in nibble c and element 2c + 1 in nibble c + 4.
 *   Ls   out, fp16 bits [r, ceil(K/128)].
 *   Rq   out, uint8 [N, r/2]: row n holds the codes of R[:, n], same word format.
 *   Rs   out, fp16 bits [N, ceil(r/128)].
 * Bytes: r (K + N) / 2 codes plus 2 (r ceil(K/128) + N ceil(r/128)) scales (4.125 bits per element
 * when 128 divides both). Returns SLIM_ENONFINITE if L or R holds a NaN/Inf. Synchronises `stream`
 * (status read back) and allocates 4 bytes of device memory for the duration of the call.
 */
int slim_pack_adapter_q(const uint16_t* L, const uint16_t* R, int64_t K, int64_t N, int64_t r, uint8_t* Lq,
                        uint16_t* Ls, uint8_t* Rq, uint16_t* Rs, void* stream);

/*
 * slim_linear_workspace - bytes of device workspace slim_linear needs for these sizes
 * (written to *bytes, host pointer). Depends only on the sizes. Pure host function.
 */
int slim_linear_workspace(int64_t M, int64_t N, int64_t K, int64_t r, size_t* bytes);

/*
 * slim_bwd_dx_workspace - bytes of device workspace slim_linear_bwd_dx needs. Pure host function.
 */
int slim_bwd_dx_workspace(int64_t M, int64_t N, int64_t K, int64_t r, size_t* bytes);

/*
 * slim_workspace_init - zero a workspace before its first use (its leading control words must
 * start at zero; every successful call leaves them at zero again). Asynchronous on `stream`.
 */
int slim_workspace_init(void* ws, size_t ws_bytes, void* stream);

/*
 * slim_linear - Y = X * Wc^T + (X * L) * R, fp32 accumulation, fp32 output.
 * Thesis: SLiM "SLiM-LoRA low-rank adapters" (W ~ W^C + L R) and SLoPe eq. sparse_plus_low_rank
 * with the adapter as a parallel path; the adapter product is fused into the same kernels.
 *
 *   X       [M, K] in `xdtype` (SLIM_BF16 or SLIM_F16), device.
 *   M, N, K M >= 1, N >= 16, N % 16 == 0, K % 128 == 0.
 *   codes, meta, scales   forward pack of W (slim_pack).
 *   Lt, Rt  the adapter laid out by slim_pack_adapter: Lt fp16 [r, K] = L^T row-major, Rt fp16 R^T
 *           in 32 x 16 tiles (a plain row-major R^T gives wrong results); both NULL when
 *           r == 0. r % 16 == 0.
 *   Y       out, fp32 [M, N]. Must not alias any input.
 *   ws      device workspace of at least slim_linear_workspace(M, N, K, r) bytes, zeroed once
 *           with slim_workspace_init before its first use. Two calls that overlap in time must
 *           not share a workspace.
 * Sizes past the kernels' 32-bit offsets return SLIM_EUNSUPPORTED: for M > 32, K above 2^23, or
 * ceil(M/32)*32*r or ceil(N/32)*32*r of 2^30 or more.
 * Operand precision: see "Precision" above (row-scaled fp16 activations, fp16 dequantised
 * weights, fp32 accumulation). Deterministic: identical inputs give identical bits.
 */
int slim_linear(const void* X, int xdtype, int64_t M, int64_t N, int64_t K, const uint8_t* codes,
                const uint8_t* meta, const uint16_t* scales, const uint16_t* Lt, const uint16_t* Rt,
                int64_t r, float* Y, void* ws, size_t ws_bytes, void* stream);

/*
 * slim_linear_qa - Y = X * Wc^T + (X * L^Q) * R^Q with the 4-bit adapters of slim_pack_adapter_q
 * (L^Q, R^Q their dequantized values (u - 8) * s16). Thesis: SLiM-LoRA^Q, the quantized adapters of
 * SLiM's deployed layer ("Low-rank adapter quantization"; quantized-adapter rows of the SLiM
 * results and speedup tables).
 *
 *   Arguments as slim_linear, with Lq, Ls, Rq, Rs in place of Lt, Rt; r >= 32, r % 32 == 0.
 *   ws      at least slim_linear_qa_workspace(M, N, K, r) bytes, zeroed once with slim_workspace_init.
 * At M <= 32 the kernels dequantize the factors in registers as they stream them; at M > 32 the
 * first launch expands them to fp16 in the workspace. The dequantized factor values are
 * (u - 8) * s16 rounded to fp16 (as for the weights); otherwise precision as slim_linear.
 */
int slim_linear_qa_workspace(int64_t M, int64_t N, int64_t K, int64_t r, size_t* bytes);
int slim_linear_qa(const void* X, int xdtype, int64_t M, int64_t N, int64_t K, const uint8_t* codes,
                   const uint8_t* meta, const uint16_t* scales, const uint8_t* Lq, const uint16_t* Ls,
                   const uint8_t* Rq, const uint16_t* Rs, int64_t r, float* Y, void* ws, size_t ws_bytes,
                   void* stream);

/*
 * slim_linear_bwd_dx - dX = dY * W^{R,C} + (dY * R^T) * L^T, fp32 accumulation, fp32 output.
 * Thesis: SLoPe eq. sparse_backward_input (BWD-2 with the double-pruned weight) plus the adapter
 * path's input gradient.
 *
 *   dY      [M, N] in `dydtype` (SLIM_BF16 or SLIM_F16), device.
 *   M, N, K M >= 1, N % 16 == 0, K % 128 == 0.
 *   codesT, metaT, scalesT   backward pack (slim_pack_bwd).
 *   L, R    fp16 [K, r] and [r, N]; both NULL when r == 0. r % 16 == 0.
 *   dX      out, fp32 [M, K].
 *   ws      workspace of at least slim_bwd_dx_workspace(M, N, K, r) bytes, zeroed once.
 * Sizes past the kernels' 32-bit offsets return SLIM_EUNSUPPORTED: for M > 32, N above 2^23, or
 * ceil(M/32)*32*r or ceil(K/32)*32*r of 2^30 or more.
 * Operand precision: the weight codes enter the matrix cores as exact small integers; the fp16
 * scale s16[n, k/128] multiplies the row-scaled gradient and the product is rounded to fp16 once
 * (see "Precision" above). Deterministic.
 */
int slim_linear_bwd_dx(const void* dY, int dydtype, int64_t M, int64_t N, int64_t K,
                       const uint8_t* codesT, const uint8_t* metaT, const uint16_t* scalesT,
                       const uint16_t* L, const uint16_t* R, int64_t r, float* dX, void* ws,
                       size_t ws_bytes, void* stream);

/*
 * slim_linear_noalloc - slim_linear without a caller workspace, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, harnesses that forbid
 * allocation). Same arguments, results and precision as slim_linear, minus ws / ws_bytes.
 *
 * The workspace is a fixed array of SLIM_NOALLOC_SCRATCH_BYTES (64 MiB) of device memory that the
 * library holds per device from the first call on that device until the process ends; its first
 * call on a device also enqueues a small kernel that clears the array's counter region. The call
 * allocates nothing (no hipMalloc, hipFree or allocating library routine) and records no timing
 * events. Sizes whose slim_linear_workspace exceeds SLIM_NOALLOC_SCRATCH_BYTES return
 * SLIM_EWORKSPACE before touching any device; that covers every M <= 32 layer of the shapes here
 * and the 11008 x 4096 layer at M = 2048, but not, for example, a 5120 x 5120 layer at M = 4096.
 * All calls on one device share its array, so two calls that overlap in time on one device
 * (different streams or threads) race and give undefined results; serialise them.
 */
#define SLIM_NOALLOC_SCRATCH_BYTES (64u << 20)
int slim_linear_noalloc(const void* X, int xdtype, int64_t M, int64_t N, int64_t K, const uint8_t* codes,
                        const uint8_t* meta, const uint16_t* scales, const uint16_t* Lt, const uint16_t* Rt,
                        int64_t r, float* Y, void* stream);

/*
 * ---- The rest of SLoPe's sparse training step (SLoPe, Alg. "Accelerated Sparse Pretraining
 * Algorithm for a Linear Layer": setup of the sparse weight and its transpose, the weight gradient
 * with the weight's mask, the sparse add of the optimizer with weight decay, and the update of both
 * sparse matrices; appendix "Implementation details"). Training weights are kept in half precision,
 * so these calls work on value packs instead of the int4 inference pack:
 *
 *   vals   fp16 bits [rows, len/2], row-major: for aligned group g of four positions of a row,
 *          the values at its two kept positions, the lower position first (2g, 2g + 1);
 *   meta   uint8 [rows, len/8], row-major, the inference pack's index format (little-endian
 *          half-word b covers positions 16b .. 16b+15; its group c holds the kept offsets
 *          i0 < i1 in bits 4c..4c+1 and 4c+2..4c+3).
 *
 * The forward pack of W^R has rows = N, len = K (2:4 along K); its transposed pack W^{R,C} has
 * rows = K, len = N (2:4 along N). Every pointer is device memory, 16-byte aligned, owned by the
 * caller; every call enqueues on `stream` and returns after the launch unless stated otherwise.
 * ----
 *
 * slim_pack16 - setup of W^R from fp32 W [N, K] (row-major): per aligned group of four along K,
 * keep the two largest |w| (ties: lower position), store them rounded to fp16 (nearest, ties to
 * even) in vals [N, K/2] with meta [N, K/8]; mask (optional, uint8 [N, K], 0/1) receives M^R.
 * K % 16 == 0. Synchronous (reads back a status word): SLIM_ENONFINITE if W holds a NaN or Inf.
 */
int slim_pack16(const float* W, int64_t N, int64_t K, uint16_t* vals, uint8_t* meta, uint8_t* mask,
                void* stream);

/*
 * slim_pack16_t - W^{R,C} from a W^R value pack (SLoPe eq. sparse_backward_input's double
 * pruning): for each column k and aligned group of four rows, keep the two entries ranked first by
 * (|v| descending, M^R bit descending, row ascending) and store them (0 for a kept slot M^R had
 * dropped) in valsT [K, N/2] with metaT [K, N/8]. Run at setup and after every update of vals.
 * N % 64 == 0 and K % 64 == 0; the values must be finite.
 */
int slim_pack16_t(const uint16_t* vals, const uint8_t* meta, int64_t N, int64_t K, uint16_t* valsT,
                  uint8_t* metaT, void* stream);

/*
 * slim_grad_w - BWD-1 with the weight's mask (SLoPe eq. sparse_backward_weight and "pruneAndCompress"):
 * gW [N, K/2] fp32 = (dY^T X) at the positions meta (M^R, [N, K/8]) keeps, in the value-pack order.
 * dY [M, N] and X [M, K] row-major, both of `dtype` (SLIM_F16 or SLIM_BF16); products exact in
 * fp32, accumulated in fp32 along M (the order differs from a sequential sum). N % 128 == 0,
 * K % 128 == 0, M >= 1; SLIM_EUNSUPPORTED if M N or M K reaches 2^31 elements.
 */
int slim_grad_w(const void* dY, const void* X, int dtype, int64_t M, int64_t N, int64_t K, const uint8_t* meta,
                float* gW, void* stream);

/*
 * slim_sparse_add - out = beta A + gamma B on `count` compressed values sharing one pattern ("sparseAdd":
 * in the training step, A the masked gradient with beta = 1 / loss scale and B the weight values
 * with gamma = the weight decay). A and out fp32, B fp16 bits; computed in fp32 as
 * fma(gamma, B, beta A). count % 8 == 0; out may alias A.
 */
int slim_sparse_add(const float* A, const uint16_t* B, float beta, float gamma, float* out, int64_t count,
                    void* stream);

/*
 * slim_update_pack16 - write the optimizer's new compressed values Wnew (fp32, `count` of them, the
 * pack's order) into vals, rounded to fp16 (nearest, ties to even); the pattern (meta) is unchanged.
 * Follow with slim_pack16_t to rebuild the transposed pack ("updateSparseMatrix" on both).
 * count % 8 == 0.
 */
int slim_update_pack16(const float* Wnew, int64_t count, uint16_t* vals, void* stream);

/*
 * SLiM-Quant: one symmetric quantisation parameter alpha for a whole weight by minimising the
 * expected squared quantisation error over the distribution of |w| (SLiM chapter, "SLiM-Quant
 * quantization method": eq. error_summation = eq. quantization_error + eq. clipping_error,
 * integrated on a histogram of |w|; Alg. quantization for the candidate grids).
 *
 * slim_quant_bins - the histogram size of the SLiM setup, max(512, min(floor(N K / 1000), 20000)).
 *
 * slim_quant_search - histogram and search.
 *   W       fp32, `count` values (any shape, e.g. a weight [N, K]), device; count % 4 == 0,
 *           16-byte aligned.
 *   bits    quantiser width q, 2..8: codes in [-(2^(q-1) - 1), 2^(q-1) - 1], step alpha / (2^(q-1) - 1).
 *   bins    1..20480 equal bins over [0, max|w|]; |w| falls in bin floor(|w| bins / max|w|) (exact
 *           rational floor; the maximum in the last bin).
 *   hist    out, device uint32 [bins]: the counts.
 *   out     out, device float64 [4 + 2 * 30]: [0] alpha*, [1] E(alpha*), [2] max|w|, [3] the number C
 *           of candidates evaluated, then C pairs (alpha_i, E(alpha_i)) in evaluation order.
 * E(alpha) weighs each bin's count at its centre (b + 1/2) max|w| / bins: a centre c <= alpha
 * contributes (delta rint(c / delta) - c)^2 (delta = alpha / (2^(q-1) - 1), ties to even), one
 * above alpha (alpha - c)^2; E is their count-weighted mean, in float64. Candidates: i max|w| / 10
 * for i = 1..10, then (a - max|w| / 10) + j max|w| / 100 for j = 0..19 around the best of those, a,
 * the positive ones only; alpha* is the first candidate of least error. All-zero W gives alpha* = 0
 * and C = 0. Returns SLIM_ENONFINITE for NaN/Inf in W. This call synchronises `stream` (it reads
 * back a status word) and allocates under 4 KiB of device memory for the duration of the call.
 *
 * slim_pack_alpha - slim_pack with the per-tensor parameter in place of each group's absmax: every
 * group's scale is s16 = fp16_RNE(fp32(alpha) / 7.0f), so weights beyond alpha clip to +-7 (same
 * layout, mask rule, codes, status codes and synchronisation as slim_pack).
 *   alpha   device pointer to one float64 (e.g. `out` of slim_quant_search), 8-byte aligned;
 *           negative or NaN gives SLIM_ERANGE.
 */
int slim_quant_bins(int64_t N, int64_t K);
int slim_quant_search(const float* W, int64_t count, int bits, int64_t bins, uint32_t* hist, double* out,
                      void* stream);
int slim_pack_alpha(const float* W, int64_t N, int64_t K, const double* alpha, uint8_t* codes, uint8_t* meta,
                    uint16_t* scales, uint8_t* mask, void* stream);

/*
 * SLiM-LoRA: saliency-based low-rank adapters fitted to the compression error (SLiM chapter,
 * "SLiM-LoRA low-rank adapters": eq. lora_wanda_objective_function, eq. lora_svd, Alg. lora).
 *
 * slim_lora_workspace - bytes of workspace slim_lora needs for an [N, K] weight, B calibration rows
 * and rank r (float64 buffers: the saliency-weighted error, its d x d Gram matrix and eigenvectors,
 * d = min(N, K) rounded up to 64; about 8 (d max(N, K) + 2 d^2) bytes).
 *
 * slim_lora - the adapters.
 *   W                fp32 [N, K], device: the uncompressed weight.
 *   codes/meta/scales its forward pack (slim_pack or slim_pack_alpha), device: W^C.
 *   X, xdtype, B     calibration activations [B, K] (bf16 or fp16), device.
 *   r                rank, 0 <= r <= min(N, K).
 *   L, R             out, fp32 [K, r] and [r, N], device: W ~ W^C + (L R)^T, i.e. the layer's adapter.
 *   sigma            out, optional (NULL to skip): float64 [r], the r largest singular values of S.
 *   sweeps           out, optional host int: Jacobi sweeps run.
 *   ws, ws_bytes     workspace (slim_lora_workspace), 16-byte aligned; contents undefined after.
 * With x_k = mean_i |X[i, k]| + min_j mean_i |X[i, j]| (the per-channel mean input magnitude shifted
 * by its smallest value) and S = diag(x) (W^C - W)^T [K, N], L = -diag(1/x) U_r Sigma_r^(1/2) and
 * R = Sigma_r^(1/2) V_r^T from the r largest singular triplets of S (ties to the lower index of
 * the Gram side); each row of R has its largest-magnitude entry positive (the first on equal
 * magnitudes), L's column following. The singular vectors come from a float64 two-sided block-
 * Jacobi eigendecomposition (blocks of 32, one inner sweep per pair) of S S^T (K <= N) or S^T S
 * (N < K), run until the off-diagonal norm is
 * below 1e-13 of the Frobenius norm (or stalls at rounding level). Returns SLIM_ERANGE if some x_k is
 * zero (a channel that is zero in every sample and is the smallest), SLIM_ENONFINITE for NaN/Inf
 * inputs and SLIM_EUNSUPPORTED if 40 sweeps do not converge. Synchronises `stream` (the sweep loop
 * reads back the off-diagonal norm); allocates nothing.
 */
int slim_lora_workspace(int64_t N, int64_t K, int64_t B, int64_t r, size_t* bytes);
int slim_lora(const float* W, int64_t N, int64_t K, const uint8_t* codes, const uint8_t* meta,
              const uint16_t* scales, const void* X, int xdtype, int64_t B, int64_t r, float* L, float* R,
              double* sigma, int* sweeps, void* ws, size_t ws_bytes, void* stream);

/*
 * PATCH hybrid tiles: a weight whose 128 x 128 tiles are each dense or 2:4 sparse, in fp16, and its
 * product (PATCH chapter, "Efficient deployment of PATCH": hybrid sparse-dense tiles in one GEMM,
 * 128 x 128 as the tile size; appendix "STOICC Integration").
 *
 * slim_hybrid_layout - host-only: from the tile map `kinds` (host uint8 [N/128, K/128], row-major;
 *   1 = 2:4 sparse, 0 = dense) the payload size in bytes and, if tile_info (host) is not NULL, each
 *   tile's info word: its payload's byte offset, bit 63 set for a sparse tile. Payloads follow each
 *   other in row-major tile order: a dense tile is 128 rows x 128 fp16 (32768 bytes); a sparse tile
 *   is two halves (positions 0..63, then 64..127) of 9216 bytes: 128 rows x 32 fp16 kept values
 *   (group g of the half's 16 groups at 2g, 2g+1, the lower position first), then 128 rows x 4
 *   uint16 index half-words (half-word b covers the half's positions 16b .. 16b+15; group c holds
 *   i0 in bits 4c..4c+1 and i1 in bits 4c+2..4c+3); 18432 bytes.
 *   N, K multiples of 128.
 *
 * slim_pack_hybrid - one-time pack of fp32 W [N, K] (device) with the tile map `kinds` (host):
 *   writes tile_info (device uint64 [N/128, K/128]) and the payload (device, payload_bytes from
 *   slim_hybrid_layout). A sparse tile keeps the two largest |w| of every aligned group of four along
 *   K (the lower position on equal magnitude); all kept values are rounded to fp16 (nearest, ties to
 *   even). Returns SLIM_ENONFINITE for NaN/Inf in W; synchronises `stream` (status read-back) and
 *   allocates 4 bytes of device memory for the call.
 *
 * slim_linear_hybrid_workspace / slim_linear_hybrid - Y = X Wp^T.
 *   X          fp16 [M, K], device.            tile_info, payload   the hybrid pack, device;
 *                                              payload_bytes        its size, below 4 GiB.
 *   Y          out, fp32 [M, N], device.       ws, ws_bytes         workspace (split partials of
 *              small-M calls; 0 bytes when the call needs none), 16-byte aligned.
 * Dense tiles run on v_mfma_f32_32x32x16_f16, sparse tiles on v_smfmac_f32_32x32x32_f16 (half
 * the issue for the same K); fp32 accumulation; the split partials are summed in split order, so
 * results are deterministic. Asynchronous; allocates nothing.
 */
int slim_hybrid_layout(const uint8_t* kinds, int64_t N, int64_t K, uint64_t* tile_info, size_t* payload_bytes);
int slim_pack_hybrid(const float* W, int64_t N, int64_t K, const uint8_t* kinds, uint64_t* tile_info,
                     uint8_t* payload, size_t payload_bytes, void* stream);
int slim_linear_hybrid_workspace(int64_t M, int64_t N, int64_t K, size_t* bytes);
int slim_linear_hybrid(const void* X, int64_t M, int64_t N, int64_t K, const uint64_t* tile_info,
                       const uint8_t* payload, size_t payload_bytes, float* Y, void* ws, size_t ws_bytes,
                       void* stream);

/*
 * Per-kernel timing for benchmarks (host-side bookkeeping; not part of the layer's math).
 * slim_timing_enable(1) makes every later kernel launch of this library record a hipEvent
 * before and after itself on the caller's stream. slim_timing_read waits for the recorded
 * events and writes one line per kernel name, "name launches total_ms median_ms\n", into buf (host);
 * it returns 0, or the buffer size needed when buf is NULL or too small. slim_timing_reset
 * clears the totals. These three calls are the library's only process-wide mutable state (a
 * mutex-guarded switch, event pool and totals); with timing off, which is the default, the layer
 * calls read nothing of it but the switch. Thread-safe; timing adds two event records per launch
 * while enabled, and never records inside a stream capture.
 */
int slim_timing_enable(int on);
int slim_timing_reset(void);
int slim_timing_read(char* buf, size_t buf_len);

#ifdef __cplusplus
}
#endif
#endif /* SLIM_H */
