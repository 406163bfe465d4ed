// api.cpp - status strings, version, argument checks, launch plans and workspace queries.
// Pure host code: nothing here touches the GPU, so these paths are testable without one.
#include <algorithm>

#include "slim_host.h"

namespace {
constexpr int64_t kMaxDim = int64_t(1) << 31;
constexpr int64_t kMaxLargeRed = int64_t(1) << 23;     // large M: longest reduction
constexpr int64_t kMaxTiledElems = int64_t(1) << 30;   // large M: M r and rows r (fp16, 32-bit byte offsets)
constexpr size_t kCounterSlots = SLIM_COUNTER_SLOTS;
constexpr int64_t kDecodeAdSlice = SLIM_DECODE_AD_SLICE;

int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }
size_t round256(size_t x) { return (x + 255) & ~size_t(255); }
}  // namespace

extern "C" const char* slim_status_string(int status) {
  switch (status) {
    case SLIM_OK: return "SLIM_OK";
    case SLIM_EINVAL: return "SLIM_EINVAL: null pointer or argument out of range";
    case SLIM_ESHAPE: return "SLIM_ESHAPE: size breaks a divisibility or range rule";
    case SLIM_EDTYPE: return "SLIM_EDTYPE: unsupported dtype";
    case SLIM_EALIGN: return "SLIM_EALIGN: device array not 16-byte aligned";
    case SLIM_ENONFINITE: return "SLIM_ENONFINITE: weight holds NaN or Inf";
    case SLIM_ERANGE: return "SLIM_ERANGE: group scale overflows fp16";
    case SLIM_EWORKSPACE: return "SLIM_EWORKSPACE: workspace missing or too small";
    case SLIM_EDEVICE: return "SLIM_EDEVICE: HIP runtime or launch failure";
    case SLIM_EUNSUPPORTED: return "SLIM_EUNSUPPORTED: valid but not supported by this library";
    default: return "unknown slim status";
  }
}

extern "C" int slim_abi_version(void) { return SLIM_ABI_VERSION; }

int slim_check_pack(const float* W, int64_t N, int64_t K, const void* codes, const void* meta,
                    const void* scales, const void* mask) {
  if (!W || !codes || !meta || !scales) return SLIM_EINVAL;
  if (N < 16 || K < 128 || N >= kMaxDim || K >= kMaxDim) return SLIM_ESHAPE;
  if (N % 16 || K % 128) return SLIM_ESHAPE;   // whole 16-row blocks and 128-wide chunks
  if (!slim_aligned16(W) || !slim_aligned16(codes) || !slim_aligned16(meta) || !slim_aligned16(scales) ||
      (mask && !slim_aligned16(mask)))
    return SLIM_EALIGN;
  return SLIM_OK;
}

int slim_check_pack_bwd(const void* codes, const void* meta, const void* scales, int64_t N, int64_t K,
                        const void* codesT, const void* metaT, const void* scalesT, const void* mask_rc) {
  if (!codes || !meta || !scales || !codesT || !metaT || !scalesT) return SLIM_EINVAL;
  if (N < 128 || K < 128 || N >= kMaxDim || K >= kMaxDim) return SLIM_ESHAPE;
  if (N % 128 || K % 128) return SLIM_ESHAPE;   // the transposed pack chunks N by 128
  if (!slim_aligned16(codes) || !slim_aligned16(meta) || !slim_aligned16(scales) || !slim_aligned16(codesT) ||
      !slim_aligned16(metaT) || !slim_aligned16(scalesT) || (mask_rc && !slim_aligned16(mask_rc)))
    return SLIM_EALIGN;
  return SLIM_OK;
}

int slim_make_plan(bool bwd, int64_t M, int64_t N, int64_t K, int64_t r, SlimPlan* p) {
  if (M < 1 || N < 16 || K < 128 || M >= kMaxDim || N >= kMaxDim || K >= kMaxDim) return SLIM_ESHAPE;
  if (N % 16 || K % 128 || r < 0 || r % 16 || r >= kMaxDim) return SLIM_ESHAPE;
  if (bwd && N % 128) return SLIM_ESHAPE;
  const int64_t rows = bwd ? K : N, red = bwd ? N : K;
  const int64_t nchunks = red / 128;
  SlimPlan q;
  size_t ad_counters = 0, tpart_bytes = 0, ypart_bytes = 0;
  if (M <= 32) {
    // small M: one launch of split-reduction sparse units plus adapter first-product units,
    // then the adapter's second product
    q.decode = true;
    q.dec_fm = M <= 16 ? 1 : 2;
    const int64_t mc = 16 * q.dec_fm;
    q.sp_rows_tile = 64;
    q.sp_cols_tile = (int)mc;
    q.sp_row_tiles = cdiv(rows, 64);
    q.sp_col_tiles = 1;
    // a sparse unit covers 4 * G quantisation groups of the reduction; two groups per lane group
    // when that still gives every CU a unit
    q.dec_g = (q.dec_fm == 1 && q.sp_row_tiles * cdiv(nchunks, 8) >= 256) ? 2 : 1;
    q.sp_chunks_per_split = 4 * q.dec_g;
    q.sp_split = (int)cdiv(nchunks, q.sp_chunks_per_split);
    // sparse blocks run several row tiles of one slice when there are more units than the target
    // block count (the backward's staged activations carry one 128-row group's scales: at most
    // the two row tiles of a group, starting at an even tile)
    const int64_t units = q.sp_row_tiles * q.sp_split;
    q.dec_units = (int)std::min<int64_t>(bwd ? 2 : SLIM_DECODE_MAX_UNITS, cdiv(units, SLIM_DECODE_BLOCKS));
    q.sp_blocks = cdiv(q.sp_row_tiles, q.dec_units) * q.sp_split;
    if (r > 0) {
      // adapter units: 16 ranks x 4 waves x ad_sub slices of SLIM_DECODE_AD_SLICE positions, at
      // most about SLIM_DECODE_AD_SPLITS splits (a wave takes several slices of a long reduction)
      q.ad_jblocks = cdiv(r, 16);
      const int64_t slices = cdiv(red, 4 * kDecodeAdSlice);
      q.ad_sub = (int)cdiv(slices, SLIM_DECODE_AD_SPLITS);
      q.ad_slice = 4 * kDecodeAdSlice * q.ad_sub;
      q.ad_split = (int)cdiv(slices, q.ad_sub);
      if (q.ad_split > 1) {
        ad_counters = (size_t)q.ad_jblocks;
        // per split and 16-row fragment: 256 fp32 partials and 16 row maxima
        tpart_bytes = (size_t)q.ad_jblocks * q.ad_split * q.dec_fm * 272 * 4;
      }
    }
    if (q.sp_split > 1 || r > 0) ypart_bytes = (size_t)q.sp_row_tiles * q.sp_split * 4 * q.dec_fm * 256 * 4;
    q.lds_bytes = 0;
  } else {
    // large M: dense adapter GEMM (128 x 128 tiles) then 512 x 96 or 512 x 128 sparse tiles. Their
    // per-lane buffer offsets are 32-bit: an activation offset spans up to 128 rows of the
    // reduction, and T and the adapter's second factor are addressed from their start.
    if (red > kMaxLargeRed || cdiv(M, 32) * 32 * r >= kMaxTiledElems || cdiv(rows, 32) * 32 * r >= kMaxTiledElems)
      return SLIM_EUNSUPPORTED;
    q.decode = false;
    q.sp_rows_tile = 512;
    q.sp_row_tiles = cdiv(rows, 512);
    // 512 x 128 tiles spend less dequantisation per MFMA (a tile takes about 1.12x the time of a
    // 512 x 96 one for 4/3 the work); 512 x 96 tiles are more and can fill the last round of
    // blocks (one per CU) better. Take the one with fewer rounds, weighted.
    const int64_t r96 = cdiv(q.sp_row_tiles * cdiv(M, 96), 256), r128 = cdiv(q.sp_row_tiles * cdiv(M, 128), 256);
    q.sp_cols_tile = 112 * r128 <= 100 * r96 ? 128 : 96;
    q.sp_col_tiles = cdiv(M, q.sp_cols_tile);
    q.sp_split = 1;
    q.sp_chunks_per_split = nchunks;
    // 256 x 256 adapter tiles (half the operand bytes per flop) with a 128 KiB ring, one block per
    // CU, when they fill the 256 CUs with reduction slices of at least 2048: the long reductions
    // at large M (the 70B dX product took 320 -> 253 us with its split sum; the 13B layers, whose
    // slices would be shorter or whose blocks too few, were slower); 256 rows of the reduction
    // stay within 32-bit byte offsets
    const int64_t wtiles = cdiv(M, 256) * (r / 256);
    const int64_t wsplit = wtiles > 0 ? std::max<int64_t>(1, std::min<int64_t>(256 / wtiles, red / 1024)) : 0;
    if (r > 0 && r % 256 == 0 && red < (int64_t(1) << 22) && wtiles * wsplit >= 256 && red / wsplit >= 2048) {
      q.ad_wide = true;
      q.ad_tiles_m = (int)cdiv(M, 256);
      q.ad_tiles_j = (int)(r / 256);
      const int64_t slice = cdiv(cdiv(red, wsplit), 32) * 32;
      q.ad_split = (int)cdiv(red, slice);
      q.ad_slice = slice;
      if (q.ad_split > 1) tpart_bytes = (size_t)q.ad_split * (size_t)cdiv(M, 32) * 32 * (size_t)r * 4;
    } else if (r > 0) {
      q.ad_tiles_m = (int)cdiv(M, 128);
      q.ad_tiles_j = (int)cdiv(r, 128);
      const int64_t tiles = (int64_t)q.ad_tiles_m * q.ad_tiles_j;
      // two blocks per CU (the GEMM's LDS ring takes 64 KB): at most 512 blocks, so one round
      const int64_t split = std::max<int64_t>(1, std::min<int64_t>(512 / tiles, red / 512));
      const int64_t slice = cdiv(cdiv(red, split), 64) * 64;
      q.ad_split = (int)cdiv(red, slice);
      q.ad_slice = slice;
      // split partials: fp32, one T-sized tiled array per split (summed by the next kernel)
      if (q.ad_split > 1) tpart_bytes = (size_t)q.ad_split * (size_t)cdiv(M, 32) * 32 * (size_t)r * 4;
    }
  }
  // workspace: [counters][adapter intermediate fp16 M x r][adapter partials][sparse partials]
  // [fp16 activations (large M)]
  q.n_counters = ad_counters;
  q.off_counters = 0;
  if (q.n_counters > kCounterSlots) return SLIM_EUNSUPPORTED;
  // the counter region has a fixed size so that it stays at zero across calls with other sizes
  size_t off = kCounterSlots * 4;
  // T (fp16, from row-scaled activations): row-major [M, r] at small M; at large M in 32 x 16 tiles
  // ([ceil(M/32)][r/16][32][16], see adapter_gemm.hip), which the tile kernel's epilogue reads 1 KB
  // at a time
  q.off_t = off;
  off = round256(off + (size_t)(q.decode ? M : cdiv(M, 32) * 32) * (size_t)r * 2);
  q.off_tpart = off;
  off = round256(off + tpart_bytes);
  q.off_ypart = off;
  off = round256(off + ypart_bytes);
  // large M: the row-scaled fp16 copy of the activations for the tile kernel's direct-to-LDS loads, and (backward:
  // the forward's factor comes tiled from slim_pack_adapter) the adapter's second factor P
  // [rows, r] re-laid in 32 x 16 tiles
  q.off_x16 = off;
  if (!q.decode) off = round256(off + (size_t)M * (size_t)red * 2);
  // 2^-e per activation row: large M, the rows of the fp16 copy are scaled by 2^e; small M, the
  // rows of T are
  q.off_rowinv = off;
  off = round256(off + (size_t)M * 4);
  q.off_pb = off;
  if (!q.decode && bwd) off = round256(off + (size_t)cdiv(rows, 32) * 32 * (size_t)r * 2);
  q.total = off;
  *p = q;
  return SLIM_OK;
}

int slim_check_linear(bool bwd, const void* X, int xdtype, int64_t M, int64_t N, int64_t K, const void* codes,
                      const void* meta, const void* scales, const void* L, const void* R, int64_t r, const void* Y,
                      const void* ws, size_t ws_bytes, SlimPlan* plan) {
  if (!X || !codes || !meta || !scales || !Y) return SLIM_EINVAL;
  if (r < 0) return SLIM_EINVAL;
  if (r == 0 ? (L != nullptr || R != nullptr) : (!L || !R)) return SLIM_EINVAL;
  if (xdtype != SLIM_F16 && xdtype != SLIM_BF16) return SLIM_EDTYPE;
  int st = slim_make_plan(bwd, M, N, K, r, plan);
  if (st != SLIM_OK) return st;
  if (!slim_aligned16(X) || !slim_aligned16(codes) || !slim_aligned16(meta) || !slim_aligned16(scales) ||
      !slim_aligned16(Y) || (L && !slim_aligned16(L)) || (R && !slim_aligned16(R)))
    return SLIM_EALIGN;
  if (!ws || ws_bytes < plan->total) return SLIM_EWORKSPACE;
  if (!slim_aligned16(ws)) return SLIM_EALIGN;
  plan->scaled = !plan->decode && (bwd || xdtype == SLIM_BF16 || r > 0);
  return SLIM_OK;
}

extern "C" int slim_linear_workspace(int64_t M, int64_t N, int64_t K, int64_t r, size_t* bytes) {
  if (!bytes) return SLIM_EINVAL;
  SlimPlan p;
  int st = slim_make_plan(false, M, N, K, r, &p);
  if (st == SLIM_OK) *bytes = p.total;
  return st;
}

extern "C" int slim_bwd_dx_workspace(int64_t M, int64_t N, int64_t K, int64_t r, size_t* bytes) {
  if (!bytes) return SLIM_EINVAL;
  SlimPlan p;
  int st = slim_make_plan(true, M, N, K, r, &p);
  if (st == SLIM_OK) *bytes = p.total;
  return st;
}

int slim_make_plan_qa(int64_t M, int64_t N, int64_t K, int64_t r, SlimPlan* p) {
  if (r < 32 || r % 32) return SLIM_ESHAPE;   // 4-bit factor rows are whole 16-byte runs
  int st = slim_make_plan(false, M, N, K, r, p);
  if (st != SLIM_OK) return st;
  if (!p->decode) {
    size_t off = p->total;
    p->off_q16 = off;
    off = round256(off + (size_t)r * (size_t)K * 2);
    p->off_p16 = off;
    off = round256(off + (size_t)cdiv(N, 32) * 32 * (size_t)r * 2);
    p->total = off;
  }
  return SLIM_OK;
}

int slim_check_linear_qa(const void* X, int xdtype, int64_t M, int64_t N, int64_t K, const void* codes,
                         const void* meta, const void* scales, const void* Lq, const void* Ls, const void* Rq,
                         const void* Rs, int64_t r, const void* Y, const void* ws, size_t ws_bytes, SlimPlan* plan) {
  if (!X || !codes || !meta || !scales || !Y || !Lq || !Ls || !Rq || !Rs) return SLIM_EINVAL;
  if (xdtype != SLIM_F16 && xdtype != SLIM_BF16) return SLIM_EDTYPE;
  int st = slim_make_plan_qa(M, N, K, r, plan);
  if (st != SLIM_OK) return st;
  if (!slim_aligned16(X) || !slim_aligned16(codes) || !slim_aligned16(meta) || !slim_aligned16(scales) ||
      !slim_aligned16(Y) || !slim_aligned16(Lq) || !slim_aligned16(Ls) || !slim_aligned16(Rq) || !slim_aligned16(Rs))
    return SLIM_EALIGN;
  if (!ws || ws_bytes < plan->total) return SLIM_EWORKSPACE;
  if (!slim_aligned16(ws)) return SLIM_EALIGN;
  plan->scaled = !plan->decode;
  return SLIM_OK;
}

extern "C" int slim_linear_qa_workspace(int64_t M, int64_t N, int64_t K, int64_t r, size_t* bytes) {
  if (!bytes) return SLIM_EINVAL;
  SlimPlan p;
  int st = slim_make_plan_qa(M, N, K, r, &p);
  if (st == SLIM_OK) *bytes = p.total;
  return st;
}
