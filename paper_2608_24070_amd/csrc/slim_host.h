// slim_host.h - host-side argument checks and launch planning for libslim (no device code).
#pragma once

#include <stddef.h>
#include <stdint.h>

#include "slim.h"

// Completion counters live in a fixed-size region at the start of the workspace.
#define SLIM_COUNTER_SLOTS 4096
// Reduction positions per load round of a wave of an adapter first-product unit of the small-M
// path, and the most reduction splits of that product (longer reductions give a wave several
// rounds).
#define SLIM_DECODE_AD_SLICE 128
#define SLIM_DECODE_AD_SPLITS 8
// Small-M forward: most row tiles one sparse block runs, and the block count it aims for.
#define SLIM_DECODE_MAX_UNITS 8
#define SLIM_DECODE_BLOCKS 512

// Argument checks: pure host functions, run before anything is enqueued.
int slim_check_pack(const float* W, int64_t N, int64_t K, const void* codes, const void* meta,
                    const void* scales, const void* mask);
int slim_check_pack_bwd(const void* codes, const void* meta, const void* scales, int64_t N, int64_t K,
                        const void* codesT, const void* metaT, const void* scalesT, const void* mask_rc);

// Which kernels one call runs and how its workspace is carved up.
struct SlimPlan {
  // dense adapter GEMM (T = X L forward, U = dY R^T backward)
  int ad_tiles_m = 0, ad_tiles_j = 0, ad_split = 1;
  bool ad_wide = false;                // large M: 256 x 256 adapter tiles (k_adapter_gemm_wide)
  int64_t ad_slice = 0;               // reduction length per split
  int ad_sub = 1;                      // small M: SLIM_DECODE_AD_SLICE slices per adapter wave
  int64_t ad_jblocks = 0;             // small-M path: 16-wide blocks of the adapter rank
  // sparse contraction
  bool decode = false;                // small-M kernel (16-column MFMA tiles, split reduction)
  int dec_fm = 1;                     // 16-column fragments per wave in the small-M kernel
  int dec_g = 1;                      // quantisation groups per lane group in a small-M sparse unit
  int sp_rows_tile = 0, sp_cols_tile = 0;  // output tile (rows of W or W^T, columns = M)
  int64_t sp_row_tiles = 0, sp_col_tiles = 0;
  int sp_split = 1;                   // reduction splits (small-M kernel only)
  int dec_units = 1;                  // small M: row tiles per sparse block
  int64_t sp_blocks = 0;              // small M: sparse blocks
  int64_t sp_chunks_per_split = 0;    // 128-wide chunks per split
  size_t lds_bytes = 0;               // dynamic LDS (unused: the kernels size their LDS statically)
  // large M: activations scaled per row into an fp16 copy (set by slim_check_linear: every
  // backward, bf16 activations, or an adapter; fp16 activations without one stream as given)
  bool scaled = false;
  // workspace layout (byte offsets)
  size_t off_counters = 0, n_counters = 0;
  size_t off_t = 0, off_tpart = 0, off_ypart = 0, off_x16 = 0, off_rowinv = 0, off_pb = 0, total = 0;
  // 4-bit adapters at large M: their fp16 expansions (Q = L^T row-major, P = R^T in 32 x 16 tiles)
  size_t off_q16 = 0, off_p16 = 0;
};

// Forward plan with 4-bit adapters (slim_linear_qa): slim_make_plan plus, at large M, room for the
// adapters' fp16 expansions.
int slim_make_plan_qa(int64_t M, int64_t N, int64_t K, int64_t r, SlimPlan* plan);
int slim_check_linear_qa(const void* X, int xdtype, int64_t M, int64_t N, int64_t K, const void* codes,
                         const void* meta, const void* scales, const void* Lq, const void* Ls, const void* Rq,
                         const void* Rs, int64_t r, const void* Y, const void* ws, size_t ws_bytes, SlimPlan* plan);

// Forward (bwd == false: rows = N, red = K) or backward (bwd == true: rows = K, red = N) plan.
int slim_make_plan(bool bwd, int64_t M, int64_t N, int64_t K, int64_t r, SlimPlan* plan);

int slim_check_linear(bool bwd, const void* X, int xdtype, int64_t M, int64_t N, int64_t K, const void* codes,
                      const void* meta, const void* scales, const void* L, const void* R, int64_t r, const void* Y,
                      const void* ws, size_t ws_bytes, SlimPlan* plan);

inline bool slim_aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }
