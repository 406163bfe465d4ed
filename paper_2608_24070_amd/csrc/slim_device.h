// slim_device.h - device-side helpers shared by the libslim kernels (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

typedef _Float16 h2_t __attribute__((ext_vector_type(2)));
typedef _Float16 h8_t __attribute__((ext_vector_type(8)));
typedef _Float16 h16_t __attribute__((ext_vector_type(16)));
typedef float f4_t __attribute__((ext_vector_type(4)));
typedef float f16_t __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));

#define SLIM_DEV __device__ __forceinline__

SLIM_DEV uint32_t bits_of(h2_t x) { return __builtin_bit_cast(uint32_t, x); }
SLIM_DEV h2_t h2_of(uint32_t x) { return __builtin_bit_cast(h2_t, x); }

// Packed operand layout (codes, index words, scales of a forward pack; codesT, metaT of a
// backward pack): rows in blocks of 16, the reduction in chunks of 128. Row r, chunk c owns slot
//   packed_slot(r, c) = ((r / 16) * nch + c) * 16 + r % 16,   nch = red / 128,
// i.e. 8 code words (32 B) at u32 index 8 slot, 8 index half-words (16 B) at u16 index 8 slot
// and one fp16 scale at index slot: a block of 16 rows keeps each chunk's codes (512 B), index
// words (256 B) and scales (32 B) contiguous, so loads of one chunk for many rows coalesce.
SLIM_DEV int64_t packed_slot(int64_t r, int64_t c, int64_t nch) { return ((r >> 4) * nch + c) * 16 + (r & 15); }

// s_waitcnt immediate (gfx9 layout) waiting for at most n outstanding vector-memory operations:
// vmcnt bits [3:0] and [15:14]; expcnt [6:4] and lgkmcnt [11:8] left at their maxima (no wait)
constexpr unsigned vmcnt_wait(int n) { return (unsigned)(n & 15) | ((unsigned)(n >> 4) << 14) | 0x0F70u; }
// the same with lgkmcnt 0: also every LDS read of this wave has returned
constexpr unsigned vmcnt_lgkm0_wait(int n) { return vmcnt_wait(n) & ~0x0F00u; }

// Buffer resources: a wave-uniform base in scalar registers, a per-lane 32-bit byte offset (one
// vector register per address) and a uniform offset. A read at or past the resource's extent
// returns zero without touching memory.
typedef __amdgpu_buffer_rsrc_t rsrc_t;
constexpr int kRsrcWord3 = 0x00020000;   // gfx9 buffer descriptor word 3: raw 32-bit data
SLIM_DEV rsrc_t make_rsrc(const void* base, int64_t bytes) {
  const int64_t n = bytes < 0xFFFFFFFFll ? (bytes > 0 ? bytes : 0) : 0xFFFFFFFFll;
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, (int)(uint32_t)n, kRsrcWord3);
}
typedef __attribute__((address_space(3))) void* lds_ptr_t;

// Two fp16 copies of one fp16 bit pattern.
SLIM_DEV h2_t splat_h2(uint32_t hbits) { return h2_of((hbits & 0xFFFFu) | (hbits << 16)); }

// Constants of the nibble -> fp16 step, (x & mask) | 0x64006400. Kernels that dequantise in a
// hot loop make them opaque register values (nibble_consts_reg): with no literal to fold, the
// compiler forms one v_and_or_b32 per pair instead of an AND and an OR that each carry a literal.
struct NibbleConsts {
  uint32_t lo, hi, magic;
};
SLIM_DEV NibbleConsts nibble_consts() { return NibbleConsts{0x000F000Fu, 0x00F000F0u, 0x64006400u}; }
SLIM_DEV NibbleConsts nibble_consts_reg() {
  NibbleConsts k = nibble_consts();
  asm volatile("" : "+s"(k.lo), "+s"(k.hi), "+v"(k.magic));
  return k;
}

// One packed code word (16 K positions, four 2:4 groups) -> the eight kept values as the
// compressed A operand of a sparse MFMA: dword c = (first kept, second kept) of group c.
// Nibbles are turned into exact fp16 integers with the 1024-magic: (0x6400 | u) is 1024 + u,
// (0x6400 | 16u) is 1024 + 16u; both become u - 8 exactly. The scale multiply is the only
// rounding step: (u - 8) * s16 rounded to fp16.
SLIM_DEV h8_t dequant_word(uint32_t w, h2_t s2, const NibbleConsts& k = nibble_consts()) {
  const h2_t m1032 = {(_Float16)-1032.0f, (_Float16)-1032.0f};
  const h2_t r16 = {(_Float16)0.0625f, (_Float16)0.0625f};
  const h2_t m72 = {(_Float16)-72.0f, (_Float16)-72.0f};
  const uint32_t w8 = w >> 8;
  h2_t g0 = h2_of((w & k.lo) | k.magic) + m1032;
  h2_t g1 = h2_of((w & k.hi) | k.magic) * r16 + m72;
  h2_t g2 = h2_of((w8 & k.lo) | k.magic) + m1032;
  h2_t g3 = h2_of((w8 & k.hi) | k.magic) * r16 + m72;
  g0 = g0 * s2;
  g1 = g1 * s2;
  g2 = g2 * s2;
  g3 = g3 * s2;
  h8_t a;
  a[0] = g0[0]; a[1] = g0[1]; a[2] = g1[0]; a[3] = g1[1];
  a[4] = g2[0]; a[5] = g2[1]; a[6] = g3[0]; a[7] = g3[1];
  return a;
}

// Same without the scale: exact integers q = u - 8.
SLIM_DEV h8_t dequant_word_int(uint32_t w, const NibbleConsts& k = nibble_consts()) {
  const h2_t m1032 = {(_Float16)-1032.0f, (_Float16)-1032.0f};
  const h2_t r16 = {(_Float16)0.0625f, (_Float16)0.0625f};
  const h2_t m72 = {(_Float16)-72.0f, (_Float16)-72.0f};
  const uint32_t w8 = w >> 8;
  h2_t g0 = h2_of((w & k.lo) | k.magic) + m1032;
  h2_t g1 = h2_of((w & k.hi) | k.magic) * r16 + m72;
  h2_t g2 = h2_of((w8 & k.lo) | k.magic) + m1032;
  h2_t g3 = h2_of((w8 & k.hi) | k.magic) * r16 + m72;
  h8_t a;
  a[0] = g0[0]; a[1] = g0[1]; a[2] = g1[0]; a[3] = g1[1];
  a[4] = g2[0]; a[5] = g2[1]; a[6] = g3[0]; a[7] = g3[1];
  return a;
}

// ----------------------------------------------------------------------------------------------
// Per-row power-of-two scaling of activations. fp16 covers 2^-24 .. 65504, while bf16 activations
// and gradients (dY of order 1e-3 .. 1e-6, and dY times a weight scale of order 1e-2) can lie far
// outside it. Before a row of activations is rounded to fp16 it is multiplied by 2^e, with e chosen
// so that the row's largest magnitude lies in [2^kActExp, 2^(kActExp+1)); the fp32 results are
// multiplied by 2^-e. Both multiplications are exact (powers of two, normal fp32 range), so the
// only rounding is the one to fp16, now at full relative precision for every value within 2^-18
// of the row's largest. kActExp = 4 leaves 2^11 of headroom below fp16's maximum for fp16
// intermediates formed from the scaled rows (the adapter's X L, and the backward's dY s16 with
// scales below 2048).
// ----------------------------------------------------------------------------------------------
constexpr int kActExp = 4;

// 2^e as fp32, for e in [-126, 127] (built from the exponent field, so no rounding).
SLIM_DEV float exp2i(int e) { return __builtin_bit_cast(float, (uint32_t)(e + 127) << 23); }

// Scaling exponent for a row whose largest magnitude has fp32 bit pattern `maxbits` (sign
// cleared): kActExp - floor(log2(max)), clamped to [-126, 126] so that 2^e and 2^-e are normal.
// A zero row (and a non-finite maximum) gets 0.
SLIM_DEV int act_exponent(uint32_t maxbits) {
  const int E = (int)(maxbits >> 23);   // biased exponent; 0 for zero and fp32 subnormals
  if (maxbits == 0u || E == 255) return 0;
  const int e = kActExp - (E == 0 ? -127 : E - 127);
  return e < -126 ? -126 : (e > 126 ? 126 : e);
}

SLIM_DEV uint32_t abs_bits(float x) { return __builtin_bit_cast(uint32_t, x) & 0x7FFFFFFFu; }

// Largest value over the 64 lanes of a wave, returned wave-uniform: rotations within each row of
// 16 lanes (DPP row_ror 1, 2, 4, 8) leave every lane with its row's maximum, and the four rows'
// maxima are read into scalar registers.
SLIM_DEV uint32_t wave_max_u32(uint32_t v) {
  v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x121, 0xF, 0xF, false));
  v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x122, 0xF, 0xF, false));
  v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x124, 0xF, 0xF, false));
  v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x128, 0xF, 0xF, false));
  const uint32_t a = (uint32_t)__builtin_amdgcn_readlane((int)v, 0), b = (uint32_t)__builtin_amdgcn_readlane((int)v, 16);
  const uint32_t c = (uint32_t)__builtin_amdgcn_readlane((int)v, 32), d = (uint32_t)__builtin_amdgcn_readlane((int)v, 48);
  return max(max(a, b), max(c, d));
}

// Largest value over the four lanes L % 16 + {0, 16, 32, 48} (lanes that share a column of an
// MFMA operand), returned to each of them.
SLIM_DEV uint32_t col4_max_u32(uint32_t v) {
  v = max(v, (uint32_t)__shfl_xor((int)v, 16, 64));
  return max(v, (uint32_t)__shfl_xor((int)v, 32, 64));
}

// Eight fp32 values times s (a power of two), rounded to fp16.
SLIM_DEV h8_t scale8_to_h(const float* v, float s) {
  h8_t h;
#pragma unroll
  for (int e = 0; e < 8; ++e) h[e] = (_Float16)(v[e] * s);
  return h;
}

// Eight 16-bit activations (bf16 or fp16 bits in a uint4) as fp32 (exact).
SLIM_DEV void act8_to_f(u32x4_t v, bool is_bf16, float* f) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    if (is_bf16) {
      f[2 * i] = __builtin_bit_cast(float, v[i] << 16);
      f[2 * i + 1] = __builtin_bit_cast(float, v[i] & 0xFFFF0000u);
    } else {
      f[2 * i] = (float)__builtin_bit_cast(_Float16, (uint16_t)(v[i] & 0xFFFFu));
      f[2 * i + 1] = (float)__builtin_bit_cast(_Float16, (uint16_t)(v[i] >> 16));
    }
  }
}

SLIM_DEV uint32_t max_abs_bits8(const float* f) {
  uint32_t m = 0;
#pragma unroll
  for (int e = 0; e < 8; ++e) m = max(m, abs_bits(f[e]));
  return m;
}

// bf16 bits -> fp16 (through fp32; exact for |x| in [2^-14, 65504]).
SLIM_DEV _Float16 bf16_to_h(uint32_t b) { return (_Float16)__builtin_bit_cast(float, b << 16); }

// Eight 16-bit activations (bf16 or fp16 bits in a uint4) -> h8, optionally times an fp32 factor.
SLIM_DEV h8_t load8_as_h(u32x4_t v, bool is_bf16) {
  h8_t r;
  if (is_bf16) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      r[2 * i] = (_Float16)__builtin_bit_cast(float, v[i] << 16);
      r[2 * i + 1] = (_Float16)__builtin_bit_cast(float, v[i] & 0xFFFF0000u);
    }
  } else {
    r = __builtin_bit_cast(h8_t, v);
  }
  return r;
}

SLIM_DEV float h_bits_to_f(uint32_t hb) { return (float)__builtin_bit_cast(_Float16, (uint16_t)hb); }

SLIM_DEV float act_to_f(uint32_t b16, bool is_bf16) {
  return is_bf16 ? __builtin_bit_cast(float, b16 << 16) : h_bits_to_f(b16);
}

// ----------------------------------------------------------------------------------------------
// Sparse MFMA operand mapping on gfx950 (measured with one-hot probes of
// v_smfmac_f32_{16x16x64,32x32x32}_f16). NC = 16 or 32 output rows; G = 64 / NC lane groups.
//   A (compressed, 8 x fp16 per lane): lane (row lane % NC, group g = lane / NC) covers 16
//     consecutive dense reduction positions. Slot c is at position 4*(c/2) + idx_c, where
//     idx_c is bits [2c+1:2c] of the index VGPR with ABID 0, or bits [2c+17:2c+16] with ABID 1.
//   B (dense, 16 x fp16 per lane): lane (column lane % NC, group g). Element e pairs with A lane
//     group (g >> 1) + (e >> 3) * (G / 2), at position 8*(g & 1) + (e & 7) of that group's block.
//   C/D: the standard MFMA output layouts.
// One "chunk" is one 128-position quantisation group. Inside a chunk, A lane group g takes the
// 16-blocks {S*g + s} for steps s = 0..S-1 (S = 2 for 16x16x64, 4 for 32x32x32), so its code
// words and index half-words for the whole chunk are contiguous. B lane (g) then reads two runs of
// eight activations at chunk offsets c0 and c0 + 64, with c0 from b_chunk_offset.
// ----------------------------------------------------------------------------------------------
template <int NC>
SLIM_DEV int b_chunk_offset(int lane, int step) {
  if (NC == 16) {
    const int qb = lane >> 4;                       // 0..3
    return 32 * (qb >> 1) + 16 * step + 8 * (qb & 1);
  } else {
    const int hb = lane >> 5;                       // 0..1
    return 16 * step + 8 * hb;
  }
}

SLIM_DEV f4_t smfmac16(h8_t a, h16_t b, f4_t c, int idx, int abid) {
  if (abid == 0) return __builtin_amdgcn_smfmac_f32_16x16x64_f16(a, b, c, idx, 0, 0);
  return __builtin_amdgcn_smfmac_f32_16x16x64_f16(a, b, c, idx, 0, 1);
}

SLIM_DEV f16_t smfmac32(h8_t a, h16_t b, f16_t c, int idx, int abid) {
  if (abid == 0) return __builtin_amdgcn_smfmac_f32_32x32x32_f16(a, b, c, idx, 0, 0);
  return __builtin_amdgcn_smfmac_f32_32x32x32_f16(a, b, c, idx, 0, 1);
}

// ----------------------------------------------------------------------------------------------
// Cross-block hand-off of partial tiles. The partials are stored and loaded 16 bytes per lane with
// the sc1 cache policy, the one the compiler gives device-scope relaxed atomic loads and stores
// (coherent across the XCDs' separate L2s by themselves), so no L2-wide write-back or invalidate
// (what a device-scope fence costs) is needed. Before a block bumps the tile counter,
// s_waitcnt(0) makes sure its partial stores have completed.
// ----------------------------------------------------------------------------------------------
constexpr int kCpolSc1 = 16;   // buffer instruction cache-policy operand: sc1
SLIM_DEV void st_dev4(rsrc_t r, uint32_t off, f4_t v) {
  __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4_t, v), r, off, 0, kCpolSc1);
}
SLIM_DEV f4_t ld_dev4(rsrc_t r, uint32_t off) {
  return __builtin_bit_cast(f4_t, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, kCpolSc1));
}
SLIM_DEV void st_dev1(rsrc_t r, uint32_t off, uint32_t v) { __builtin_amdgcn_raw_buffer_store_b32(v, r, off, 0, kCpolSc1); }
SLIM_DEV uint32_t ld_dev1(rsrc_t r, uint32_t off) { return __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, kCpolSc1); }
SLIM_DEV void drain_stores() { __builtin_amdgcn_s_waitcnt(0); }
SLIM_DEV uint32_t counter_arrive(uint32_t* c) {
  return __hip_atomic_fetch_add(c, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
SLIM_DEV void counter_reset(uint32_t* c) { __hip_atomic_store(c, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT); }

SLIM_DEV f4_t mfma16(h8_t a, h8_t b, f4_t c) { return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0); }
SLIM_DEV f16_t mfma32(h8_t a, h8_t b, f16_t c) { return __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c, 0, 0, 0); }

SLIM_DEV h8_t zero_h8() {
  h8_t z;
#pragma unroll
  for (int e = 0; e < 8; ++e) z[e] = (_Float16)0.0f;
  return z;
}

SLIM_DEV h8_t mul_h8(h8_t x, h8_t s) {
  h8_t r;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    h2_t a = {x[2 * i], x[2 * i + 1]}, b = {s[2 * i], s[2 * i + 1]};
    a = a * b;
    r[2 * i] = a[0];
    r[2 * i + 1] = a[1];
  }
  return r;
}

SLIM_DEV h16_t cat16(h8_t lo, h8_t hi) {
  h16_t r;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    r[i] = lo[i];
    r[8 + i] = hi[i];
  }
  return r;
}
