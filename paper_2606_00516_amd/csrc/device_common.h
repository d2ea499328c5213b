// Device helpers shared by the gfx950 kernels: bf16 conversion, wavefront
// reductions, MFMA operand types.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#define EB_DEV __device__ __forceinline__

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));

// bf16 bits <-> fp32.  Widening is exact; narrowing rounds to nearest even,
// NaN maps to a quiet NaN.
EB_DEV float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
EB_DEV float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }
EB_DEV float bf16_to_f32(uint16_t b) { return __uint_as_float(((uint32_t)b) << 16); }
EB_DEV uint32_t f32_to_bf16_bits(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7FFFFFFFu) > 0x7F800000u) return 0x7FC0u;
  return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}
EB_DEV uint32_t pack_bf16x2(float lo, float hi) { return f32_to_bf16_bits(lo) | (f32_to_bf16_bits(hi) << 16); }
// The same rounding (nearest even) by the hardware's packed conversion, one
// instruction for the pair.
EB_DEV uint32_t bf16_pair_rne(float lo, float hi) {
  typedef float f32x2_v __attribute__((ext_vector_type(2)));
  const f32x2_v f = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f, bf16x2_t));
}

// DPP row controls (a "row" is 16 lanes).
#define EB_DPP_QUAD_XOR1 0xB1   // quad_perm [1,0,3,2]
#define EB_DPP_QUAD_XOR2 0x4E   // quad_perm [2,3,0,1]
#define EB_DPP_ROW_HALF_MIRROR 0x141
#define EB_DPP_ROW_MIRROR 0x140

template <int CTRL>
EB_DEV float dpp_f32(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, true));
}

// Sum over aligned groups of LANES lanes (LANES in {8, 16}); every lane of the
// group receives the group sum.  Stays inside a 16-lane DPP row.
template <int LANES>
EB_DEV float group_sum(float v) {
  static_assert(LANES == 8 || LANES == 16, "group size");
  v += dpp_f32<EB_DPP_QUAD_XOR1>(v);
  v += dpp_f32<EB_DPP_QUAD_XOR2>(v);
  v += dpp_f32<EB_DPP_ROW_HALF_MIRROR>(v);
  if (LANES == 16) v += dpp_f32<EB_DPP_ROW_MIRROR>(v);
  return v;
}

EB_DEV float shfl_xor_f32(float v, int mask) { return __shfl_xor(v, mask, 64); }

EB_DEV float wave_max(float v) {
  for (int m = 32; m >= 1; m >>= 1) v = fmaxf(v, __shfl_xor(v, m, 64));
  return v;
}
EB_DEV float wave_sum(float v) {
  for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m, 64);
  return v;
}

EB_DEV u32x4_t ld_u32x4(const void *p) { return *reinterpret_cast<const u32x4_t *>(p); }
EB_DEV void st_u32x4(void *p, u32x4_t v) { *reinterpret_cast<u32x4_t *>(p) = v; }

// Non-temporal 16-byte global load (streamed data read exactly once).
EB_DEV u32x4_t ld_stream_u32x4(const void *p) {
  return __builtin_nontemporal_load(reinterpret_cast<const u32x4_t *>(p));
}

// Raw buffer access: a descriptor over [base, base + bytes); loads past the
// end return zero without touching memory, so a wave-uniform "no data"
// case needs no branch.  (Word 3 of the descriptor as gfx9 requires.)
typedef __amdgpu_buffer_rsrc_t buf_rsrc_t;
EB_DEV buf_rsrc_t make_rsrc(const void *base, int bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, bytes, 0x00020000);
}
// 16-byte load at byte offset `off`; AUX = 2 marks data read exactly once
// (non-temporal).
constexpr int kAuxNT = 2;
template <int AUX = 0>
EB_DEV u32x4_t buf_ld_u32x4(buf_rsrc_t r, int off) {
  return __builtin_bit_cast(u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, AUX));
}

// 8-byte load at byte offset `off` (same conventions).
template <int AUX = 0>
EB_DEV u32x2_t buf_ld_u32x2(buf_rsrc_t r, int off) {
  return __builtin_bit_cast(u32x2_t, __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, AUX));
}

EB_DEV bf16x8_t as_bf16x8(u32x4_t v) { return __builtin_bit_cast(bf16x8_t, v); }

// 8-bit E4M3 cache codes (OCP: bias 7, no infinity, 0x7F / 0xFF NaN,
// largest finite 448).  Eight codes (element i in byte i of the two words) as
// eight bf16 values: every code's value is exact in bf16.
template <bool HI>
EB_DEV uint32_t e4m3x2_to_bf16x2(uint32_t w) {
  return __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8((int)w, 1.0f, HI));
}
EB_DEV u32x4_t e4m3x8_to_bf16x8(u32x2_t w) {
  return u32x4_t{e4m3x2_to_bf16x2<false>(w[0]), e4m3x2_to_bf16x2<true>(w[0]), e4m3x2_to_bf16x2<false>(w[1]),
                 e4m3x2_to_bf16x2<true>(w[1])};
}
// Nearest codes (ties to even) of four fp32 values, byte i for value i,
// saturated to +-448 (the conversion itself does not saturate); a NaN keeps
// its sign with the all-ones exponent and mantissa.
EB_DEV uint32_t e4m3x4_from_f32(float a, float b, float c, float d) {
  const float x[4] = {a, b, c, d};
  float y[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) y[i] = __builtin_amdgcn_fmed3f(x[i], -448.0f, 448.0f);
  uint32_t w = (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(y[0], y[1], 0, false);
  w = (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(y[2], y[3], (int)w, true);
#pragma unroll
  for (int i = 0; i < 4; ++i)
    if (x[i] != x[i]) w = (w & ~(0xFFu << (8 * i))) | ((0x7Fu | ((__float_as_uint(x[i]) >> 24) & 0x80u)) << (8 * i));
  return w;
}

// D = A B + C on one 16x16x32 bf16 tile.  Operand layout (lane l):
//   A: row l % 16, k = 8 (l / 16) .. + 7      B: col l % 16, same k
//   C/D: rows 4 (l / 16) .. + 3, col l % 16
EB_DEV f32x4_t mfma16x16x32(u32x4_t a, u32x4_t b, f32x4_t c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(a), as_bf16x8(b), c, 0, 0, 0);
}

// D = A B + C on one 32x32x16 bf16 tile.  Operand layout (lane l):
//   A: row l % 32, k = 8 (l / 32) .. + 7      B: col l % 32, same k
//   C/D (16 values): value i at row 8 (i / 4) + 4 (l / 32) + i % 4, col l % 32
EB_DEV f32x16_t mfma32x32x16(u32x4_t a, u32x4_t b, f32x16_t c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(a), as_bf16x8(b), c, 0, 0, 0);
}

// D = A B + C on one 16x16x16 bf16 tile.  Operand layout (lane l):
//   A: row l % 16, k = 4 (l / 16) .. + 3      B: col l % 16, same k
//   C/D: as for the 16x16x32 tile
EB_DEV f32x4_t mfma16x16x16(u32x2_t a, u32x2_t b, f32x4_t c) {
  typedef short i16x4_t __attribute__((ext_vector_type(4)));
  return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(i16x4_t, a), __builtin_bit_cast(i16x4_t, b), c,
                                                    0, 0, 0);
}

// c + a.lo * b.lo + a.hi * b.hi on bf16 pairs packed in 32-bit words.  (The
// words arrive as plain values: bit-casting a vector element in place has
// been seen to read element 0 instead.)
EB_DEV float dot2_bf16(uint32_t a, uint32_t b, float c) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a), __builtin_bit_cast(bf16x2_t, b), c, false);
}

EB_DEV float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

constexpr float kLog2e = 1.4426950408889634f;
