// Device helpers of the codec kernels: number formats and the scalar quantiser step.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "codec_gauge.h"

namespace cg {

__device__ __forceinline__ float bf16_to_f32(uint32_t h) { return __uint_as_float(h << 16); }

// binary32 -> bfloat16 bits, round to nearest even (NaN stays a quiet NaN).
__device__ __forceinline__ uint32_t f32_to_bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (u >> 16) | 0x40u;
  u += 0x7fffu + ((u >> 16) & 1u);
  return u >> 16;
}

__device__ __forceinline__ float f16_bits_to_f32(uint32_t bits) {
  return (float)__builtin_bit_cast(_Float16, (uint16_t)bits);
}

// Binary16 bits of v rounded toward -inf: the hardware conversion rounds to nearest even;
// when that lands above v, step one binary16 ulp down.  -0 is returned as +0.
__device__ __forceinline__ uint32_t f16_bits_down(float v) {
  _Float16 h = (_Float16)v;
  uint32_t bits = __builtin_bit_cast(uint16_t, h);
  if ((float)h > v) bits = (bits & 0x8000u) ? bits + 1u : bits - 1u;
  return bits == 0x8000u ? 0u : bits;
}

// Binary16 bits of v rounded toward +inf (-0 returned as +0).
__device__ __forceinline__ uint32_t f16_bits_up(float v) {
  _Float16 h = (_Float16)v;
  uint32_t bits = __builtin_bit_cast(uint16_t, h);
  if ((float)h < v) bits = (bits & 0x8000u) ? bits - 1u : bits + 1u;
  return bits == 0x8000u ? 0u : bits;
}

// The same two binary16 roundings by the hardware conversion under a directed rounding mode:
// bits [3:2] of the MODE register set the rounding of binary16 and binary64 results (0
// nearest even, 1 toward +inf, 2 toward -inf; the binary32 field, bits [1:0], is untouched).
// The mode switch and the conversion are one asm block, so that the compiler neither resets
// the mode for the conversion nor fuses the conversion into the instruction producing v (which
// would round an unrounded product); s_nop 1 covers the wait states between s_setreg and a
// VALU instruction that depends on the mode.  The mode is per wave and restored to nearest
// even.  cg_selftest(2) checks both against f16_bits_down / f16_bits_up for every binary32
// bit pattern.
template <int MODE>
__device__ __forceinline__ uint32_t f16_bits_directed_hw(float v) {
  uint32_t bits;
  asm volatile(
      "s_setreg_imm32_b32 hwreg(HW_REG_MODE, 2, 2), %2\n\t"
      "s_nop 1\n\t"
      "v_cvt_f16_f32_e32 %0, %1\n\t"
      "s_setreg_imm32_b32 hwreg(HW_REG_MODE, 2, 2), 0\n\t"
      "s_nop 1"
      : "=v"(bits)
      : "v"(v), "i"(MODE));
  bits &= 0xffffu;
  return bits == 0x8000u ? 0u : bits;
}
__device__ __forceinline__ uint32_t f16_bits_down_hw(float v) { return f16_bits_directed_hw<2>(v); }
__device__ __forceinline__ uint32_t f16_bits_up_hw(float v) { return f16_bits_directed_hw<1>(v); }

// RN(a / (2^b - 1)) without a division: q0 = RN(a r) with r = RN(1 / d), the exact residual
// e = a - q0 d (one FMA), then RN(q0 + e r) (Markstein's correction step).  cg_selftest(1)
// checks it against correctly rounded division for every binary32 mantissa of the binades
// the quantiser meets.
__device__ __forceinline__ float div_by_qmax(float a, int bits) {
  const float d = float((1 << bits) - 1);
  const float r = 1.0f / d;
  const float q0 = a * r;
  const float e = fmaf(-q0, d, a);
  return fmaf(e, r, q0);
}

// RN(1 / s) for a positive binary16 value s: hardware estimate, then one Newton step on the
// exact residual.  cg_selftest(0) checks it for every positive finite binary16 value.
__device__ __forceinline__ float rcp_of_f16(float s) {
  const float y = __builtin_amdgcn_rcpf(s);
  const float e = fmaf(-s, y, 1.0f);
  return fmaf(e, y, y);
}

// Side information of one quantisation block from its exact min and max (section 4.3
// block range): binary16 min rounded down, binary16 scale rounded up, binary32 reciprocal.
struct Side {
  float mn, sc, inv;
  uint32_t word;  // min bits | scale bits << 16 (min at the lower address)
  int flags;
};

// HW: the binary16 roundings by the hardware conversion under a directed mode (same results)
template <bool HW = false>
__device__ __forceinline__ Side make_side(float mn, float mx, int bits) {
#pragma clang fp contract(off)
  Side s;
  uint32_t mnb = HW ? f16_bits_down_hw(mn) : f16_bits_down(mn);
  s.mn = f16_bits_to_f32(mnb);
  float diff = mx - s.mn;
  float s32 = div_by_qmax(diff, bits);           // = RN(diff / (2^b - 1))
  uint32_t scb = HW ? f16_bits_up_hw(s32) : f16_bits_up(s32);
  s.sc = f16_bits_to_f32(scb);
  s.inv = (s.sc == 0.0f) ? 0.0f : rcp_of_f16(s.sc);  // = RN(1 / sc)
  s.word = mnb | (scb << 16);
  s.flags = (((mnb & 0x7c00u) == 0x7c00u) || ((scb & 0x7c00u) == 0x7c00u)) ? CG_FLAG_SIDE_OVERFLOW : 0;
  return s;
}

// q = clamp(rint_even(fl32(fl32(z - mn) * inv)), 0, qmax)
__device__ __forceinline__ uint32_t quantize(float z, float mn, float inv, float qmax) {
#pragma clang fp contract(off)
  float t = (z - mn) * inv;
  float r = __builtin_rintf(t);
  r = fminf(fmaxf(r, 0.0f), qmax);
  return (uint32_t)r;
}

// rint_even(fl32(fl32(z - mn) * inv)) as an integer-valued float.  No clamp is needed: with
// mn_h <= min z the difference is >= 0, and with sc_h >= RN(range / qmax) the product is at
// most qmax (1 + 4 * 2^-24) < qmax + 1/2, so the rounded value lies in [0, qmax] for finite
// blocks (non-finite blocks raise an error flag and their codes are unspecified).
__device__ __forceinline__ float quantize_rint(float z, float mn, float inv) {
#pragma clang fp contract(off)
  float t = (z - mn) * inv;
  return __builtin_rintf(t);
}

// t = fl32(fl32(z - mn) * inv) before rounding: for consumers that round to nearest even
// themselves (v_cvt_pk_u8_f32 rounds to nearest even and saturates to [0, 255]).
__device__ __forceinline__ float quantize_t(float z, float mn, float inv) {
#pragma clang fp contract(off)
  return (z - mn) * inv;
}

// The code of t as an integer in one instruction: v_cvt_pk_u8_f32 rounds to nearest even and
// saturates to [0, 255] (codes of at most 8 bits lie in [0, 2^b - 1] for finite blocks, so
// this equals rint_even(t)), writing byte 0 of a zeroed word.
__device__ __forceinline__ uint32_t code_u8(float t) { return __builtin_amdgcn_cvt_pk_u8_f32(t, 0, 0u); }

// zhat = fl32(mn + q * sc); q * sc is exact in binary32.
__device__ __forceinline__ float dequantize(uint32_t q, float mn, float sc) {
#pragma clang fp contract(off)
  float p = (float)q * sc;
  return mn + p;
}

// Code `idx` of an LSB-first stream of b-bit codes starting at a 4-byte boundary.
__device__ __forceinline__ uint32_t extract_code(const uint32_t* stream, int idx, int bits) {
  int bit = idx * bits;
  int w = bit >> 5, off = bit & 31;
  uint32_t v = stream[w] >> off;
  if (off + bits > 32) v |= stream[w + 1] << (32 - off);
  return v & ((1u << bits) - 1u);
}

}  // namespace cg
