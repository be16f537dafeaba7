// Definitions shared by the matrix-core kernels (one copy per translation unit).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace cg {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

constexpr int kD = 128;          // head dimension handled here
constexpr int kTok = 32;         // tokens per tile (MFMA N)
constexpr int kThreads = 256;    // four waves
constexpr int kRowBytes = kD * 2;
// s_waitcnt immediate (gfx9 encoding: vmcnt[3:0] and [15:14], expcnt[6:4], lgkmcnt[11:8])
// waiting until at most `vm` vector-memory operations are outstanding, with lgkmcnt = 0 (all
// LDS operations of the wave done) and no wait on expcnt
constexpr int waitcnt_imm(int vm) { return (vm & 15) | ((vm >> 4) << 14) | (7 << 4) | (0 << 8); }

// Cache policy of the large streams.  A kernel that reads one large stream and writes a small
// one (or the reverse) streams faster when the large stream is marked non-temporal: the
// encoder's bf16 tiles are loaded with the `nt` bit (the cache-policy operand of the LDS-direct
// load), the decoders' bf16 / binary32 output rows leave as non-temporal stores; the small
// streams (codes, side words) keep the default policy.
constexpr int kLoadStreamPolicy = 2;  // cache-policy bits of global_load_lds: nt
__device__ __forceinline__ void store_stream(void* p, const u32x4_t& v) { __builtin_nontemporal_store(v, (u32x4_t*)p); }

__device__ __forceinline__ int xcd_remap(int bid, int nwg) {
  // workgroups are dealt round-robin to the 8 XCDs; give each XCD a contiguous range of
  // logical workgroups so that the ranges of one slice share an L2
  const int per = nwg >> 3;
  return (bid & 7) * per + (bid >> 3);
}

// physical 16-byte granule of logical granule j in token row n
__device__ __forceinline__ int swz(int n, int j) { return j ^ (n & 15); }

__device__ __forceinline__ f32x16_t mfma(const bf16x8_t& a, const bf16x8_t& b, const f32x16_t& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ bf16x8_t as_bf16x8(const u32x4_t& v) { return __builtin_bit_cast(bf16x8_t, v); }

// a lane's value moved through DPP (all rows and banks enabled).  Every control used here
// (quad permutes, row rotations, row mirror) reads a lane of the same row, so no lane is out of
// bounds and the move needs no `old` value (which would cost a v_mov of it before each move).
template <int CTRL>
__device__ __forceinline__ float dpp_mov(float v) {
  static_assert(CTRL <= 0xFF || (CTRL >= 0x121 && CTRL <= 0x12F) || CTRL == 0x140 || CTRL == 0x141,
                "quad_perm, row_ror, row_mirror or row_half_mirror only");
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), CTRL, 0xF, 0xF, true));
}
template <int CTRL>
__device__ __forceinline__ int dpp_mov_i(int v) {
  static_assert(CTRL <= 0xFF || (CTRL >= 0x121 && CTRL <= 0x12F) || CTRL == 0x140 || CTRL == 0x141,
                "quad_perm, row_ror, row_mirror or row_half_mirror only");
  return __builtin_amdgcn_mov_dpp(v, CTRL, 0xF, 0xF, true);
}

// Block ranges use the IEEE minimum / maximum (v_minimum3_f32 / v_maximum3_f32): equal to the
// ordinary min / max on finite and infinite values, and NaN as soon as one element is NaN, so
// a single test of the range flags a non-finite block (whose codes are unspecified).
__device__ __forceinline__ float min_nan(float a, float b) { return __builtin_elementwise_minimum(a, b); }
__device__ __forceinline__ float max_nan(float a, float b) { return __builtin_elementwise_maximum(a, b); }

// (min, max) of a lane and the lane 32 away.  v_permlane32_swap exchanges the upper half-wave
// of one register with the lower half-wave of another; with both registers holding the value,
// the two results hold, in every lane, the lane's own value and its partner's.
__device__ __forceinline__ void halves_minmax(float& mn, float& mx) {
  const auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(mn), __float_as_uint(mn), false, false);
  const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(mx), __float_as_uint(mx), false, false);
  mn = min_nan(__uint_as_float(a[0]), __uint_as_float(a[1]));
  mx = max_nan(__uint_as_float(b[0]), __uint_as_float(b[1]));
}

// B fragment of K-step u of a region (RW packed words starting at the region's first channel)
// `one` = 0x3F803F80 (the bf16 pair (1, 1)) and `m` = the mantissa field mask of the code
// width, both held in VGPRs by the caller so that (x & m) | one selects the single
// three-operand v_and_or_b32 (that encoding takes no literal constants on gfx9)
template <int BITS, int RW>
__device__ __forceinline__ bf16x8_t code_frag(const uint32_t (&rw)[RW], int u, uint32_t one, uint32_t m) {
  constexpr uint32_t ONE = 0x3F803F80u;
  u32x4_t f;
  if constexpr (BITS == 4) {
    const uint32_t w = rw[u];  // m = 0x00780078: mantissa bits 3..6 of both halves
    f[0] = ((w << 3) & m) | one;
    f[1] = ((w >> 1) & m) | one;
    f[2] = ((w >> 5) & m) | one;
    f[3] = ((w >> 9) & m) | one;
  } else if constexpr (BITS == 2) {
    const uint32_t w = rw[u >> 1];  // m = 0x00600060: mantissa bits 5..6
    if ((u & 1) == 0) {
      f[0] = ((w << 5) & m) | one;
      f[1] = ((w << 3) & m) | one;
      f[2] = ((w << 1) & m) | one;
      f[3] = ((w >> 1) & m) | one;
    } else {
      f[0] = ((w >> 3) & m) | one;
      f[1] = ((w >> 5) & m) | one;
      f[2] = ((w >> 7) & m) | one;
      f[3] = ((w >> 9) & m) | one;
    }
  } else if constexpr (BITS == 6) {
    // codes 8u + (0,4,1,5,2,6,3,7) at mantissa bits 0..5 (B = 1 + q / 128; m = 0x003F003F):
    // code 8u + j starts at byte 6u + 6j/8, bit 6j % 8 of the region and its partner 8u + j + 4
    // three bytes later, so one byte permute (bytes o, o+1, o+3, o+4 of the word pair) puts
    // the two exactly 16 bits apart; bytes past the region only reach masked-off bits
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int byte = 6 * u + (6 * j) / 8, r = (6 * j) % 8;
      const int wi = byte >> 2, o = byte & 3;
      const uint32_t sel = uint32_t(o) | (uint32_t(o + 1) << 8) | (uint32_t(o + 3) << 16) | (uint32_t(o + 4) << 24);
      const uint32_t x = __builtin_amdgcn_perm(rw[wi + 1 < RW ? wi + 1 : wi], rw[wi], sel);
      f[j] = ((x >> r) & m) | one;
    }
  } else if constexpr (BITS == 3) {
    // codes 16 (u/2) + 4 (u%2) + (0,8,1,9,2,10,3,11) at mantissa bits 4..6 (m = 0x00700070):
    // code j of a 16-code group starts at byte 3j/8, bit 3j % 8, its partner j + 8 three bytes
    // later; one byte permute puts the pair 16 bits apart, one shift moves it to bit 4
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int j = 4 * (u & 1) + k, byte = 6 * (u >> 1) + (3 * j) / 8, r = (3 * j) % 8;
      const int wi = byte >> 2, o = byte & 3;
      const uint32_t sel = uint32_t(o) | (uint32_t(o + 1) << 8) | (uint32_t(o + 3) << 16) | (uint32_t(o + 4) << 24);
      const uint32_t x = __builtin_amdgcn_perm(rw[wi + 1 < RW ? wi + 1 : wi], rw[wi], sel);
      const uint32_t y = r <= 4 ? (x << (4 - r)) : (x >> (r - 4));
      f[k] = (y & m) | one;
    }
  } else if constexpr (BITS == 8) {
    // codes as themselves: bytes to binary32 (exact), high halves are the bf16 values
    const uint32_t w0 = rw[2 * u], w1 = rw[2 * u + 1];
    auto pk = [](float lo, float hi) { return __builtin_amdgcn_perm(__float_as_uint(hi), __float_as_uint(lo), 0x07060302u); };
    f[0] = pk(float(w0 & 255u), float((w0 >> 8) & 255u));
    f[1] = pk(float((w0 >> 16) & 255u), float(w0 >> 24));
    f[2] = pk(float(w1 & 255u), float((w1 >> 8) & 255u));
    f[3] = pk(float((w1 >> 16) & 255u), float(w1 >> 24));
  } else {
    // other widths: 8 codes of the LSB-first stream at bit 8 u BITS of the region
    constexpr int b0 = 8 * BITS;
    const int bit = u * b0, wi = bit >> 5, sh = bit & 31;
    const uint64_t win = ((uint64_t(rw[wi + 1 < RW ? wi + 1 : wi]) << 32) | rw[wi]) >> sh;
#pragma unroll
    for (int k2 = 0; k2 < 4; ++k2) {
      const uint32_t c0 = uint32_t(win >> (2 * k2 * BITS)) & ((1u << BITS) - 1u);
      const uint32_t c1 = uint32_t(win >> ((2 * k2 + 1) * BITS)) & ((1u << BITS) - 1u);
      f[k2] = ONE | (c0 << (7 - BITS)) | (c1 << (23 - BITS));
    }
  }
  return as_bf16x8(f);
}

}  // namespace
}  // namespace cg
