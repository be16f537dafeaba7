// zfp-style fixed-rate block coder shared by the codec kernels (one copy per translation unit).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "codec_gauge.h"

namespace cg {
namespace {

// ------------------------------------------------------------------------------------------
// zfp-style fixed-rate blocks: 4 tokens x 4 channels of z, 16 rate bits each (zfp's published
// algorithm: block exponent, 30-bit fixed point, lifted 4-point transform along channels then
// tokens, sequency order, negabinary, embedded bit planes with group tests)
//
// The embedded coder is written in closed form, one bit plane at a time, with no loop over the
// bits of a plane.  For plane P, with n coefficients significant before it (n only grows) and x
// the plane's 16 bits (bit k = bit P of coefficient k in sequency order):
//   * the first n bits of x go out verbatim;
//   * if n < 16, y = x >> n goes through the group tests: a 1 before each run "0...01" of y that
//     ends in a 1, the run itself, and a closing 0 once no 1 is left; when a run reaches the last
//     candidate (coefficient 15) its 1 is implied and the plane ends without a closing bit.
// With y's ones at r_1 < ... < r_m and F(y) = sum_j 2^(r_j + j), the group bits are
// G = 1 + 3F - 2^(h+1) (bit 0: the first test; each one at r_j + j followed by the next test at
// r_j + j + 1; h = r_m + m is F's top bit), minus 2^h more when the last one is implied; the
// plane takes n' + m + 1 bits (n' = significant count after the plane), one bit fewer when the
// last one is implied (n' = 16), n + 1 when y = 0 and n < 16, 16 when n = 16.  n' is the
// position after the highest set bit of the OR of all planes so far.  F comes from a 256-entry
// table per byte of y (the high byte's positions move up by the low byte's popcount).
//
// Decoding reads the group bits after a leading 1 as alternating data and test bits: inside a
// run of ones the first, third, ... are data ones (a one of y) and the others their test bits;
// the first run of odd length ends the plane (its last one is a data one, the zero after it the
// closing test).  Runs are classified by the parity of their start with one addition each
// (adding a run's start bit clears the run and sets the bit after it).  The data ones map back
// to y by removing the test bits before them (a 256-entry table per byte again).  When the data
// bits reach the last candidate before that, its 1 is implied, provided the bits up to it lie
// inside the budget.  Bits past the budget read as 0; a plane cut by the budget keeps what it
// read before the cut, as zfp's bit-serial decoder does, and decoding stops there.
// ------------------------------------------------------------------------------------------
__host__ __device__ __forceinline__ int32_t wadd(int32_t a, int32_t b) { return int32_t(uint32_t(a) + uint32_t(b)); }
__host__ __device__ __forceinline__ int32_t wsub(int32_t a, int32_t b) { return int32_t(uint32_t(a) - uint32_t(b)); }
__host__ __device__ __forceinline__ int32_t wdbl(int32_t a) { return int32_t(uint32_t(a) << 1); }

// 1/16 [[4 4 4 4] [5 1 -1 -5] [-4 4 4 -4] [-2 6 -6 2]] applied to (a, b, c, e) by lifting
__host__ __device__ __forceinline__ void zfp_fwd4(int32_t& a, int32_t& b, int32_t& c, int32_t& e) {
  a = wadd(a, e) >> 1; e = wsub(e, a);
  c = wadd(c, b) >> 1; b = wsub(b, c);
  a = wadd(a, c) >> 1; c = wsub(c, a);
  e = wadd(e, b) >> 1; b = wsub(b, e);
  e = wadd(e, b >> 1); b = wsub(b, e >> 1);
}
__host__ __device__ __forceinline__ void zfp_inv4(int32_t& a, int32_t& b, int32_t& c, int32_t& e) {
  b = wadd(b, e >> 1); e = wsub(e, b >> 1);
  b = wadd(b, e); e = wsub(wdbl(e), b);
  c = wadd(c, a); a = wsub(wdbl(a), c);
  b = wadd(b, c); c = wsub(wdbl(c), b);
  e = wadd(e, a); a = wsub(wdbl(a), e);
}

// sequency position k -> block entry 4 j + i (by i + j, then i^2 + j^2, then j)
constexpr int kZfpOrder[16] = {0, 1, 4, 5, 2, 8, 6, 9, 3, 12, 10, 7, 13, 11, 14, 15};

// Per-byte tables of the plane coder, in LDS (zfp_tables_init by every thread of the workgroup,
// then a barrier before the first use).
//   spread[b]   = sum over the ones of b at r_1 < r_2 < ... of 2^(r_j + j)
//   unspread[b] = sum over the ones of b at d_1 < d_2 < ... of 2^(d_j - j + 1)
struct ZfpTables {
  uint16_t spread[256];
  uint8_t unspread[256];
};

__host__ __device__ inline void zfp_table_entry(int b, uint16_t& sp, uint8_t& un) {
  uint32_t f = 0u, g = 0u;
  int j = 0;
  for (int r = 0; r < 8; ++r)
    if ((b >> r) & 1) {
      ++j;
      f |= 1u << (r + j);
      g |= 1u << (r - j + 1);
    }
  sp = uint16_t(f);
  un = uint8_t(g);
}

__device__ inline void zfp_tables_init(ZfpTables& t) {
  for (int i = int(threadIdx.x); i < 256; i += int(blockDim.x)) zfp_table_entry(i, t.spread[i], t.unspread[i]);
}

__host__ __device__ __forceinline__ uint32_t bsel(uint32_t m, uint32_t a, uint32_t b) { return (m & a) | (~m & b); }

// 8 x 8 bit transpose of (lo, hi): bit 8 i + j <-> bit 8 j + i (three delta swaps)
__host__ __device__ __forceinline__ void transpose8(uint32_t& lo, uint32_t& hi) {
  lo = bsel(0x00AA00AAu, lo >> 7, bsel(0x55005500u, lo << 7, lo));
  hi = bsel(0x00AA00AAu, hi >> 7, bsel(0x55005500u, hi << 7, hi));
  lo = bsel(0x0000CCCCu, lo >> 14, bsel(0x33330000u, lo << 14, lo));
  hi = bsel(0x0000CCCCu, hi >> 14, bsel(0x33330000u, hi << 14, hi));
  const uint32_t l2 = bsel(0xF0F0F0F0u, hi << 4, lo);
  hi = bsel(0x0F0F0F0Fu, lo >> 4, hi);
  lo = l2;
}

// bytes (a.b0, b.b0, a.b1, b.b1) and (a.b2, b.b2, a.b3, b.b3) of two words
__host__ __device__ __forceinline__ uint32_t interleave_lo(uint32_t a, uint32_t b) {
  return (a & 0xFFu) | ((b & 0xFFu) << 8) | ((a & 0xFF00u) << 8) | ((b & 0xFF00u) << 16);
}
__host__ __device__ __forceinline__ uint32_t interleave_hi(uint32_t a, uint32_t b) {
  return ((a >> 16) & 0xFFu) | ((b >> 8) & 0xFF00u) | ((a >> 8) & 0xFF0000u) | (b & 0xFF000000u);
}
// even bytes (w0.b0, w0.b2, w1.b0, w1.b2) and odd bytes (w0.b1, w0.b3, w1.b1, w1.b3)
__host__ __device__ __forceinline__ uint32_t even_bytes(uint32_t w0, uint32_t w1) {
  return (w0 & 0xFFu) | ((w0 >> 8) & 0xFF00u) | ((w1 & 0xFFu) << 16) | ((w1 << 8) & 0xFF000000u);
}
__host__ __device__ __forceinline__ uint32_t odd_bytes(uint32_t w0, uint32_t w1) {
  return ((w0 >> 8) & 0xFFu) | ((w0 >> 16) & 0xFF00u) | ((w1 << 8) & 0xFF0000u) | (w1 & 0xFF000000u);
}

// Planes lo .. lo+7 of u[16] (lo in [-7, 24]; planes below 0 read as 0) as 16-bit masks:
// xp[q] holds plane lo + 2q in bits 0..15 and plane lo + 2q + 1 in bits 16..31.
__host__ __device__ __forceinline__ void plane_window(const uint32_t (&u)[16], int lo, uint32_t (&xp)[4]) {
  const int off = lo < 0 ? 0 : lo, ls = off - lo;
  const uint32_t mk = 0xFFu >> ls;
  uint32_t D[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    uint32_t acc = 0u;
#pragma unroll
    for (int i = 0; i < 4; ++i) acc |= ((u[4 * q + i] >> off) & mk) << (8 * i + ls);
    D[q] = acc;
  }
  transpose8(D[0], D[1]);  // coefficients 0..7: byte p = plane lo + p
  transpose8(D[2], D[3]);  // coefficients 8..15
  xp[0] = interleave_lo(D[0], D[2]);
  xp[1] = interleave_hi(D[0], D[2]);
  xp[2] = interleave_lo(D[1], D[3]);
  xp[3] = interleave_hi(D[1], D[3]);
}

// The inverse: u[k] |= bits of coefficient k in planes lo .. lo+7 held as plane_window does
__host__ __device__ __forceinline__ void plane_unwindow(const uint32_t (&xp)[4], int lo, uint32_t (&u)[16]) {
  uint32_t A0 = even_bytes(xp[0], xp[1]), A1 = even_bytes(xp[2], xp[3]);  // coefficients 0..7
  uint32_t B0 = odd_bytes(xp[0], xp[1]), B1 = odd_bytes(xp[2], xp[3]);    // coefficients 8..15
  transpose8(A0, A1);
  transpose8(B0, B1);
  const uint32_t W[4] = {A0, A1, B0, B1};
  if (lo >= 0) {
#pragma unroll
    for (int k = 0; k < 16; ++k) u[k] |= ((W[k >> 2] >> (8 * (k & 3))) & 0xFFu) << lo;
  } else {
#pragma unroll
    for (int k = 0; k < 16; ++k) u[k] |= ((W[k >> 2] >> (8 * (k & 3))) & 0xFFu) >> -lo;
  }
}

// p on every active lane of the wave (WAVE), or on this lane (the CPU build of this header, which
// checks each path lane by lane).  The plane coders pick the short path of the last two
// candidates for the whole wave: a wave whose lanes need different paths runs the general one.
template <bool WAVE>
__host__ __device__ __forceinline__ bool all_lanes(bool p) {
  if constexpr (WAVE) return __builtin_amdgcn_ballot_w64(!p) == 0;
  else return p;
}

// 16 RATE bits of one block held in one (RATE <= 4) or two 64-bit words, LSB-first
template <int RATE>
struct ZBits {
  static constexpr int kCap = 16 * RATE;
  static constexpr bool kWide = kCap > 64;
  uint64_t w0 = 0u, w1 = 0u;
  // OR in the bits of s (< 2^32) at position o < kCap
  __host__ __device__ __forceinline__ void put(uint32_t s, int o) {
    if constexpr (!kWide) {
      w0 |= uint64_t(s) << o;
    } else {
      const uint64_t v = s;
      w0 |= o < 64 ? v << (o & 63) : 0u;
      w1 |= o >= 64 ? v << (o & 63) : (o > 32 ? v >> ((64 - o) & 63) : 0u);
    }
  }
  // bits [o, o + 64) for o < kCap (0 past the block)
  __host__ __device__ __forceinline__ uint64_t window(int o) const {
    if constexpr (!kWide) {
      return w0 >> o;
    } else {
      const uint64_t lo = o < 64 ? w0 : w1, hi = o < 64 ? w1 : 0u;
      const int sh = o & 63;
      return sh ? (lo >> sh) | (hi << (64 - sh)) : lo;
    }
  }
  __host__ __device__ __forceinline__ void clip() {
    if constexpr (kCap < 64) w0 &= (uint64_t(1) << kCap) - 1u;
    if constexpr (kCap > 64 && kCap < 128) w1 &= (uint64_t(1) << (kCap - 64)) - 1u;
  }
};

// First half of the encoder, without a branch (so that it can be interleaved with other work):
// block range, exponent, 30-bit fixed point, transform, negabinary, and the top eight planes.
// v[4 j + i]: channel i of token j.
struct ZfpPrep {
  uint32_t u[16];   // negabinary coefficients in sequency order
  uint32_t xp[4];   // planes top-7 .. top as plane_window holds them
  int e, top;       // block exponent, highest plane with a set bit
  bool coded;       // finite and not all zero
  bool finite;
};

__host__ __device__ __forceinline__ void zfp_prepare(const float (&v)[16], ZfpPrep& z) {
  // NaN-propagating maximum of |v|: one test flags a non-finite block (coded as an empty block)
  float amax = fabsf(v[0]);
#pragma unroll
  for (int k = 1; k < 16; ++k) amax = __builtin_elementwise_maximum(amax, fabsf(v[k]));
  z.finite = amax <= 3.40282347e38f;
  z.coded = z.finite && amax != 0.0f;
  int e;
  frexpf(amax, &e);
  e = e < -126 ? -126 : e;
  z.e = e;
  int32_t q[16];
  // exact scaling and truncation (|q| < 2^30 for a coded block; the clamp only keeps the
  // conversion defined for the blocks that are not coded)
#pragma unroll
  for (int k = 0; k < 16; ++k) q[k] = int32_t(fminf(fmaxf(ldexpf(v[k], 30 - e), -2147483648.0f), 2147483520.0f));
#pragma unroll
  for (int j = 0; j < 4; ++j) zfp_fwd4(q[4 * j], q[4 * j + 1], q[4 * j + 2], q[4 * j + 3]);
#pragma unroll
  for (int i = 0; i < 4; ++i) zfp_fwd4(q[i], q[4 + i], q[8 + i], q[12 + i]);
  uint32_t any = 0u;
#pragma unroll
  for (int k = 0; k < 16; ++k) {
    z.u[k] = (uint32_t(q[kZfpOrder[k]]) + 0xAAAAAAAAu) ^ 0xAAAAAAAAu;
    any |= z.u[k];
  }
  z.top = 31 - __builtin_clz(any | 1u);  // a coded block has |q| >= 2^29 somewhere, so any != 0
  plane_window(z.u, z.top - 7, z.xp);
}

// Second half: the bit planes.  w: the block's 16 RATE bits, LSB-first (words past the block
// are 0).  Returns flags.
template <int RATE, bool WAVE = true>
__host__ __device__ __forceinline__ int zfp_encode_planes(const ZfpPrep& z, const ZfpTables& tb, uint32_t (&w)[4]) {
  constexpr int CAP = ZBits<RATE>::kCap;
  ZBits<RATE> st;
  if (z.coded) {
    st.put(1u | (uint32_t(z.e + 127) << 1), 0);
    // planes above the highest set bit: one 0 test bit each
    int o = 9 + 31 - z.top, n = 0;
    uint32_t X = 0u;
    uint32_t xp[4] = {z.xp[0], z.xp[1], z.xp[2], z.xp[3]};
    for (int P0 = z.top; P0 >= 0 && o < CAP; P0 -= 8) {
      if (P0 != z.top) plane_window(z.u, P0 - 7, xp);
#pragma unroll
      for (int p = 7; p >= 0; --p) {
        if (P0 - 7 + p >= 0 && o < CAP) {
          const uint32_t x = (xp[p >> 1] >> (16 * (p & 1))) & 0xFFFFu;
          if (all_lanes<WAVE>(n >= 14)) {
            // at most two candidates left.  n = 15: the last candidate's test bit is the plane's
            // bit 15 (a 1 makes it significant, its 1 implied), so the plane is its 16 bits, as
            // for n = 16.  n = 14: test bit, then coefficient 14's bit and, after a 1, the test
            // for coefficient 15
            const uint32_t y = x >> 14;
            const uint32_t gb = y == 0 ? 0u : (y == 1 ? 3u : (y == 2 ? 1u : 7u));
            const bool two = n == 14;
            st.put(two ? (x & 0x3FFFu) | (gb << 14) : x, o);
            o += two ? (y == 0 ? 15 : (y == 2 ? 16 : 17)) : 16;
            n = two ? (y == 0 ? 14 : (y == 1 ? 15 : 16)) : ((x >> 15) ? 16 : n);
          } else {
            X |= x;
            const int n2 = 32 - __builtin_clz(X | 1u);
            const uint32_t y = x >> n, V = x & ((1u << n) - 1u);
            const uint32_t lo8 = y & 0xFFu;
            const uint32_t F = uint32_t(tb.spread[lo8]) +
                               (uint32_t(tb.spread[y >> 8]) << (8 + __builtin_popcount(lo8)));
            const uint32_t hb = 1u << (31 - __builtin_clz(F | 1u));
            const uint32_t G = 3u * F + 1u - (n2 == 16 ? 3u * hb : 2u * hb);
            const int m = __builtin_popcount(y);
            st.put(y ? V | (G << n) : V, o);
            o += y ? n2 + m + (n2 < 16 ? 1 : -1) : n + (n < 16 ? 1 : 0);
            n = y ? n2 : n;
          }
        }
      }
    }
  }
  st.clip();
  w[0] = uint32_t(st.w0);
  w[1] = uint32_t(st.w0 >> 32);
  w[2] = uint32_t(st.w1);
  w[3] = uint32_t(st.w1 >> 32);
  return z.finite ? 0 : CG_FLAG_NONFINITE;
}

template <int RATE, bool WAVE = true>
__host__ __device__ __forceinline__ int zfp_encode_block(const float (&v)[16], const ZfpTables& tb, uint32_t (&w)[4]) {
  ZfpPrep z;
  zfp_prepare(v, z);
  return zfp_encode_planes<RATE, WAVE>(z, tb, w);
}

// First half of the decoder: the bit planes of a block's 16 RATE bits w (LSB-first, words past
// the block 0) into the negabinary coefficients u (sequency order) and the block exponent e; an
// empty block gives u = 0.
template <int RATE, bool WAVE = true>
__host__ __device__ __forceinline__ void zfp_decode_planes(const uint32_t (&w)[4], const ZfpTables& tb, uint32_t (&u)[16],
                                                           int& e) {
  constexpr int CAP = ZBits<RATE>::kCap;
  ZBits<RATE> st;
  st.w0 = uint64_t(w[0]) | (uint64_t(w[1]) << 32);
  st.w1 = uint64_t(w[2]) | (uint64_t(w[3]) << 32);
  st.clip();
#pragma unroll
  for (int k = 0; k < 16; ++k) u[k] = 0u;
  e = 0;
  if (!(st.w0 & 1u)) return;
  e = int((st.w0 >> 1) & 0xFFu) - 127;
  // leading empty planes: one 0 test bit each
  const uint64_t lead = st.window(9);
  const int z = lead ? __builtin_ctzll(lead) : 64;
  int o = 9 + z, n = 0;
  for (int P0 = 31 - z; P0 >= 0 && o < CAP; P0 -= 8) {
    uint32_t xp[4] = {0u, 0u, 0u, 0u};
#pragma unroll
    for (int p = 7; p >= 0; --p) {
      if (P0 - 7 + p >= 0 && o < CAP) {
        const uint64_t win = st.window(o);
        uint32_t x;
        if (all_lanes<WAVE>(n >= 14)) {
          // at most two candidates left.  n >= 15: the plane's 16 bits (for n = 15 the last
          // candidate's test bit is its bit; a 1 read inside the budget implies the 1).  n = 14:
          // test bit t; after a 1, coefficient 14's bit r0, and after a 1 there the test r1 for
          // coefficient 15 (its 1 implied); after r0 = 0 coefficient 15's 1 is implied if r0 lay
          // inside the budget
          const uint32_t wl = uint32_t(win);
          const uint32_t t = (wl >> 14) & 1u, r0 = (wl >> 15) & 1u, r1 = (wl >> 16) & 1u;
          const uint32_t V = wl & 0x3FFFu;
          const bool fits = o + 16 <= CAP, two = n == 14;
          const uint32_t x14 = !t ? V : (r0 ? (V | (1u << 14) | (r1 << 15)) : (V | (fits ? 1u << 15 : 0u)));
          x = two ? x14 : (wl & 0xFFFFu);
          o += two ? (!t ? 15 : (r0 ? 17 : 16)) : 16;
          n = two ? (!t ? 14 : (r0 ? (r1 ? 16 : 15) : 16)) : (((wl >> 15) & 1u) ? 16 : n);
        } else {
          const uint32_t V = uint32_t(win) & ((1u << n) - 1u);
          const uint32_t rest = uint32_t(win >> (n + 1));
          // runs of ones by the parity of their start
          const uint32_t st0 = rest & ~(rest << 1);
          const uint32_t ae = rest + (st0 & 0x55555555u), ao = rest + (st0 & 0xAAAAAAAAu);
          const uint32_t re = rest & ~ae;                           // ones of even-start runs
          const uint32_t data1 = rest & ~(re ^ 0x55555555u);         // data ones: even offset in their run
          // the zero after an odd-length run (the closing test): after an even-start run at an odd
          // position, after an odd-start run at an even position
          const uint32_t close = bsel(0x55555555u, ao, ae) & ~rest;
          const int e1 = close ? __builtin_ctz(close) : 32;
          const uint32_t below = e1 >= 32 ? ~0u : (1u << e1) - 1u;
          const uint32_t dm = data1 & below;
          const int dcount = e1 - (__builtin_popcount(rest & below) - __builtin_popcount(dm));
          const int pc0 = __builtin_popcount(dm & 0xFFu), pc1 = __builtin_popcount(dm & 0xFFFFu),
                    pc2 = __builtin_popcount(dm & 0xFFFFFFu);
          const uint32_t y = uint32_t(tb.unspread[dm & 0xFFu]) | (uint32_t(tb.unspread[(dm >> 8) & 0xFFu]) << (8 - pc0)) |
                             (uint32_t(tb.unspread[(dm >> 16) & 0xFFu]) << (16 - pc1)) |
                             (uint32_t(tb.unspread[dm >> 24]) << (24 - pc2));
          const int L = 15 - n;  // explicit candidates before the last one (n < 16 here)
          const bool implied = dcount > L;
          const uint32_t yl = y & ((1u << L) - 1u);
          const int glen = implied ? 1 + L + __builtin_popcount(yl) : e1 + 2;
          const bool fits = o + n + glen <= CAP;
          const uint32_t yn = implied ? (yl | (fits ? 1u << L : 0u)) : y;
          const bool t0 = (uint32_t(win) >> n) & 1u;  // n < 16
          const bool all = n == 16;  // lanes whose candidates are all significant: 16 verbatim bits
          x = all ? (uint32_t(win) & 0xFFFFu) : (t0 ? V | (yn << n) : V);
          o += all ? 16 : (t0 ? n + glen : n + 1);
          n = all ? 16 : (t0 ? (implied ? 16 : n + dcount) : n);
        }
        xp[p >> 1] |= x << (16 * (p & 1));
      }
    }
    plane_unwindow(xp, P0 - 7, u);
  }
}

// Second half, without a branch: negabinary to two's complement, inverse transform, scaling.
// v[4 j + i]: channel i of token j.
__host__ __device__ __forceinline__ void zfp_decode_finish(const uint32_t (&u)[16], int e, float (&v)[16]) {
  int32_t q[16];
#pragma unroll
  for (int k = 0; k < 16; ++k) q[kZfpOrder[k]] = int32_t((u[k] ^ 0xAAAAAAAAu) - 0xAAAAAAAAu);
#pragma unroll
  for (int i = 0; i < 4; ++i) zfp_inv4(q[i], q[4 + i], q[8 + i], q[12 + i]);
#pragma unroll
  for (int j = 0; j < 4; ++j) zfp_inv4(q[4 * j], q[4 * j + 1], q[4 * j + 2], q[4 * j + 3]);
#pragma unroll
  for (int k = 0; k < 16; ++k) v[k] = ldexpf(float(q[k]), e - 30);
}

template <int RATE, bool WAVE = true>
__host__ __device__ __forceinline__ void zfp_decode_block(const uint32_t (&w)[4], const ZfpTables& tb, float (&v)[16]) {
  uint32_t u[16];
  int e;
  zfp_decode_planes<RATE, WAVE>(w, tb, u, e);
  zfp_decode_finish(u, e, v);
}

// a block's 2 RATE bytes to / from the cache (blocks start at multiples of 2 RATE bytes)
template <int RATE>
__device__ __forceinline__ void zfp_store(uint8_t* p, const uint32_t (&w)[4]) {
  if constexpr (RATE == 2) {
    *(uint32_t*)p = w[0];
  } else if constexpr (RATE == 4) {
    *(uint2*)p = make_uint2(w[0], w[1]);
  } else if constexpr (RATE == 8) {
    *(uint4*)p = make_uint4(w[0], w[1], w[2], w[3]);
  } else if constexpr (RATE == 6) {
    uint32_t* q = (uint32_t*)p;
    q[0] = w[0]; q[1] = w[1]; q[2] = w[2];
  } else {
    uint16_t* q = (uint16_t*)p;
#pragma unroll
    for (int r = 0; r < RATE; ++r) q[r] = uint16_t(w[r >> 1] >> (16 * (r & 1)));
  }
}
template <int RATE>
__device__ __forceinline__ void zfp_load(const uint8_t* p, uint32_t (&w)[4]) {
  w[0] = w[1] = w[2] = w[3] = 0u;
  if constexpr (RATE == 2) {
    w[0] = *(const uint32_t*)p;
  } else if constexpr (RATE == 4) {
    const uint2 t = *(const uint2*)p;
    w[0] = t.x; w[1] = t.y;
  } else if constexpr (RATE == 8) {
    const uint4 t = *(const uint4*)p;
    w[0] = t.x; w[1] = t.y; w[2] = t.z; w[3] = t.w;
  } else if constexpr (RATE == 6) {
    const uint32_t* q = (const uint32_t*)p;
    w[0] = q[0]; w[1] = q[1]; w[2] = q[2];
  } else {
    const uint16_t* q = (const uint16_t*)p;
#pragma unroll
    for (int r = 0; r < RATE; ++r) w[r >> 1] |= uint32_t(q[r]) << (16 * (r & 1));
  }
}

// runtime rate -> template
template <typename Fn>
__host__ __device__ __forceinline__ auto zfp_by_rate(int rate, Fn&& fn) {
  switch (rate) {
    case 2: return fn(std::integral_constant<int, 2>());
    case 3: return fn(std::integral_constant<int, 3>());
    case 6: return fn(std::integral_constant<int, 6>());
    case 8: return fn(std::integral_constant<int, 8>());
    default: return fn(std::integral_constant<int, 4>());
  }
}

}  // namespace
}  // namespace cg
