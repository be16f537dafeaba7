// zfp-style fixed-rate block coder shared by the codec kernels (one copy per translation unit).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "codec_gauge.h"

namespace cg {
namespace {

// ------------------------------------------------------------------------------------------
// zfp-style fixed-rate blocks: 4 tokens x 4 channels of z, 16 rate bits each (zfp's published
// algorithm: block exponent, 30-bit fixed point, lifted 4-point transform along channels then
// tokens, sequency order, negabinary, embedded bit planes with group tests)
// ------------------------------------------------------------------------------------------
__device__ __forceinline__ int32_t wadd(int32_t a, int32_t b) { return int32_t(uint32_t(a) + uint32_t(b)); }
__device__ __forceinline__ int32_t wsub(int32_t a, int32_t b) { return int32_t(uint32_t(a) - uint32_t(b)); }
__device__ __forceinline__ int32_t wdbl(int32_t a) { return int32_t(uint32_t(a) << 1); }

// 1/16 [[4 4 4 4] [5 1 -1 -5] [-4 4 4 -4] [-2 6 -6 2]] applied to (a, b, c, e) by lifting
__device__ __forceinline__ void zfp_fwd4(int32_t& a, int32_t& b, int32_t& c, int32_t& e) {
  a = wadd(a, e) >> 1; e = wsub(e, a);
  c = wadd(c, b) >> 1; b = wsub(b, c);
  a = wadd(a, c) >> 1; c = wsub(c, a);
  e = wadd(e, b) >> 1; b = wsub(b, e);
  e = wadd(e, b >> 1); b = wsub(b, e >> 1);
}
__device__ __forceinline__ void zfp_inv4(int32_t& a, int32_t& b, int32_t& c, int32_t& e) {
  b = wadd(b, e >> 1); e = wsub(e, b >> 1);
  b = wadd(b, e); e = wsub(wdbl(e), b);
  c = wadd(c, a); a = wsub(wdbl(a), c);
  b = wadd(b, c); c = wsub(wdbl(c), b);
  e = wadd(e, a); a = wsub(wdbl(a), e);
}

// sequency position k -> block entry 4 j + i (by i + j, then i^2 + j^2, then j)
constexpr int kZfpOrder[16] = {0, 1, 4, 5, 2, 8, 6, 9, 3, 12, 10, 7, 13, 11, 14, 15};

__device__ __forceinline__ uint32_t word_of(const uint32_t (&w)[4], int i) {
  return i == 0 ? w[0] : (i == 1 ? w[1] : (i == 2 ? w[2] : w[3]));
}

// Bit stream of one block (at most 128 bits) in two 64-bit words, LSB-first.
struct ZStream {
  uint64_t lo = 0, hi = 0;
  int pos = 0, cap = 0;
  // append the k <= 32 low bits of v; past the budget only the prefix that fits is kept and
  // false is returned
  __device__ __forceinline__ bool put(uint32_t v, int k) {
    const int kk = min(k, cap - pos);
    if (kk <= 0) return k == 0;
    const uint64_t x = uint64_t(v) & ((uint64_t(1) << kk) - 1u);
    if (pos < 64) {
      lo |= x << pos;
      if (pos + kk > 64) hi |= x >> (64 - pos);
    } else {
      hi |= x << (pos - 64);
    }
    pos += kk;
    return kk == k;
  }
  // the next k <= 32 bits (bits past the block read as 0)
  __device__ __forceinline__ uint32_t peek(int k) const {
    uint64_t v;
    if (pos == 0) v = lo;
    else if (pos < 64) v = (lo >> pos) | (hi << (64 - pos));
    else v = hi >> (pos - 64);
    return k >= 32 ? uint32_t(v) : uint32_t(v) & ((1u << k) - 1u);
  }
};

// v[4 j + i]: channel i of token j.  w: the block's 16 rate bits, LSB-first.  Returns flags.
// Each plane is emitted in chunks: the verbatim bits of the significant coefficients at once,
// then per 1 found by the group tests one chunk (test bit, the zeros before the 1, the 1 unless
// it is the last candidate's, which is implied), then a closing 0 test bit if candidates remain;
// leading planes with no 1 at all are one run of 0 test bits.
__device__ int zfp_encode_block(const float (&v)[16], int rate, uint32_t (&w)[4]) {
  ZStream st;
  st.cap = 16 * rate;
  int flags = 0;
  float amax = 0.0f;
#pragma unroll
  for (int k = 0; k < 16; ++k) {
    if (!isfinite(v[k])) flags = CG_FLAG_NONFINITE;
    else amax = fmaxf(amax, fabsf(v[k]));
  }
  if (!flags && amax != 0.0f) {
    int e;
    frexpf(amax, &e);
    e = max(e, -126);
    st.put(1u | (uint32_t(e + 127) << 1), 9);
    int32_t q[16];
#pragma unroll
    for (int k = 0; k < 16; ++k) q[k] = int32_t(ldexpf(v[k], 30 - e));  // exact scaling, truncation
#pragma unroll
    for (int j = 0; j < 4; ++j) zfp_fwd4(q[4 * j], q[4 * j + 1], q[4 * j + 2], q[4 * j + 3]);
#pragma unroll
    for (int i = 0; i < 4; ++i) zfp_fwd4(q[i], q[4 + i], q[8 + i], q[12 + i]);
    uint32_t u[16], any = 0u;
#pragma unroll
    for (int k = 0; k < 16; ++k) {
      u[k] = (uint32_t(q[kZfpOrder[k]]) + 0xAAAAAAAAu) ^ 0xAAAAAAAAu;
      any |= u[k];
    }
    // planes above the highest set bit: a 0 test bit each (no coefficient is significant yet)
    const int top = any ? 31 - __builtin_clz(any) : -1;
    bool ok = st.put(0u, 31 - top);
    int n = 0;
    for (int plane = top; ok && plane >= 0; --plane) {
      uint32_t x = 0u;
#pragma unroll
      for (int c = 0; c < 16; ++c) x |= __builtin_amdgcn_ubfe(u[c], plane, 1) << c;  // v_bfe_u32 + v_lshl_or_b32
      if (n && !st.put(x, n)) break;
      x >>= n;
      while (n < 16) {
        if (x == 0u) {
          ok = st.put(0u, 1);
          break;
        }
        const int p = __builtin_ctz(x);
        if (n + p == 15) {  // the last candidate holds the 1: test bit and p zeros
          ok = st.put(1u, 1 + p);
          n = 16;
          break;
        }
        if (!(ok = st.put(1u | (1u << (p + 1)), p + 2))) break;
        n += p + 1;
        x >>= p + 1;
      }
    }
  } else {
    st.put(0u, 1);
  }
  w[0] = uint32_t(st.lo);
  w[1] = uint32_t(st.lo >> 32);
  w[2] = uint32_t(st.hi);
  w[3] = uint32_t(st.hi >> 32);
  return flags;
}

__device__ void zfp_decode_block(const uint32_t (&w)[4], int rate, float (&v)[16]) {
  ZStream st;
  st.cap = 16 * rate;
  st.lo = uint64_t(w[0]) | (uint64_t(w[1]) << 32);
  st.hi = uint64_t(w[2]) | (uint64_t(w[3]) << 32);
#pragma unroll
  for (int k = 0; k < 16; ++k) v[k] = 0.0f;
  const uint32_t head = st.peek(9);
  if (!(head & 1u) || st.cap < 9) return;
  st.pos = 9;
  const int e = int(head >> 1) - 127;
  uint32_t u[16];
#pragma unroll
  for (int k = 0; k < 16; ++k) u[k] = 0u;
  int n = 0;
  bool done = false;
  for (int plane = 31; plane >= 0 && !done; --plane) {
    uint32_t x = 0u;
    int avail = st.cap - st.pos;
    if (avail <= 0) break;
    if (n) {
      const int k = min(n, avail);
      x = st.peek(k);
      st.pos += k;
      if (k < n) done = true;
    }
    while (!done && n < 16) {
      avail = st.cap - st.pos;
      if (avail <= 0) {
        done = true;
        break;
      }
      const uint32_t t = st.peek(1);
      st.pos += 1;
      if (!t) break;
      // explicit coefficient bits before the last candidate, as far as the budget reaches
      const int m = 15 - n;
      avail = st.cap - st.pos;
      const int k = min(m, avail);
      const uint32_t bits = k ? st.peek(k) : 0u;
      if (bits) {
        const int p = __builtin_ctz(bits);
        st.pos += p + 1;
        x |= 1u << (n + p);
        n += p + 1;
      } else if (avail >= m) {  // all zero up to the last candidate: its 1 is implied
        st.pos += m;
        x |= 1u << 15;
        n = 16;
      } else {
        st.pos = st.cap;
        done = true;
      }
    }
#pragma unroll
    for (int c = 0; c < 16; ++c) u[c] |= ((x >> c) & 1u) << plane;
  }
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

}  // namespace
}  // namespace cg
