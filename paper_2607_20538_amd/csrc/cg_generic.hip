// General-purpose codec kernels (any supported g, n, b, backend, bf16 or binary32 input).
//
// One workgroup owns a tile of tokens of one (layer, batch, head) slice.  The tile is staged
// in LDS in binary32, the gauge z = G x of every channel group is applied on the VALU with a
// binary32 accumulator (section 3: Z[b,h,t,r] = G_{l,s,h,r} X[b,h,t,r]), and the backend of
// section 4.3 quantises the gauge-space tile from LDS: block-uniform / KIVI values one block
// per thread, KIVI keys one channel of a token group per thread.  Decode mirrors it: codes
// are unpacked and dequantised into an LDS tile, then Xhat = G^T Zhat is applied per
// channel.  These kernels carry every configuration; the MFMA kernels take over the
// large-group bf16 block-uniform case.
#include "cg_internal.h"
#include "cg_device.h"
#include "cg_zfp.h"

namespace cg {

namespace {

constexpr int kThreads = 256;

__device__ __forceinline__ size_t gauge_block(int l, int s, int h, int r, int H, int R) {
  return ((size_t(l) * 2 + s) * H + h) * R + r;
}

__device__ __forceinline__ float load_x(const ViewDev& v, size_t off) {
  return v.bf16 ? bf16_to_f32(((const uint16_t*)v.ptr)[off]) : ((const float*)v.ptr)[off];
}

// LDS row pitch of the token tiles (floats): a multiple of 4 so that rows stay 16-byte aligned
// for vector reads, offset by 4 banks from row to row
constexpr int kPad = 4;

// zs[t][i] = sum_j G_{l,s,h,r}[i%g][j] xs[t][r*g + j] for t < ntok: one binary32 FMA chain per
// element in increasing j.  With g a multiple of 4 each thread computes a 4-token x 4-channel
// block, reading 4 consecutive j of 4 rows of G and of 4 token rows per step (16-byte loads).
__device__ void gauge_tile(const float* xs, float* zs, int ntok, int d, int dp, const GaugeDev& G, int l, int s,
                           int h) {
  const int g = G.g;
  if (g % 4) {
    for (int idx = threadIdx.x; idx < ntok * d; idx += blockDim.x) {
      const int t = idx / d, i = idx - t * d;
      const int r = i / g, ii = i - r * g;
      const float* Gr = G.f32 + gauge_block(l, s, h, r, G.H, G.R) * g * g + size_t(ii) * g;
      const float* xr = xs + t * dp + r * g;
      float acc = 0.0f;
      for (int j = 0; j < g; ++j) acc = fmaf(Gr[j], xr[j], acc);
      zs[t * dp + i] = acc;
    }
    return;
  }
  const int ntb = (ntok + 3) / 4, ncb = d / 4;
  for (int idx = threadIdx.x; idx < ntb * ncb; idx += blockDim.x) {
    const int tb = idx / ncb, cb = idx - tb * ncb;
    const int t0 = 4 * tb, i0 = 4 * cb, r = i0 / g;
    const float* Gb = G.f32 + gauge_block(l, s, h, r, G.H, G.R) * g * g + size_t(i0 - r * g) * g;
    const float4 zero = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
    float acc[4][4];
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
      for (int a = 0; a < 4; ++a) acc[t][a] = 0.0f;
    for (int j = 0; j < g; j += 4) {
      float4 gv[4], xv[4];
#pragma unroll
      for (int a = 0; a < 4; ++a) gv[a] = *reinterpret_cast<const float4*>(Gb + size_t(a) * g + j);
#pragma unroll
      for (int t = 0; t < 4; ++t)
        xv[t] = t0 + t < ntok ? *reinterpret_cast<const float4*>(xs + (t0 + t) * dp + r * g + j) : zero;
#pragma unroll
      for (int t = 0; t < 4; ++t)
#pragma unroll
        for (int a = 0; a < 4; ++a) {
          acc[t][a] = fmaf(gv[a].x, xv[t].x, acc[t][a]);
          acc[t][a] = fmaf(gv[a].y, xv[t].y, acc[t][a]);
          acc[t][a] = fmaf(gv[a].z, xv[t].z, acc[t][a]);
          acc[t][a] = fmaf(gv[a].w, xv[t].w, acc[t][a]);
        }
    }
#pragma unroll
    for (int t = 0; t < 4; ++t)
      if (t0 + t < ntok) *reinterpret_cast<float4*>(zs + (t0 + t) * dp + i0) = make_float4(acc[t][0], acc[t][1], acc[t][2], acc[t][3]);
  }
}

// xs[t][i] = sum_j G_{l,s,h,r}[j][i%g] zs[t][r*g + j] (inverse gauge, G^T), the same chains and
// blocking (4 consecutive columns of G are one 16-byte read of row j).
__device__ void inverse_tile(const float* zs, float* xs, int ntok, int d, int dp, const GaugeDev& G, int l, int s,
                             int h) {
  const int g = G.g;
  if (g % 4) {
    for (int idx = threadIdx.x; idx < ntok * d; idx += blockDim.x) {
      const int t = idx / d, i = idx - t * d;
      const int r = i / g, ii = i - r * g;
      const float* Gr = G.f32 + gauge_block(l, s, h, r, G.H, G.R) * g * g + ii;
      const float* zr = zs + t * dp + r * g;
      float acc = 0.0f;
      for (int j = 0; j < g; ++j) acc = fmaf(Gr[size_t(j) * g], zr[j], acc);
      xs[t * dp + i] = acc;
    }
    return;
  }
  const int ntb = (ntok + 3) / 4, ncb = d / 4;
  for (int idx = threadIdx.x; idx < ntb * ncb; idx += blockDim.x) {
    const int tb = idx / ncb, cb = idx - tb * ncb;
    const int t0 = 4 * tb, i0 = 4 * cb, r = i0 / g;
    const float* Gb = G.f32 + gauge_block(l, s, h, r, G.H, G.R) * g * g + (i0 - r * g);
    const float4 zero = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
    float acc[4][4];
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
      for (int a = 0; a < 4; ++a) acc[t][a] = 0.0f;
    for (int j = 0; j < g; j += 4) {
      float4 gv[4], zv[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) gv[q] = *reinterpret_cast<const float4*>(Gb + size_t(j + q) * g);  // G[j+q][i0..i0+3]
#pragma unroll
      for (int t = 0; t < 4; ++t)
        zv[t] = t0 + t < ntok ? *reinterpret_cast<const float4*>(zs + (t0 + t) * dp + r * g + j) : zero;
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const float zz[4] = {zv[t].x, zv[t].y, zv[t].z, zv[t].w};
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          acc[t][0] = fmaf(gv[q].x, zz[q], acc[t][0]);
          acc[t][1] = fmaf(gv[q].y, zz[q], acc[t][1]);
          acc[t][2] = fmaf(gv[q].z, zz[q], acc[t][2]);
          acc[t][3] = fmaf(gv[q].w, zz[q], acc[t][3]);
        }
      }
    }
#pragma unroll
    for (int t = 0; t < 4; ++t)
      if (t0 + t < ntok) *reinterpret_cast<float4*>(xs + (t0 + t) * dp + i0) = make_float4(acc[t][0], acc[t][1], acc[t][2], acc[t][3]);
  }
}

// Quantise n values (stride `stride` in LDS) as one block and write its packed stream and
// side word.  n * bits is a multiple of 32.
__device__ int quantize_block_to(const float* z, int stride, int n, int bits, uint32_t* dst, uint32_t* side_dst) {
  float mn = z[0], mx = z[0];
  for (int e = 1; e < n; ++e) {
    mn = fminf(mn, z[e * stride]);
    mx = fmaxf(mx, z[e * stride]);
  }
  Side sd = make_side(mn, mx, bits);
  const float qmax = (float)((1 << bits) - 1);
  uint64_t acc = 0;
  int nbit = 0, wi = 0;
  for (int e = 0; e < n; ++e) {
    acc |= (uint64_t)quantize(z[e * stride], sd.mn, sd.inv, qmax) << nbit;
    nbit += bits;
    if (nbit >= 32) {
      dst[wi++] = (uint32_t)acc;
      acc >>= 32;
      nbit -= 32;
    }
  }
  *side_dst = sd.word;
  return sd.flags;
}

// Block-uniform (or KIVI value) rows: tile rows t < ntok go to cache positions pos0 + t.
__device__ int store_rows_blocks(const float* zs, int ntok, int d, int dp, int n, int bits, const CacheDev& k,
                                 size_t slc, int pos0) {
  int flags = 0;
  const int nb = d / n, row_bytes = d * bits / 8, blk_bytes = n * bits / 8;
  for (int w = threadIdx.x; w < ntok * nb; w += blockDim.x) {
    const int t = w / nb, kb = w - t * nb;
    const size_t row = slc * k.T_cap + pos0 + t;
    uint32_t* dst = (uint32_t*)(k.codes + row * row_bytes + size_t(kb) * blk_bytes);
    flags |= quantize_block_to(zs + t * dp + kb * n, 1, n, bits, dst, k.side + row * nb + kb);
  }
  return flags;
}

// Block-uniform token-channel tiles: tile rows [u*bt, u*bt + bt) form tile (pos0 / bt) + u; one
// (tile, channel block) per thread takes the range of its bt x n values and packs every token's
// n codes into that token's row.
__device__ int store_tiles(const float* zs, int ntile, int bt, int d, int dp, int n, int bits, const CacheDev& k,
                           size_t slc, int pos0) {
  int flags = 0;
  const int nb = d / n, row_bytes = d * bits / 8, blk_bytes = n * bits / 8;
  for (int w = threadIdx.x; w < ntile * nb; w += blockDim.x) {
    const int u = w / nb, kb = w - u * nb;
    const float* zt = zs + (u * bt) * dp + kb * n;
    float mn = zt[0], mx = zt[0];
    for (int v = 0; v < bt; ++v)
      for (int e = 0; e < n; ++e) {
        mn = fminf(mn, zt[v * dp + e]);
        mx = fmaxf(mx, zt[v * dp + e]);
      }
    const Side sd = make_side(mn, mx, bits);
    const float qmax = (float)((1 << bits) - 1);
    for (int v = 0; v < bt; ++v) {
      const size_t row = slc * k.T_cap + pos0 + u * bt + v;
      uint32_t* dst = (uint32_t*)(k.codes + row * row_bytes + size_t(kb) * blk_bytes);
      uint64_t acc = 0;
      int nbit = 0, wi = 0;
      for (int e = 0; e < n; ++e) {
        acc |= (uint64_t)quantize(zt[v * dp + e], sd.mn, sd.inv, qmax) << nbit;
        nbit += bits;
        if (nbit >= 32) {
          dst[wi++] = (uint32_t)acc;
          acc >>= 32;
          nbit -= 32;
        }
      }
    }
    k.side[(slc * (k.T_cap / bt) + (pos0 / bt + u)) * nb + kb] = sd.word;
    flags |= sd.flags;
  }
  return flags;
}

// KIVI key groups: tile rows [u*kg, u*kg + kg) form token group grp0 + u; one channel per
// thread.
__device__ int store_key_groups(const float* zs, int ngrp, int kg, int d, int dp, int bits, const CacheDev& k,
                                size_t slc, int grp0) {
  int flags = 0;
  const int cb = kg * bits / 8;
  for (int w = threadIdx.x; w < ngrp * d; w += blockDim.x) {
    const int u = w / d, ch = w - u * d;
    const size_t gi = slc * (k.T_cap / kg) + grp0 + u;
    uint32_t* dst = (uint32_t*)(k.codes + (gi * d + ch) * cb);
    flags |= quantize_block_to(zs + (u * kg) * dp + ch, dp, kg, bits, dst, k.side + gi * d + ch);
  }
  return flags;
}

__device__ void store_rows_pass(const float* zs, int ntok, int d, int dp, const CacheDev& k, size_t slc, int pos0) {
  float* out = (float*)k.codes;
  for (int idx = threadIdx.x; idx < ntok * d; idx += blockDim.x) {
    const int t = idx / d, ch = idx - t * d;
    out[(slc * k.T_cap + pos0 + t) * d + ch] = zs[t * dp + ch];
  }
}

// zfp-style rows: tile rows [4u, 4u + 4) x channels [4cb, 4cb + 4) form block (pos0 / 4 + u, cb)
__device__ int store_zfp(const float* zs, int ntok, int d, int dp, int rate, const CacheDev& k, size_t slc,
                         int pos0, const ZfpTables& tab) {
  return zfp_by_rate(rate, [&](auto R) {
    constexpr int RATE = decltype(R)::value;
    int flags = 0;
    const int nbc = d / 4;
    for (int idx = threadIdx.x; idx < (ntok / 4) * nbc; idx += blockDim.x) {
      const int u = idx / nbc, cb = idx - u * nbc;
      float v[16];
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int i = 0; i < 4; ++i) v[4 * j + i] = zs[(4 * u + j) * dp + 4 * cb + i];
      uint32_t w[4];
      flags |= zfp_encode_block<RATE>(v, tab, w);
      zfp_store<RATE>(k.codes + ((slc * (k.T_cap / 4) + pos0 / 4 + u) * nbc + cb) * size_t(2 * RATE), w);
    }
    return flags;
  });
}

__device__ void load_zfp(float* zs, int ntok, int d, int dp, int rate, const CacheDev& k, size_t slc, int pos0,
                         const ZfpTables& tab) {
  zfp_by_rate(rate, [&](auto R) {
    constexpr int RATE = decltype(R)::value;
    const int nbc = d / 4;
    for (int idx = threadIdx.x; idx < (ntok / 4) * nbc; idx += blockDim.x) {
      const int u = idx / nbc, cb = idx - u * nbc;
      uint32_t w[4];
      zfp_load<RATE>(k.codes + ((slc * (k.T_cap / 4) + pos0 / 4 + u) * nbc + cb) * size_t(2 * RATE), w);
      float v[16];
      zfp_decode_block<RATE>(w, tab, v);
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int i = 0; i < 4; ++i) zs[(4 * u + j) * dp + 4 * cb + i] = v[4 * j + i];
    }
    return 0;
  });
}

// ------------------------------------------------------------------------------------------
// encode
// ------------------------------------------------------------------------------------------
__global__ __launch_bounds__(kThreads) void enc_generic(int s, ViewDev X, int l0, GaugeDev G, CodecDev c, CacheDev k,
                                                        int t0, int tq, int TT, int* err, PageDev pt) {
  extern __shared__ float sm[];
  const int d = X.d, dp = d + kPad;
  float* xs = sm;
  float* zs = sm + TT * dp;
  const int sv = blockIdx.y;
  const int h = sv % X.H, b = (sv / X.H) % X.B, lv = sv / (X.H * X.B);
  const int l = lv + l0;
  const int tile0 = blockIdx.x * TT;
  const int ntok = min(TT, X.T - tile0);
  int crow = b;  // cache batch row: the page of a paged cache (a tile never crosses a page)
  if (pt.pages) {
    const int lp = (t0 + tile0) / pt.page_size;
    crow = lp < pt.max_pages ? pt.pages[size_t(b) * pt.max_pages + lp] : -1;
    if (crow < 0 || crow >= k.B) {
      if (threadIdx.x == 0 && err) atomicOr(err, CG_FLAG_POS_RANGE);
      return;
    }
    t0 -= lp * pt.page_size;  // positions inside the page
  }
  const size_t slc = (size_t(l) * k.B + crow) * k.H + h;
  const size_t xbase = size_t(lv) * X.sl + size_t(b) * X.sb + size_t(h) * X.sh;

  if (c.backend == CG_BACKEND_KIVI && tile0 >= tq) {
    // full-precision window: raw bf16 rows into the ring
    const int ringsz = c.win + c.kg;
    for (int idx = threadIdx.x; idx < ntok * d; idx += blockDim.x) {
      const int t = idx / d, ch = idx - t * d;
      const int tok = tile0 + t;
      k.ring[(slc * ringsz + tok % ringsz) * d + ch] = ((const uint16_t*)X.ptr)[xbase + size_t(tok) * X.st + ch];
    }
    return;
  }
  // block-uniform tiles: rows of the unfinished tile (view rows >= tq) wait raw in the
  // staging window (slot = cache position mod bt; t0 is a multiple of bt)
  const bool tiles = c.backend == CG_BACKEND_BLOCK_UNIFORM && c.bt > 1;
  const int nq = tiles ? max(0, min(ntok, tq - tile0)) : ntok;
  if (tiles) {
    for (int idx = nq * d + threadIdx.x; idx < ntok * d; idx += blockDim.x) {
      const int t = idx / d, ch = idx - t * d;
      const int tok = tile0 + t;
      k.ring[(slc * c.bt + (t0 + tok) % c.bt) * d + ch] = ((const uint16_t*)X.ptr)[xbase + size_t(tok) * X.st + ch];
    }
    if (nq == 0) return;
  }

  __shared__ ZfpTables ztab;
  if (c.backend == CG_BACKEND_ZFP) zfp_tables_init(ztab);  // read after the barriers below
  int flags = 0;
  for (int idx = threadIdx.x; idx < TT * d; idx += blockDim.x) {
    const int t = idx / d, ch = idx - t * d;
    float v = 0.0f;
    if (t < ntok) {
      v = load_x(X, xbase + size_t(tile0 + t) * X.st + ch);
      if (t < nq && !isfinite(v)) flags |= CG_FLAG_NONFINITE;  // staged rows: checked when quantised
    }
    xs[t * dp + ch] = v;
  }
  __syncthreads();
  gauge_tile(xs, zs, ntok, d, dp, G, l, s, h);
  __syncthreads();

  if (c.backend == CG_BACKEND_PASSTHROUGH) {
    store_rows_pass(zs, ntok, d, dp, k, slc, t0 + tile0);
  } else if (c.backend == CG_BACKEND_ZFP) {
    flags |= store_zfp(zs, ntok, d, dp, c.bits, k, slc, t0 + tile0, ztab);
  } else if (tiles) {
    flags |= store_tiles(zs, nq / c.bt, c.bt, d, dp, c.n, c.bits, k, slc, t0 + tile0);
  } else if (c.backend == CG_BACKEND_BLOCK_UNIFORM) {
    flags |= store_rows_blocks(zs, ntok, d, dp, c.n, c.bits, k, slc, t0 + tile0);
  } else if (s == 1) {
    flags |= store_rows_blocks(zs, ntok, d, dp, c.kvc, c.bits, k, slc, tile0);
  } else {
    flags |= store_key_groups(zs, ntok / c.kg, c.kg, d, dp, c.bits, k, slc, tile0 / c.kg);
  }
  if (flags && err) atomicOr(err, flags);
}

// ------------------------------------------------------------------------------------------
// decode
// ------------------------------------------------------------------------------------------
__global__ __launch_bounds__(kThreads) void dec_generic(int s, CacheDev k, int l0, GaugeDev G, CodecDev c, int t0,
                                                        int len, const int* pos, int pos_add, ViewDev Y, int TT,
                                                        int* err) {
  extern __shared__ float sm[];
  const int d = Y.d, dp = d + kPad;
  float* zs = sm;
  float* xs = sm + TT * dp;
  const int sv = blockIdx.y;
  const int h = sv % Y.H, b = (sv / Y.H) % Y.B, lv = sv / (Y.H * Y.B);
  const int l = lv + l0;
  const int tile0 = blockIdx.x * TT;
  int ntok = min(TT, Y.T - tile0);
  const size_t slc = (size_t(l) * k.B + b) * k.H + h;
  const size_t ybase = size_t(lv) * Y.sl + size_t(b) * Y.sb + size_t(h) * Y.sh;

  // Positions the cache holds bound the rows written: pos[b] + pos_add per row (a rolling step's
  // newest position + 1, or kv_decode's per-row lengths; outside [0, T_cap] the row is flagged
  // and skipped), else `len` for a KIVI or tile cache, otherwise every requested position (the
  // host checked the capacity).
  const bool kivi = c.backend == CG_BACKEND_KIVI;
  const bool tiles = c.backend == CG_BACKEND_BLOCK_UNIFORM && c.bt > 1;
  int held = INT_MAX;
  if (pos) {
    const int hb = pos[b] + pos_add;
    if (hb < 0 || hb > k.T_cap) {
      if (err && blockIdx.x == 0 && threadIdx.x == 0) atomicOr(err, CG_FLAG_POS_RANGE);
      return;
    }
    held = hb;
  } else if (kivi || tiles) {
    held = len;
  }
  const int p0 = t0 + tile0;  // cache position of tile row 0
  if (held != INT_MAX) ntok = min(ntok, held - p0);
  if (ntok <= 0) return;
  // KIVI quantises the first T_q positions and keeps the rest in the window, tiles the whole
  // tiles and keep the unfinished one staged; the other backends quantise every position.
  const int tq = kivi ? (held < c.win ? 0 : ((held - c.win) / c.kg) * c.kg)
                      : (tiles ? (held / c.bt) * c.bt : INT_MAX);
  const int nq = max(0, min(ntok, tq - p0));  // quantised rows of this tile

  // 1. dequantise the quantised rows into zs
  const int bits = c.bits;
  if (c.backend == CG_BACKEND_ZFP) {  // the backend is the same for the whole workgroup
    __shared__ ZfpTables ztab;
    zfp_tables_init(ztab);
    __syncthreads();
    load_zfp(zs, nq, d, dp, bits, k, slc, p0, ztab);
  }
  for (int idx = threadIdx.x; c.backend != CG_BACKEND_ZFP && idx < nq * d; idx += blockDim.x) {
    const int t = idx / d, ch = idx - t * d;
    const int p = p0 + t;
    float zv;
    if (c.backend == CG_BACKEND_PASSTHROUGH) {
      zv = ((const float*)k.codes)[(slc * k.T_cap + p) * d + ch];
    } else if (c.backend == CG_BACKEND_BLOCK_UNIFORM || s == 1) {
      const int n = c.backend == CG_BACKEND_BLOCK_UNIFORM ? c.n : c.kvc;
      const int nb = d / n, kb = ch / n;
      const size_t row = slc * k.T_cap + p;
      const uint32_t* stream = (const uint32_t*)(k.codes + row * (d * bits / 8) + size_t(kb) * (n * bits / 8));
      const uint32_t q = extract_code(stream, ch - kb * n, bits);
      const uint32_t sw = k.side[(tiles ? slc * (k.T_cap / c.bt) + p / c.bt : row) * nb + kb];
      zv = dequantize(q, f16_bits_to_f32(sw & 0xffffu), f16_bits_to_f32(sw >> 16));
    } else {
      const int kg = c.kg;
      const size_t gi = slc * (k.T_cap / kg) + p / kg;
      const uint32_t* stream = (const uint32_t*)(k.codes + (gi * d + ch) * (kg * bits / 8));
      const uint32_t q = extract_code(stream, p % kg, bits);
      const uint32_t sw = k.side[gi * d + ch];
      zv = dequantize(q, f16_bits_to_f32(sw & 0xffffu), f16_bits_to_f32(sw >> 16));
    }
    zs[t * dp + ch] = zv;
  }
  __syncthreads();
  // 2. inverse gauge
  inverse_tile(zs, xs, nq, d, dp, G, l, s, h);
  __syncthreads();
  // 3. write rows: inverse-gauged rows, then window / staged rows copied raw
  const int ringsz = tiles ? c.bt : c.win + c.kg;
  for (int idx = threadIdx.x; idx < ntok * d; idx += blockDim.x) {
    const int t = idx / d, ch = idx - t * d;
    const size_t off = ybase + size_t(tile0 + t) * Y.st + ch;
    if (t < nq) {
      const float v = xs[t * dp + ch];
      if (Y.bf16) ((uint16_t*)Y.ptr)[off] = (uint16_t)f32_to_bf16_rne(v);
      else ((float*)Y.ptr)[off] = v;
    } else if (kivi || tiles) {
      const uint16_t raw = k.ring[(slc * ringsz + (p0 + t) % ringsz) * d + ch];
      if (Y.bf16) ((uint16_t*)Y.ptr)[off] = raw;
      else ((float*)Y.ptr)[off] = bf16_to_f32(raw);
    }
  }
}

// ------------------------------------------------------------------------------------------
// rolling append: one workgroup per (layer, b, h)
// ------------------------------------------------------------------------------------------
__global__ __launch_bounds__(kThreads) void append_generic(int s, ViewDev Xn, int l0, const int* pos, GaugeDev G,
                                                           CodecDev c, CacheDev k, int* err, PageDev pt) {
  extern __shared__ float sm[];
  const int d = Xn.d, dp = d + kPad;
  const int sv = blockIdx.x;
  const int h = sv % Xn.H, b = (sv / Xn.H) % Xn.B, lv = sv / (Xn.H * Xn.B);
  const int l = lv + l0;
  const size_t xbase = size_t(lv) * Xn.sl + size_t(b) * Xn.sb + size_t(h) * Xn.sh;
  int p = pos[b];
  int row = b;  // cache batch row (the page of a paged cache)
  if (pt.pages) {
    // the position's page; a position past the table or a page outside the pool is an error
    const int lp = p >= 0 ? p / pt.page_size : -1;
    row = lp >= 0 && lp < pt.max_pages ? pt.pages[size_t(b) * pt.max_pages + lp] : -1;
    if (row < 0 || row >= k.B) {
      if (threadIdx.x == 0 && err) atomicOr(err, CG_FLAG_POS_RANGE);
      return;
    }
    p -= lp * pt.page_size;
  }
  const size_t slc = (size_t(l) * k.B + row) * k.H + h;
  if (p < 0 || p >= k.T_cap) {
    if (threadIdx.x == 0 && err) atomicOr(err, CG_FLAG_POS_RANGE);
    return;
  }
  int flags = 0;
  if (c.backend == CG_BACKEND_KIVI) {
    const int ringsz = c.win + c.kg;
    const uint16_t* src = (const uint16_t*)Xn.ptr + xbase;
    for (int ch = threadIdx.x; ch < d; ch += blockDim.x) k.ring[(slc * ringsz + p % ringsz) * d + ch] = src[ch];
    const int T = p + 1;
    if (!(T - c.win >= c.kg && (T - c.win) % c.kg == 0)) return;
    __syncthreads();
    // flush the kg oldest window tokens [T - W - kg, T - W)
    const int tb = T - c.win - c.kg;
    float* xs = sm;
    float* zs = sm + c.kg * dp;
    for (int idx = threadIdx.x; idx < c.kg * d; idx += blockDim.x) {
      const int t = idx / d, ch = idx - t * d;
      xs[t * dp + ch] = bf16_to_f32(k.ring[(slc * ringsz + (tb + t) % ringsz) * d + ch]);
    }
    __syncthreads();
    gauge_tile(xs, zs, c.kg, d, dp, G, l, s, h);
    __syncthreads();
    if (s == 0) flags |= store_key_groups(zs, 1, c.kg, d, dp, c.bits, k, slc, tb / c.kg);
    else flags |= store_rows_blocks(zs, c.kg, d, dp, c.kvc, c.bits, k, slc, tb);
  } else if (c.backend == CG_BACKEND_BLOCK_UNIFORM && c.bt > 1) {
    // stage the token; its tile is quantised once the tile's last token is there
    const uint16_t* src = (const uint16_t*)Xn.ptr + xbase;
    for (int ch = threadIdx.x; ch < d; ch += blockDim.x) k.ring[(slc * c.bt + p % c.bt) * d + ch] = src[ch];
    if ((p + 1) % c.bt == 0) {
      __syncthreads();
      const int tb = p + 1 - c.bt;
      float* xs = sm;
      float* zs = sm + c.bt * dp;
      for (int idx = threadIdx.x; idx < c.bt * d; idx += blockDim.x) {
        const int t = idx / d, ch = idx - t * d;
        const float v = bf16_to_f32(k.ring[(slc * c.bt + (tb + t) % c.bt) * d + ch]);
        if (!isfinite(v)) flags |= CG_FLAG_NONFINITE;
        xs[t * dp + ch] = v;
      }
      __syncthreads();
      gauge_tile(xs, zs, c.bt, d, dp, G, l, s, h);
      __syncthreads();
      flags |= store_tiles(zs, 1, c.bt, d, dp, c.n, c.bits, k, slc, tb);
    }
  } else {
    float* xs = sm;
    float* zs = sm + dp;
    for (int ch = threadIdx.x; ch < d; ch += blockDim.x) {
      const float v = load_x(Xn, xbase + ch);
      if (!isfinite(v)) flags |= CG_FLAG_NONFINITE;
      xs[ch] = v;
    }
    __syncthreads();
    gauge_tile(xs, zs, 1, d, dp, G, l, s, h);
    __syncthreads();
    if (c.backend == CG_BACKEND_PASSTHROUGH) store_rows_pass(zs, 1, d, dp, k, slc, p);
    else flags |= store_rows_blocks(zs, 1, d, dp, c.n, c.bits, k, slc, p);
  }
  if (flags && err) atomicOr(err, flags);
}

// KIVI tiles are exactly one key token group, so the quantised / window split (a multiple of
// the group) never cuts a tile.
int tile_tokens(const CodecDev& c) { return c.backend == CG_BACKEND_KIVI ? c.kg : 32; }

hipError_t set_smem(const void* fn, size_t bytes) {
  if (bytes <= 65536) return hipSuccess;
  return hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
}

}  // namespace

hipError_t launch_encode_generic(int s, const ViewDev& X, int l0, const GaugeDev& G, const CodecDev& c,
                                 const CacheDev& k, int t0, int tq, int* err, hipStream_t st, const PageDev& pt) {
  if (X.T == 0) return hipSuccess;
  const int TT = tile_tokens(c);
  const size_t smem = size_t(2) * TT * (X.d + kPad) * sizeof(float);
  hipError_t e = set_smem((const void*)enc_generic, smem);
  if (e != hipSuccess) return e;
  dim3 grid((X.T + TT - 1) / TT, X.L * X.B * X.H);
  hipLaunchKernelGGL(enc_generic, grid, dim3(kThreads), smem, st, s, X, l0, G, c, k, t0, tq, TT, err, pt);
  return hipGetLastError();
}

hipError_t launch_decode_generic(int s, const CacheDev& k, int l0, const GaugeDev& G, const CodecDev& c, int t0,
                                 int len, const int* pos, int pos_add, const ViewDev& Y, int* err, hipStream_t st) {
  if (Y.T == 0) return hipSuccess;
  const int TT = tile_tokens(c);
  const size_t smem = size_t(2) * TT * (Y.d + kPad) * sizeof(float);
  hipError_t e = set_smem((const void*)dec_generic, smem);
  if (e != hipSuccess) return e;
  dim3 grid((Y.T + TT - 1) / TT, Y.L * Y.B * Y.H);
  hipLaunchKernelGGL(dec_generic, grid, dim3(kThreads), smem, st, s, k, l0, G, c, t0, len, pos, pos_add, Y, TT, err);
  return hipGetLastError();
}

hipError_t launch_append(int s, const ViewDev& Xn, int l0, const int* pos, const GaugeDev& G, const CodecDev& c,
                         const CacheDev& k, int* err, hipStream_t st, const PageDev& pt) {
  const int rows = c.backend == CG_BACKEND_KIVI ? c.kg : c.bt;
  const size_t smem = size_t(2) * rows * (Xn.d + kPad) * sizeof(float);
  hipError_t e = set_smem((const void*)append_generic, smem);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(append_generic, dim3(Xn.L * Xn.B * Xn.H), dim3(kThreads), smem, st, s, Xn, l0, pos, G, c, k,
                     err, pt);
  return hipGetLastError();
}

}  // namespace cg
