// Decode-phase attention over the compressed caches, with the inverse gauge folded into the
// attention consumer instead of materialising Xhat: the paper leaves this fusion to deployments
// (section 4.1 on where the recovery can go; section 6: its timings charge explicit recovery).
//
// For one query q of KV head h (query heads h * grp .. h * grp + grp - 1 share that head, as in
// grouped-query attention) over positions [0, len):
//   key of position t:   Khat_t = G_K^T zhat^K_t (gauge-space token) or the raw bf16 token
//                        (KIVI window, staged tokens of an unfinished block-uniform tile)
//   score:               s_t = scale q . Khat_t = (scale G_K q) . zhat^K_t   (G orthogonal)
//   output:              o = sum_t p_t Vhat_t = G_V^T (sum_t p_t zhat^V_t) + sum_raw p_t x^V_t,
//                        p = softmax(s)
// so the gauge is applied once to the query and once to the output, never per cached token.
// The token range of a row is cut into splits (flash-decoding); each workgroup keeps a running
// maximum, normaliser and unnormalised accumulators, and a combine kernel merges the splits and
// applies G_V^T.  A row with no positions gets a zero output.
#include <algorithm>
#include <mutex>
#include <type_traits>

#include "cg_internal.h"
#include "cg_device.h"
#include "cg_mfma_util.h"

namespace cg {

namespace {

constexpr int kAThreads = 256;  // four waves
constexpr int kJQ = 8;          // query heads per workgroup (at most)
constexpr int kATile = 64;      // positions per wave step (one per lane)

__device__ __forceinline__ size_t gauge_block(int l, int s, int h, int r, int H, int R) {
  return ((size_t(l) * 2 + s) * H + h) * R + r;
}

__device__ __forceinline__ float wave_max(float v) {
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}
__device__ __forceinline__ float wave_sum(float v) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

// Positions row b holds and how many of them are quantised (the rest raw in the window or the
// staging tile).  Rows with a count outside [0, T_cap] hold nothing and raise a flag.
struct RowSpan {
  int held, tq;
};
__device__ __forceinline__ RowSpan row_span(const AttendDev& a, const CodecDev& c, int b) {
  RowSpan r;
  r.held = a.lens ? a.lens[b] : a.len;
  if (r.held < 0 || r.held > a.cap) r.held = 0;
  if (c.backend == CG_BACKEND_KIVI) r.tq = r.held < c.win ? 0 : ((r.held - c.win) / c.kg) * c.kg;
  else if (c.backend == CG_BACKEND_BLOCK_UNIFORM && c.bt > 1) r.tq = (r.held / c.bt) * c.bt;
  else r.tq = r.held;
  return r;
}

// Cache slice and position offset of the step of batch row b starting at position t0 (a
// step never crosses a page): with a page table, the slice of the page holding t0 and the
// page's first position; without, the row's own slice and 0.  Returns false (and flags) when
// the table sends the step outside the pool.
__device__ __forceinline__ bool step_slice(const AttendDev& a, int l, int b, int h, int t0, size_t& slc, int& off) {
  if (!a.pt.pages) {
    slc = (size_t(l) * a.kc.B + b) * a.kc.H + h;
    off = 0;
    return true;
  }
  const int lp = t0 / a.pt.page_size;
  const int pg = lp < a.pt.max_pages ? a.pt.pages[size_t(b) * a.pt.max_pages + lp] : -1;
  if (pg < 0 || pg >= a.kc.B) {
    if (a.err) atomicOr(a.err, CG_FLAG_POS_RANGE);
    return false;
  }
  slc = (size_t(l) * a.kc.B + pg) * a.kc.H + h;
  off = lp * a.pt.page_size;
  return true;
}

// zhat of channel ch at quantised cache position p of slice slc (section 4.3 decode).
__device__ __forceinline__ float zhat_at(const CacheDev& k, const CodecDev& c, int s, size_t slc, int p, int ch,
                                         int d) {
  if (c.backend == CG_BACKEND_PASSTHROUGH) return ((const float*)k.codes)[(slc * k.T_cap + p) * d + ch];
  const int bits = c.bits;
  uint32_t q, sw;
  if (c.backend == CG_BACKEND_BLOCK_UNIFORM || s == 1) {
    // token rows: the d/n blocks of a row form one LSB-first stream
    const int n = c.backend == CG_BACKEND_BLOCK_UNIFORM ? c.n : c.kvc;
    const size_t row = slc * k.T_cap + p;
    q = extract_code((const uint32_t*)(k.codes + row * (d * bits / 8)), ch, bits);
    sw = k.side[(c.bt > 1 ? slc * (k.T_cap / c.bt) + p / c.bt : row) * (d / n) + ch / n];
  } else {
    // KIVI keys: one stream per (token group, channel)
    const int kg = c.kg;
    const size_t gi = slc * (k.T_cap / kg) + p / kg;
    q = extract_code((const uint32_t*)(k.codes + (gi * d + ch) * (kg * bits / 8)), p % kg, bits);
    sw = k.side[gi * d + ch];
  }
  return dequantize(q, f16_bits_to_f32(sw & 0xffffu), f16_bits_to_f32(sw >> 16));
}

__device__ __forceinline__ float raw_at(const CacheDev& k, const CodecDev& c, size_t slc, int p, int ch, int d) {
  const int ringsz = c.backend == CG_BACKEND_KIVI ? c.win + c.kg : c.bt;
  return bf16_to_f32(k.ring[(slc * ringsz + p % ringsz) * d + ch]);
}

// Channels ch0 .. ch0 + 7 (ch0 % 8 == 0) of cache position p: raw bf16 tokens (raw) or the
// dequantised gauge-space values, with as few loads as the layout allows (one or two dwords of a
// code row and one side word per block; eight streams for KIVI keys).
__device__ __forceinline__ void load8(const CacheDev& k, const CodecDev& c, int s, size_t slc, int p, int ch0, int d,
                                      bool raw, float (&out)[8]) {
  if (raw) {
    const int ringsz = c.backend == CG_BACKEND_KIVI ? c.win + c.kg : c.bt;
    const uint4 v = *reinterpret_cast<const uint4*>(k.ring + (slc * ringsz + p % ringsz) * d + ch0);
    const uint32_t wv[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      out[2 * e] = __uint_as_float(wv[e] << 16);
      out[2 * e + 1] = __uint_as_float(wv[e] & 0xffff0000u);
    }
    return;
  }
  if (c.backend == CG_BACKEND_PASSTHROUGH) {
    const float* src = (const float*)k.codes + (slc * k.T_cap + p) * d + ch0;
    const float4 a0 = *reinterpret_cast<const float4*>(src), a1 = *reinterpret_cast<const float4*>(src + 4);
    out[0] = a0.x; out[1] = a0.y; out[2] = a0.z; out[3] = a0.w;
    out[4] = a1.x; out[5] = a1.y; out[6] = a1.z; out[7] = a1.w;
    return;
  }
  const int bits = c.bits;
  const uint32_t mask = (1u << bits) - 1u;
  if (c.backend == CG_BACKEND_BLOCK_UNIFORM || s == 1) {
    const int n = c.backend == CG_BACKEND_BLOCK_UNIFORM ? c.n : c.kvc;
    const size_t row = slc * k.T_cap + p;
    const int rw = d * bits / 32;  // dwords per code row (n b is a multiple of 32)
    const uint32_t* w = reinterpret_cast<const uint32_t*>(k.codes + row * (d * bits / 8));
    const int byte = ch0 * bits / 8, d0 = byte >> 2;
    const uint64_t chunk = ((uint64_t(w[min(d0 + 1, rw - 1)]) << 32) | w[d0]) >> ((byte & 3) * 8);
    const uint32_t* side = k.side + (c.bt > 1 ? slc * (k.T_cap / c.bt) + p / c.bt : row) * (d / n);
    const uint32_t s0 = side[ch0 / n], s1 = side[(ch0 + 4) / n];  // blocks of 4 channels at least
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const uint32_t sw = e < 4 ? s0 : s1;
      const uint32_t q = uint32_t(chunk >> (bits * e)) & mask;
      out[e] = dequantize(q, f16_bits_to_f32(sw & 0xffffu), f16_bits_to_f32(sw >> 16));
    }
    return;
  }
  // KIVI keys: one stream per (token group, channel)
  const int kg = c.kg;
  const size_t gi = slc * (k.T_cap / kg) + p / kg;
  const int cb = kg * bits / 8, bit = (p % kg) * bits, wd = bit >> 5, off = bit & 31;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const uint32_t* st = reinterpret_cast<const uint32_t*>(k.codes + (gi * d + ch0 + e) * cb);
    uint32_t v = st[wd] >> off;
    if (off + bits > 32) v |= st[wd + 1] << (32 - off);
    const uint32_t sw = k.side[gi * d + ch0 + e];
    out[e] = dequantize(v & mask, f16_bits_to_f32(sw & 0xffffu), f16_bits_to_f32(sw >> 16));
  }
}

// o_i = (sum_j G_V[j][i] acc_j + accr_i) / lsum for the group of channel i, written to the output
// view (bf16 rounded to nearest even, or binary32).  acc: LDS [nj][d].
__device__ void finalize_rows(const AttendDev& a, const GaugeDev& G, const float* acc, const float* accr,
                              const float* lsum, int nj, int lv, int b, int h, int hq0) {
  const int d = a.q.d, g = G.g, l = lv + a.l0;
  for (int idx = threadIdx.x; idx < nj * d; idx += blockDim.x) {
    const int jj = idx / d, i = idx - jj * d;
    const int r = i / g, ii = i - r * g;
    const float* Gc = G.f32 + gauge_block(l, 1, h, r, G.H, G.R) * g * g + ii;
    const float* z = acc + jj * d + r * g;
    float x = 0.0f;
    for (int j = 0; j < g; ++j) x = fmaf(Gc[size_t(j) * g], z[j], x);
    if (accr) x += accr[jj * d + i];
    const float ls = lsum[jj];
    const float o = ls > 0.0f ? x / ls : 0.0f;
    const size_t off = size_t(lv) * a.o.sl + size_t(b) * a.o.sb + size_t(hq0 + jj) * a.o.sh + i;
    if (a.o.bf16) ((uint16_t*)a.o.ptr)[off] = (uint16_t)f32_to_bf16_rne(o);
    else ((float*)a.o.ptr)[off] = o;
  }
}

// ------------------------------------------------------------------------------------------
// general kernel: any backend, group size and head dimension; one workgroup per
// (layer, batch row, KV head, query chunk, split)
// ------------------------------------------------------------------------------------------
// The workgroup walks its positions 64 at a time: the keys of the step are dequantised into an
// LDS tile by all threads (consecutive threads on consecutive channels of a row), each
// (position, query) score is a binary32 FMA chain over the channels read from LDS (gauge-space
// query for quantised positions, the raw query for raw ones), one wave updates the running
// maximum, the weights and the normalisers, the values of the step replace the keys in the
// tile, and each thread folds the step into its (query, channel) accumulators (rescaled by
// exp(m_old - m_new)), quantised positions into the gauge-space sums, raw ones into the raw sums.
constexpr int kGTile = 64;  // positions per step
constexpr int kGAcc = 8;    // (query, channel) accumulators per thread: kJQ * d / 256 for d <= 256

__global__ __launch_bounds__(kAThreads) void att_generic(AttendDev a, GaugeDev G, CodecDev c) {
  extern __shared__ float sm[];
  const int d = a.q.d, H = a.kc.H, B = a.q.B;
  const int dp = d + 4;                 // tile row pitch (16-byte aligned rows)
  float* qg = sm;                       // [kJQ][d] scale * G_K q
  float* qr = qg + kJQ * d;             // [kJQ][d] scale * q
  float* tile = qr + kJQ * d;           // [kGTile][dp] keys, then values of the step
  float* pw = tile + kGTile * dp;       // [kJQ][kGTile] scores, then weights of the step
  float* st = pw + kJQ * kGTile;        // [3][kJQ] running max, normaliser, step factor

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int sp = blockIdx.x;
  int sv = blockIdx.y;
  const int qc = sv % a.nqc;
  sv /= a.nqc;
  const int h = sv % H, b = (sv / H) % B, lv = sv / (H * B);
  const int l = lv + a.l0;
  const int j0 = qc * kJQ, nj = min(kJQ, a.grp - j0);
  const int hq0 = h * a.grp + j0;  // first query head of this workgroup

  if (tid == 0 && a.lens && sp == 0 && qc == 0 && h == 0 && lv == 0) {
    const int n = a.lens[b];
    if ((n < 0 || n > a.cap) && a.err) atomicOr(a.err, CG_FLAG_POS_RANGE);
  }
  const RowSpan rs = row_span(a, c, b);
  const int t_begin = sp * a.chunk, t_end = min(rs.held, t_begin + a.chunk);

  // 1. queries: raw (scaled) and gauged (z_i = sum_j G_K[i][j] q_j, scaled)
  for (int idx = tid; idx < kJQ * d; idx += kAThreads) {
    const int jj = idx / d, ch = idx - jj * d;
    float v = 0.0f;
    if (jj < nj) {
      const size_t off = size_t(lv) * a.q.sl + size_t(b) * a.q.sb + size_t(hq0 + jj) * a.q.sh + ch;
      v = a.q.bf16 ? bf16_to_f32(((const uint16_t*)a.q.ptr)[off]) : ((const float*)a.q.ptr)[off];
    }
    qr[idx] = v;
  }
  if (tid < kJQ) {
    st[tid] = -INFINITY;
    st[kJQ + tid] = 0.0f;
  }
  __syncthreads();
  {
    const int g = G.g;
    for (int idx = tid; idx < kJQ * d; idx += kAThreads) {
      const int jj = idx / d, i = idx - jj * d;
      const int r = i / g, ii = i - r * g;
      const float* Gr = G.f32 + gauge_block(l, 0, h, r, G.H, G.R) * g * g + size_t(ii) * g;
      const float* x = qr + jj * d + r * g;
      float z = 0.0f;
      for (int j = 0; j < g; ++j) z = fmaf(Gr[j], x[j], z);
      qg[idx] = a.scale * z;
    }
  }
  __syncthreads();
  for (int idx = tid; idx < kJQ * d; idx += kAThreads) qr[idx] *= a.scale;

  // this thread's accumulators: pairs tid + 256 k -> (query jj, channel ch)
  const int npair = kJQ * d;
  float acc[kGAcc], accr[kGAcc];
#pragma unroll
  for (int k = 0; k < kGAcc; ++k) acc[k] = accr[k] = 0.0f;

  for (int t0 = t_begin; t0 < t_end; t0 += kGTile) {
    const int nt = min(kGTile, t_end - t0);
    size_t sslc;
    int poff;
    if (!step_slice(a, l, b, h, t0, sslc, poff)) continue;  // uniform over the workgroup
    __syncthreads();  // the previous step's values are folded; qr / qg written
    // 2. keys of the step, 8 channels per thread
    const int d8 = d / 8;
    for (int idx = tid; idx < nt * d8; idx += kAThreads) {
      const int t = idx / d8, c8 = idx - t * d8;
      const int p = t0 + t;
      float v[8];
      load8(a.kc, c, 0, sslc, p - poff, 8 * c8, d, p >= rs.tq, v);
      float* dst = tile + t * dp + 8 * c8;
      *reinterpret_cast<float4*>(dst) = make_float4(v[0], v[1], v[2], v[3]);
      *reinterpret_cast<float4*>(dst + 4) = make_float4(v[4], v[5], v[6], v[7]);
    }
    __syncthreads();
    // 3. scores: thread (position t, query pair jq, jq + 4) reads the key row once
    {
      const int t = tid & (kGTile - 1), jq = tid >> 6;
      float s0 = -INFINITY, s1 = -INFINITY;
      if (t < nt) {
        const float* q = (t0 + t >= rs.tq ? qr : qg);
        const float* q0 = q + jq * d;
        const float* q1 = q + (jq + 4) * d;
        const float* kr = tile + t * dp;
        s0 = s1 = 0.0f;
        for (int ch = 0; ch < d; ch += 4) {
          const float4 kv = *reinterpret_cast<const float4*>(kr + ch);
          const float4 a0 = *reinterpret_cast<const float4*>(q0 + ch);
          const float4 a1 = *reinterpret_cast<const float4*>(q1 + ch);
          s0 = fmaf(a0.x, kv.x, s0);
          s0 = fmaf(a0.y, kv.y, s0);
          s0 = fmaf(a0.z, kv.z, s0);
          s0 = fmaf(a0.w, kv.w, s0);
          s1 = fmaf(a1.x, kv.x, s1);
          s1 = fmaf(a1.y, kv.y, s1);
          s1 = fmaf(a1.z, kv.z, s1);
          s1 = fmaf(a1.w, kv.w, s1);
        }
      }
      pw[jq * kGTile + t] = s0;
      pw[(jq + 4) * kGTile + t] = s1;
    }
    __syncthreads();
    // 4. online softmax (wave 0, lane = position): new maximum, weights, normaliser, factor
    if (w == 0) {
      for (int jj = 0; jj < nj; ++jj) {
        const float s = pw[jj * kGTile + lane];
        const float mold = st[jj];
        const float mnew = fmaxf(mold, wave_max(s));
        const float pv = lane < nt ? __expf(s - mnew) : 0.0f;
        const float sum = wave_sum(pv);
        pw[jj * kGTile + lane] = pv;
        if (lane == 0) {
          const float alpha = __expf(mold - mnew);  // exp(-inf) = 0 on the first step
          st[jj] = mnew;
          st[kJQ + jj] = st[kJQ + jj] * alpha + sum;
          st[2 * kJQ + jj] = alpha;
        }
      }
    }
    // 5. values of the step (the keys are no longer read)
    for (int idx = tid; idx < nt * d8; idx += kAThreads) {
      const int t = idx / d8, c8 = idx - t * d8;
      const int p = t0 + t;
      float v[8];
      load8(a.vc, c, 1, sslc, p - poff, 8 * c8, d, p >= rs.tq, v);
      float* dst = tile + t * dp + 8 * c8;
      *reinterpret_cast<float4*>(dst) = make_float4(v[0], v[1], v[2], v[3]);
      *reinterpret_cast<float4*>(dst + 4) = make_float4(v[4], v[5], v[6], v[7]);
    }
    __syncthreads();
    // 6. fold the step into the accumulators (quantised positions of the step come first)
    const int nq = min(nt, max(0, rs.tq - t0));
    int pj[kGAcc], pc[kGAcc];
#pragma unroll
    for (int k = 0; k < kGAcc; ++k) {
      const int pi = tid + kAThreads * k;
      pj[k] = pi < npair ? pi / d : kJQ;  // kJQ: no pair
      pc[k] = pi < npair ? pi - pj[k] * d : 0;
      const float alpha = pj[k] < nj ? st[2 * kJQ + pj[k]] : 0.0f;
      acc[k] *= alpha;
      accr[k] *= alpha;
    }
    if (kAThreads % d == 0) {
      // every pair of this thread has channel tid % d: one tile read per position
      const int ch = tid % d;
      for (int t = 0; t < nq; ++t) {
        const float v = tile[t * dp + ch];
#pragma unroll
        for (int k = 0; k < kGAcc; ++k)
          if (pj[k] < nj) acc[k] = fmaf(pw[pj[k] * kGTile + t], v, acc[k]);
      }
      for (int t = nq; t < nt; ++t) {
        const float v = tile[t * dp + ch];
#pragma unroll
        for (int k = 0; k < kGAcc; ++k)
          if (pj[k] < nj) accr[k] = fmaf(pw[pj[k] * kGTile + t], v, accr[k]);
      }
    } else {
      for (int t = 0; t < nt; ++t) {
        const bool raw = t >= nq;
#pragma unroll
        for (int k = 0; k < kGAcc; ++k) {
          if (pj[k] < nj) {
            const float pv = pw[pj[k] * kGTile + t], v = tile[t * dp + pc[k]];
            if (raw) accr[k] = fmaf(pv, v, accr[k]);
            else acc[k] = fmaf(pv, v, acc[k]);
          }
        }
      }
    }
  }
  __syncthreads();

  // 7. results: the accumulators into LDS (qg / qr are free), then finalize or write partials
  float* macc = qg;
  float* maccr = qr;
#pragma unroll
  for (int k = 0; k < kGAcc; ++k) {
    const int pi = tid + kAThreads * k;
    if (pi < npair) {
      macc[pi] = acc[k];
      maccr[pi] = accr[k];
    }
  }
  __syncthreads();
  if (a.nsplit == 1) {
    finalize_rows(a, G, macc, maccr, st + kJQ, nj, lv, b, h, hq0);
    return;
  }
  const size_t pstride = size_t(2 + 2 * d);
  for (int jj = 0; jj < nj; ++jj) {
    float* P = a.part + ((((size_t(lv) * B + b) * a.Hq + hq0 + jj) * a.nsplit) + sp) * pstride;
    for (int idx = tid; idx < 2 + 2 * d; idx += kAThreads) {
      float v;
      if (idx == 0) v = st[jj];
      else if (idx == 1) v = st[kJQ + jj];
      else if (idx < 2 + d) v = macc[jj * d + idx - 2];
      else v = maccr[jj * d + idx - 2 - d];
      P[idx] = v;
    }
  }
}

// ------------------------------------------------------------------------------------------
// combine: one workgroup per (layer, batch row, KV head, query chunk)
// ------------------------------------------------------------------------------------------
__global__ __launch_bounds__(kAThreads) void att_combine(AttendDev a, GaugeDev G) {
  extern __shared__ float sm[];
  const int d = a.q.d, H = a.kc.H, B = a.q.B;
  float* macc = sm;             // [kJQ][d]
  float* maccr = macc + kJQ * d;  // [kJQ][d]
  float* mm = maccr + kJQ * d;    // [2][kJQ]
  int sv = blockIdx.x;
  const int qc = sv % a.nqc;
  sv /= a.nqc;
  const int h = sv % H, b = (sv / H) % B, lv = sv / (H * B);
  const int j0 = qc * kJQ, nj = min(kJQ, a.grp - j0);
  const int hq0 = h * a.grp + j0;
  const size_t pstride = size_t(2 + 2 * d);
  auto part = [&](int jj, int sp) {
    return a.part + ((((size_t(lv) * B + b) * a.Hq + hq0 + jj) * a.nsplit) + sp) * pstride;
  };
  if (threadIdx.x < nj) {
    const int jj = threadIdx.x;
    float M = -INFINITY, L = 0.0f;
    for (int sp = 0; sp < a.nsplit; ++sp) M = fmaxf(M, part(jj, sp)[0]);
    for (int sp = 0; sp < a.nsplit; ++sp) {
      const float* P = part(jj, sp);
      if (P[0] != -INFINITY) L += P[1] * __expf(P[0] - M);
    }
    mm[jj] = M;
    mm[kJQ + jj] = L;
  }
  __syncthreads();
  for (int idx = threadIdx.x; idx < nj * 2 * d; idx += kAThreads) {
    const int jj = idx / (2 * d), e = idx - jj * 2 * d;
    const float M = mm[jj];
    float v = 0.0f;
    for (int sp = 0; sp < a.nsplit; ++sp) {
      const float* P = part(jj, sp);
      if (P[0] != -INFINITY) v += P[2 + e] * __expf(P[0] - M);
    }
    if (e < d) macc[jj * d + e] = v;
    else maccr[jj * d + e - d] = v;
  }
  __syncthreads();
  finalize_rows(a, G, macc, maccr, mm + kJQ, nj, lv, b, h, hq0);
}

// ------------------------------------------------------------------------------------------
// matrix-core kernel: block-uniform caches with one range per token and block (TB = 1) or per
// 16-token tile and block (TB = 16), d = 128, blocks of 64 or 128 channels (NBLK = 2 or 1
// blocks per row)
// ------------------------------------------------------------------------------------------
// Both contractions run on v_mfma_f32_16x16x32_bf16 with the codes entering as the exact bf16
// values B = 1 + q 2^-k (code_frag; 8-bit codes as q), so zhat = mn + sc k (B - 1) and
//   scores  s_t = sum_blk [ (mn - k sc) Q_blk + k sc (qt . B_t)_blk ],  Q_blk = sum_blk qt
//   values  sum_t p_t zhat_t,c = sum_t (p mn - w)_t + sum_t w_t B_t,c,  w_t = k p_t sc_t
// where the binary32 operands qt (scale G_K q) and w enter as two bf16 planes hi + lo and the
// offset terms Q and sum w are formed from the same planes, so the split only perturbs them by
// 2^-17 relative (what multiplies B - 1, i.e. the code itself).
//   scores: A = qt planes, rows (query j, block, plane), block rows zero outside their block;
//           B = the codes of 16 tokens (lane = token n, lane group = 32-channel region);
//           D lane (token n, group) holds the rows of query group (NBLK = 2) or of queries
//           2 group, 2 group + 1 (NBLK = 1), folded in-lane with the token's side words.
//   values: A = w planes, rows as above (w of the row's block), K = 32 tokens;
//           B = for lane (column c, group) the codes of channel 8c + nt of tokens
//           8 group .. 8 group + 7 (N-tile nt): each lane reads its 8-code chunk of 8 rows and
//           builds the 8 N-tile fragments from them, a transpose done in registers.
// A wave takes 32 positions per step (steps w, w + 4, ... of the split); the running maximum
// of every query lives in the lanes of its D rows, the per-step probabilities and value side
// words go through a small per-wave LDS buffer to the lanes building the value A operand.
// With tiles, a step covers two whole tiles (steps start at multiples of 32) and the side word
// of a position is its tile's; the at most 15 staged raw positions after the last whole tile
// are scored with the raw query by the workgroup whose split holds them, and enter the merge of
// the waves as one more partial softmax with raw value sums.
typedef float f32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ f32x4_t mfma16(const bf16x8_t& a, const bf16x8_t& b, const f32x4_t& c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ float row16_max(float v) {
  v = fmaxf(v, dpp_mov<0xB1>(v));   // quad_perm [1,0,3,2]
  v = fmaxf(v, dpp_mov<0x4E>(v));   // quad_perm [2,3,0,1]
  v = fmaxf(v, dpp_mov<0x124>(v));  // row_ror:4
  return fmaxf(v, dpp_mov<0x128>(v));  // row_ror:8
}
__device__ __forceinline__ float row16_sum(float v) {
  v += dpp_mov<0xB1>(v);
  v += dpp_mov<0x4E>(v);
  v += dpp_mov<0x124>(v);
  return v + dpp_mov<0x128>(v);
}

// Channel (within a lane's 32-channel region) of element e of K-step u, in code_frag's order.
template <int BITS>
__device__ __forceinline__ int frag_chan(int u, int e) {
  if constexpr (BITS == 4 || BITS == 6) return 8 * u + ((e & 1) ? 4 : 0) + (e >> 1);
  else if constexpr (BITS == 2 || BITS == 3) return 16 * (u >> 1) + 4 * (u & 1) + ((e & 1) ? 8 : 0) + (e >> 1);
  else return 8 * u + e;
}

// The 8-code chunk of channels 8c .. 8c + 7 of a packed row (BITS bytes from byte c BITS) from
// the dword holding its first byte (w0) and the next one (w1), its first bit at `sh` of w0:
// lo / hi = the chunk's bytes 0..3 / 4..7.
template <int BITS>
__device__ __forceinline__ void vchunk(uint32_t w0, uint32_t w1, uint32_t sh, uint32_t& lo, uint32_t& hi) {
  if constexpr (BITS == 4) {
    lo = w0;
    hi = 0u;
  } else if constexpr (BITS == 2) {
    lo = w0 >> sh;
    hi = 0u;
  } else if constexpr (BITS == 8) {
    lo = w0;
    hi = w1;
  } else {
    lo = __builtin_amdgcn_alignbit(w1, w0, sh);
    hi = w1 >> sh;
  }
}

// Value B fragment of N-tile k: code k of the 8 tokens' chunks as bf16 1 + q 2^-BITS (8 bits: q
// itself), token pair (2i, 2i + 1) in dword i.  4 and 6 bits: one byte permute puts the two
// tokens' bytes holding code k 16 bits apart, one shift aligns the code with the mantissa.
template <int BITS>
__device__ __forceinline__ bf16x8_t vfrag(const uint32_t (&lo)[8], const uint32_t (&hi)[8], int k, uint32_t one) {
  constexpr uint32_t M = (1u << BITS) - 1u;
  u32x4_t f;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const uint32_t a0 = lo[2 * i], a1 = lo[2 * i + 1];
    if constexpr (BITS == 4) {
      // code k in byte k/2 (low nibble for even k)
      const uint32_t b = uint32_t(k >> 1);
      const uint32_t x = __builtin_amdgcn_perm(a1, a0, b | (0x0Cu << 8) | ((b + 4) << 16) | (0x0Cu << 24));
      f[i] = (k & 1) ? (((x >> 1) & 0x00780078u) | one) : (((x << 3) & 0x00780078u) | one);
    } else if constexpr (BITS == 6) {
      const int bit = 6 * k, ob = bit >> 3, r = bit & 7;
      uint32_t x;
      if (ob <= 2 || (ob == 3 && r == 0)) {
        // codes 0..4: bytes ob, ob + 1 (or byte 3 alone) of lo
        const uint32_t o0 = uint32_t(ob), o1 = uint32_t(min(ob + 1, 3));
        x = __builtin_amdgcn_perm(a1, a0, o0 | (o1 << 8) | ((o0 + 4) << 16) | ((o1 + 4) << 24));
      } else if (ob == 3) {
        // code 5 straddles byte 3 of lo and byte 0 of hi: bytes 3..6 of the chunk first
        const uint32_t m0 = __builtin_amdgcn_alignbit(hi[2 * i], a0, 24);
        const uint32_t m1 = __builtin_amdgcn_alignbit(hi[2 * i + 1], a1, 24);
        x = __builtin_amdgcn_perm(m1, m0, 0x05040100u);
      } else {
        // codes 6, 7: bytes ob - 4, ob - 3 of hi
        const uint32_t h0 = uint32_t(ob - 4), h1 = uint32_t(ob - 3);
        x = __builtin_amdgcn_perm(hi[2 * i + 1], hi[2 * i], h0 | (h1 << 8) | ((h0 + 4) << 16) | ((h1 + 4) << 24));
      }
      // the code sits at bit r of each half: move it to mantissa bits 1..6
      const uint32_t y = r >= 1 ? (x >> (r - 1)) : (x << 1);
      f[i] = (y & 0x007E007Eu) | one;
    } else {
      const uint64_t c0w = (uint64_t(hi[2 * i]) << 32) | a0, c1w = (uint64_t(hi[2 * i + 1]) << 32) | a1;
      const uint32_t c0 = uint32_t(c0w >> (BITS * k)) & M, c1 = uint32_t(c1w >> (BITS * k)) & M;
      if constexpr (BITS == 8) {
        f[i] = __builtin_amdgcn_perm(__float_as_uint(float(c1)), __float_as_uint(float(c0)), 0x07060302u);
      } else {
        f[i] = one | (c0 << (7 - BITS)) | (c1 << (23 - BITS));
      }
    }
  }
  return as_bf16x8(f);
}

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));

// bf16 pair (RN(a), RN(b)), a in the low half (the hardware conversion, round to nearest even)
__device__ __forceinline__ uint32_t pk_bf16(float a, float b) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t{a, b}), bf16x2_t));
}

// bf16 planes of v: hi = RN(v), lo = RN(v - hi)
__device__ __forceinline__ void split2(float v, uint32_t& hi, uint32_t& lo) {
  hi = f32_to_bf16_rne(v);
  lo = f32_to_bf16_rne(v - bf16_to_f32(hi));
}

template <int BITS, int NBLK, int TB, bool KIVI = false>
__global__ __launch_bounds__(kAThreads, 2) void att_mfma(AttendDev a, GaugeDev G) {
  static_assert(TB == 1 || TB == 16, "token tiles of 16");
  static_assert(!KIVI || (TB == 1 && NBLK == 2), "KIVI: 32-position key groups, 64-channel value blocks");
  constexpr bool RAW = TB > 1 || KIVI;         // raw bf16 positions after the quantised ones
  constexpr int JQ = 8 / NBLK;                 // query heads per workgroup (16 A rows)
  constexpr int NQL = 2 / NBLK;                // queries per D lane
  constexpr int NB = kD / NBLK;                // channels per block
  constexpr int RB = kD * BITS / 8;            // code bytes per row
  constexpr float kSK = BITS == 8 ? 1.0f : (BITS == 6 ? 128.0f : float(1 << BITS));  // code_frag scale
  constexpr float kSV = BITS == 8 ? 1.0f : float(1 << BITS);                           // vfrag scale
  constexpr float kSK2 = BITS == 8 ? 1.0f : float(1 << BITS);                          // KIVI key scale
  __shared__ __attribute__((aligned(16))) float qt[JQ][kD];
  __shared__ __attribute__((aligned(16))) float macc[JQ][kD];
  __shared__ float qsum[JQ][NBLK];
  __shared__ __attribute__((aligned(16))) float pbuf[4][JQ][32];
  __shared__ float abuf[4][JQ];
  __shared__ __attribute__((aligned(16))) uint32_t vsd[4][NBLK][32];
  __shared__ float offs[4][16][4];
  __shared__ float ml[4][2][JQ];
  __shared__ float mm[2][JQ];
  // raw positions (staged tile tokens, the KIVI window): scores then weights of a chunk of 16,
  // running maximum and sum per query, the chunk's rescaling factor, value sums
  constexpr int RJ = RAW ? JQ : 1;
  __shared__ float rs[RJ][16];
  __shared__ float rml[2][RJ];
  __shared__ float rfac[RJ];
  __shared__ __attribute__((aligned(16))) float accr[RJ][RAW ? kD : 1];
  // KIVI keys: the step's key group in a per-wave region, token-major (row t: the bf16 B values
  // of channels 2i, 2i + 1 in word i; rows of 68 words, so the 16-byte reads of 16 tokens and the
  // word writes of 64 lanes both spread over all banks), and the side word of each channel
  constexpr int KROW = 68;
  __shared__ __attribute__((aligned(16))) uint32_t ktk[KIVI ? 4 : 1][KIVI ? 32 * KROW : 1];
  __shared__ __attribute__((aligned(16))) uint32_t kgs[KIVI ? 4 : 1][KIVI ? kD : 1];

  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int n = lane & 15, gq = lane >> 4;
  const int H = a.kc.H, B = a.q.B;
  const int sp = blockIdx.x;
  int sv = blockIdx.y;
  const int qc = sv % a.nqc;
  sv /= a.nqc;
  const int h = sv % H, b = (sv / H) % B, lv = sv / (H * B);
  const int l = lv + a.l0;
  const int j0 = qc * JQ, nj = min(JQ, a.grp - j0);
  const int hq0 = h * a.grp + j0;

  if (threadIdx.x == 0 && a.lens && sp == 0 && qc == 0 && h == 0 && lv == 0) {
    const int nn = a.lens[b];
    if ((nn < 0 || nn > a.cap) && a.err) atomicOr(a.err, CG_FLAG_POS_RANGE);
  }
  int held = a.lens ? a.lens[b] : a.len;
  if (held < 0 || held > a.cap) held = 0;
  const int t_begin = sp * a.chunk, t_end = min(held, t_begin + a.chunk);
  // positions in whole tiles / key groups go through the matrix cores, the staged tile tokens
  // or the KIVI window after them are raw
  const int tq = KIVI ? (held < a.win ? 0 : (held - a.win) / 32 * 32) : (TB > 1 ? held / TB * TB : held);
  const int t_endq = min(t_end, tq);

  // 1. queries: macc <- q, qt <- scale G_K q, qsum <- the per-block sums of its two planes
  for (int idx = threadIdx.x; idx < JQ * kD; idx += kAThreads) {
    const int jj = idx / kD, ch = idx % kD;
    float v = 0.0f;
    if (jj < nj) {
      const size_t off = size_t(lv) * a.q.sl + size_t(b) * a.q.sb + size_t(hq0 + jj) * a.q.sh + ch;
      v = a.q.bf16 ? bf16_to_f32(((const uint16_t*)a.q.ptr)[off]) : ((const float*)a.q.ptr)[off];
    }
    macc[jj][ch] = v;
  }
  __syncthreads();
  {
    const int g = G.g;
    for (int idx = threadIdx.x; idx < JQ * kD; idx += kAThreads) {
      const int jj = idx / kD, i = idx % kD;
      const int r = i / g, ii = i - r * g;
      const float* Gr = G.f32 + gauge_block(l, 0, h, r, G.H, G.R) * g * g + size_t(ii) * g;
      float z = 0.0f;
      for (int j = 0; j < g; ++j) z = fmaf(Gr[j], macc[jj][r * g + j], z);
      qt[jj][i] = a.scale * z;
    }
  }
  __syncthreads();
  if (threadIdx.x < JQ * NBLK) {
    const int jj = threadIdx.x / NBLK, k = threadIdx.x % NBLK;
    float acc = 0.0f;
    for (int ch = k * NB; ch < (k + 1) * NB; ++ch) {
      uint32_t hi, lo;
      split2(qt[jj][ch], hi, lo);
      acc += bf16_to_f32(hi) + bf16_to_f32(lo);
    }
    qsum[jj][k] = acc;
  }
  __syncthreads();

  // 2. score A fragments: row m = n -> (query, block, plane), region 32 gq
  bf16x8_t AK[4];
  if constexpr (!KIVI) {
    const int j = n / (2 * NBLK), blk = (n / 2) % NBLK, plane = n & 1;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      u32x4_t f = {0u, 0u, 0u, 0u};
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int ch = 32 * gq + frag_chan<BITS>(u, e);
        uint32_t hi = 0u, lo = 0u;
        if (ch / NB == blk) split2(qt[j][ch], hi, lo);
        f[e >> 1] |= (plane ? lo : hi) << (16 * (e & 1));
      }
      AK[u] = as_bf16x8(f);
    }
  }
  // the D rows of this lane: 4 gq + i -> query jr[i], block br[i], plane i & 1
  float qrow[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int m = 4 * gq + i;
    qrow[i] = qsum[m / (2 * NBLK)][(m / 2) % NBLK];
  }
  // value A rows: row m = n -> (query jw, block bw, plane pw)
  const int jw = n / (2 * NBLK), bw = (n / 2) % NBLK, pw = n & 1;
  // KIVI score rows use the same (query, block, plane) mapping: row n holds qt of its query at the
  // 16 channels 64 bw + 32 v + 8 gq + i (K-steps 2 bw + v), zero at the other K-steps
  float qk[KIVI ? 16 : 1];
  if constexpr (KIVI) {
#pragma unroll
    for (int v = 0; v < 2; ++v)
#pragma unroll
      for (int i = 0; i < 8; ++i) qk[8 * v + i] = qt[jw][64 * bw + 32 * v + 8 * gq + i];
  }

  float mrun[NQL], lp[NQL];
#pragma unroll
  for (int qi = 0; qi < NQL; ++qi) {
    mrun[qi] = -INFINITY;
    lp[qi] = 0.0f;
  }
  f32x4_t accV[8];
#pragma unroll
  for (int nt = 0; nt < 8; ++nt) accV[nt] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
  float offl = 0.0f;

  uint32_t one = 0x3F803F80u,
           fmask = BITS == 2 ? 0x00600060u : (BITS == 3 ? 0x00700070u : (BITS == 6 ? 0x003F003Fu : 0x00780078u));
  asm volatile("" : "+v"(one), "+v"(fmask));

  // per-lane constant parts of the addresses (byte offsets from a slice's first row)
  const uint32_t koff = uint32_t(n) * RB + uint32_t(gq) * BITS * 4;    // key region of token n
  const uint32_t vcb = uint32_t(n) * BITS;                             // value chunk byte in the row
  const uint32_t voff = uint32_t(8 * gq) * RB + (vcb & ~3u);           // its first dword, token 8 gq
  const uint32_t vsh = (vcb & 3u) * 8;                                 // chunk bit offset in that dword

  // One 32-position step; FULL: all 32 positions lie before t_end (no clamping)
  auto step = [&](int t0, auto fullc) {
    constexpr bool FULL = decltype(fullc)::value;
    const int lim = t_endq - 1 - t0;  // last valid position offset in the step
    auto clampt = [&](int x) { return FULL ? x : min(x, lim); };
    // cache row of position t0 (a step never crosses a page)
    size_t sslc;
    int poff;
    if (!step_slice(a, l, b, h, t0, sslc, poff)) return;  // uniform over the wave
    const size_t srow = sslc * size_t(a.kc.T_cap) + (t0 - poff);
    const uint8_t* kb = a.kc.codes + srow * RB;
    const uint8_t* vb = a.vc.codes + srow * RB;
    // side words of the step's first position (tiles: of its tile; t0 is a multiple of 32)
    const size_t sidx = TB > 1 ? sslc * size_t(a.kc.T_cap / TB) + (t0 - poff) / TB : srow;
    const uint32_t* ksd = a.kc.side + sidx * NBLK;
    const uint32_t* vsdg = a.vc.side + sidx * NBLK;
    // loads: key regions of tokens t0 + 16 sb + n, value chunks of tokens t0 + 8 gq + e
    uint32_t rk[2][BITS];
    uint32_t swk[2][NBLK];
    uint2 kcv[KIVI ? BITS : 1], ksv;
    if constexpr (KIVI) {
      // the step's key group (t0 is a multiple of 32): codes and side words of channels 2 lane,
      // 2 lane + 1
      const size_t gi = sslc * size_t(a.kc.T_cap / 32) + size_t(t0 - poff) / 32;
      const uint2* src = reinterpret_cast<const uint2*>(a.kc.codes + (gi * kD + 2 * lane) * (4 * BITS));
#pragma unroll
      for (int i = 0; i < BITS; ++i) kcv[i] = src[i];
      ksv = *reinterpret_cast<const uint2*>(a.kc.side + gi * kD + 2 * lane);
    } else {
#pragma unroll
      for (int sb = 0; sb < 2; ++sb) {
        const uint32_t* src = reinterpret_cast<const uint32_t*>(
            kb + (FULL ? koff + 16u * sb * RB : uint32_t(clampt(16 * sb + n)) * RB + uint32_t(gq) * BITS * 4));
#pragma unroll
        for (int i = 0; i < BITS; ++i) rk[sb][i] = src[i];
        const uint32_t* sd = ksd + uint32_t(clampt(16 * sb + n) / TB) * NBLK;
#pragma unroll
        for (int k = 0; k < NBLK; ++k) swk[sb][k] = sd[k];
      }
    }
    uint32_t vw0[8], vw1[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const uint32_t* src = reinterpret_cast<const uint32_t*>(
          vb + (FULL ? voff + uint32_t(e) * RB : uint32_t(clampt(8 * gq + e)) * RB + (vcb & ~3u)));
      vw0[e] = src[0];
      // 4-bit chunks are one dword, 2-bit chunks half of one; the others may reach the next
      // dword, which lies inside the row whenever the chunk needs it (the last chunk of a
      // 3-bit row does not)
      if constexpr (BITS == 6 || BITS == 8) vw1[e] = src[1];
      else if constexpr (BITS == 3) vw1[e] = (n == 15) ? 0u : src[1];
      else vw1[e] = 0u;
    }
    if (lane < 32 * NBLK) {
      const int k = lane >> 5, t = lane & 31;
      vsd[w][k][t] = vsdg[size_t(clampt(t) / TB) * NBLK + k];
    }

    // scores of the two 16-token halves
    float s[2][NQL];
    if constexpr (KIVI) {
      // the group to the wave's LDS region: this lane's two channel streams (words 0 .. BITS - 1
      // of channel 2 lane, then those of channel 2 lane + 1) become, for every token t, the bf16
      // pair of B values of the two channels: 1 + q 2^-b (8 bits: q)
      constexpr uint32_t QM = (1u << BITS) - 1u;
      uint32_t sw2[2 * BITS];
#pragma unroll
      for (int i = 0; i < BITS; ++i) {
        sw2[2 * i] = kcv[i].x;
        sw2[2 * i + 1] = kcv[i].y;
      }
#pragma unroll
      for (int t = 0; t < 32; ++t) {
        const int bit = t * BITS, wd = bit >> 5, off = bit & 31;
        uint32_t qa, qb;
        if (off + BITS <= 32) {
          qa = (sw2[wd] >> off) & QM;
          qb = (sw2[BITS + wd] >> off) & QM;
        } else {
          qa = __builtin_amdgcn_alignbit(sw2[wd + 1], sw2[wd], off) & QM;
          qb = __builtin_amdgcn_alignbit(sw2[BITS + wd + 1], sw2[BITS + wd], off) & QM;
        }
        uint32_t pr;
        if constexpr (BITS == 8) pr = __builtin_amdgcn_perm(__float_as_uint(float(qb)), __float_as_uint(float(qa)), 0x07060302u);
        else pr = one | (qa << (7 - BITS)) | (qb << (23 - BITS));
        ktk[w][t * KROW + lane] = pr;
      }
      *reinterpret_cast<uint2*>(&kgs[w][2 * lane]) = ksv;
      __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
      __builtin_amdgcn_wave_barrier();
      // A: a = qt sc of the row's channels as two bf16 planes (the row keeps plane pw); the
      // codes enter as B = 1 + q 2^-b (8 bits: q), so with k = 2^b (8 bits: 1)
      //   s_t = sum_c qt_c (mn_c + q_tc sc_c) = k (sum_c a_c B_tc + part),
      //   part = sum_c qt_c mn_c / k - sum_c a_c   (8 bits: sum_c qt_c mn_c),
      // each row adding its own terms of part (the mn term on plane-0 rows, each plane's entries
      // of a on its own rows); part enters through one more product, its three bf16 planes
      // against a B of ones, which sums the four lane groups of each row
      u32x4_t fa[2];
      float part = 0.0f;
#pragma unroll
      for (int v = 0; v < 2; ++v) {
        const int c0 = 64 * bw + 32 * v + 8 * gq;
        const u32x4_t sa = *reinterpret_cast<const u32x4_t*>(&kgs[w][c0]);
        const u32x4_t sb4 = *reinterpret_cast<const u32x4_t*>(&kgs[w][c0 + 4]);
        const uint32_t se[8] = {sa[0], sa[1], sa[2], sa[3], sb4[0], sb4[1], sb4[2], sb4[3]};
#pragma unroll
        for (int e2 = 0; e2 < 4; ++e2) {
          const float q0 = qk[8 * v + 2 * e2], q1 = qk[8 * v + 2 * e2 + 1];
          const float x0 = q0 * f16_bits_to_f32(se[2 * e2] >> 16), x1 = q1 * f16_bits_to_f32(se[2 * e2 + 1] >> 16);
          const uint32_t hi = pk_bf16(x0, x1);
          const float h0 = __uint_as_float(hi << 16), h1 = __uint_as_float(hi & 0xffff0000u);
          const uint32_t lo = pk_bf16(x0 - h0, x1 - h1);
          fa[v][e2] = pw ? lo : hi;
          if (pw == 0) {
            part = fmaf(q0, f16_bits_to_f32(se[2 * e2] & 0xffffu) * (1.0f / kSK2), part);
            part = fmaf(q1, f16_bits_to_f32(se[2 * e2 + 1] & 0xffffu) * (1.0f / kSK2), part);
            if constexpr (BITS != 8) part -= h0 + h1;
          } else if constexpr (BITS != 8) {
            part -= __uint_as_float(lo << 16) + __uint_as_float(lo & 0xffff0000u);
          }
        }
      }
      const u32x4_t zero4 = {0u, 0u, 0u, 0u};
      bf16x8_t AKk[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) AKk[u] = as_bf16x8((u >> 1) == bw ? fa[u & 1] : zero4);
      uint32_t p0, p1, p2;
      split2(part, p0, p1);
      p2 = f32_to_bf16_rne(part - bf16_to_f32(p0) - bf16_to_f32(p1));
      const bf16x8_t AO = as_bf16x8(u32x4_t{p0 | (p1 << 16), p2, 0u, 0u});
      const bf16x8_t BONE = as_bf16x8(u32x4_t{one, one, one, one});
#pragma unroll
      for (int sb = 0; sb < 2; ++sb) {
        // token 16 sb + n: channels 32 u + 8 gq .. + 7 are words 16 u + 4 gq .. + 3 of its row
        const uint32_t* kr = &ktk[w][(16 * sb + n) * KROW + 4 * gq];
        f32x4_t d = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int u = 0; u < 4; ++u) d = mfma16(AKk[u], as_bf16x8(*reinterpret_cast<const u32x4_t*>(kr + 16 * u)), d);
        d = mfma16(AO, BONE, d);
        const bool valid = FULL || 16 * sb + n <= lim;
        s[sb][0] = valid ? kSK2 * ((d[0] + d[1]) + (d[2] + d[3])) : -INFINITY;
      }
    } else {
#pragma unroll
    for (int sb = 0; sb < 2; ++sb) {
      f32x4_t d = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
      for (int u = 0; u < 4; ++u) d = mfma16(AK[u], code_frag<BITS, BITS>(rk[sb], u, one, fmask), d);
      float gam[NBLK], bet[NBLK];
#pragma unroll
      for (int k = 0; k < NBLK; ++k) {
        const float mn = f16_bits_to_f32(swk[sb][k] & 0xffffu), sc = f16_bits_to_f32(swk[sb][k] >> 16);
        gam[k] = kSK * sc;
        bet[k] = BITS == 8 ? mn : mn - gam[k];
      }
      const bool valid = FULL || 16 * sb + n <= lim;
      if constexpr (NBLK == 2) {
        const float v = fmaf(gam[0], d[0] + d[1], bet[0] * qrow[0]) + fmaf(gam[1], d[2] + d[3], bet[1] * qrow[2]);
        s[sb][0] = valid ? v : -INFINITY;
      } else {
        s[sb][0] = valid ? fmaf(gam[0], d[0] + d[1], bet[0] * qrow[0]) : -INFINITY;
        s[sb][1] = valid ? fmaf(gam[0], d[2] + d[3], bet[0] * qrow[2]) : -INFINITY;
      }
    }
    }
    // online softmax (queries of the lane's D rows)
    float alpha[NQL];
#pragma unroll
    for (int qi = 0; qi < NQL; ++qi) {
      const int j = NBLK == 2 ? gq : 2 * gq + qi;
      const float mx = row16_max(fmaxf(s[0][qi], s[1][qi]));
      const float mnew = fmaxf(mrun[qi], mx);
      alpha[qi] = __expf(mrun[qi] - mnew);
      const float p0 = __expf(s[0][qi] - mnew), p1 = __expf(s[1][qi] - mnew);
      lp[qi] = fmaf(lp[qi], alpha[qi], p0 + p1);
      mrun[qi] = mnew;
      pbuf[w][j][n] = p0;
      pbuf[w][j][16 + n] = p1;
      if (n == 0) abuf[w][j] = alpha[qi];
    }
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    __builtin_amdgcn_wave_barrier();
    // rescale the value accumulators when a maximum moved
    bool moved = false;
#pragma unroll
    for (int qi = 0; qi < NQL; ++qi) moved |= alpha[qi] != 1.0f;
    if (__builtin_amdgcn_ballot_w64(moved)) {
#pragma unroll
      for (int nt = 0; nt < 8; ++nt) {
#pragma unroll
        for (int i = 0; i < 4; ++i) accV[nt][i] *= alpha[NBLK == 2 ? 0 : (i >> 1)];
      }
    }
    // value A fragment: w = kSV p sc of tokens 8 gq .. 8 gq + 7 for row (jw, bw, pw), split
    // into bf16 planes by the hardware conversion (round to nearest even)
    bf16x8_t AV;
    {
      const float4 pa = *reinterpret_cast<const float4*>(&pbuf[w][jw][8 * gq]);
      const float4 pb = *reinterpret_cast<const float4*>(&pbuf[w][jw][8 * gq + 4]);
      const uint4 sa = *reinterpret_cast<const uint4*>(&vsd[w][bw][8 * gq]);
      const uint4 sb4 = *reinterpret_cast<const uint4*>(&vsd[w][bw][8 * gq + 4]);
      const float pe[8] = {pa.x, pa.y, pa.z, pa.w, pb.x, pb.y, pb.z, pb.w};
      const uint32_t se[8] = {sa.x, sa.y, sa.z, sa.w, sb4.x, sb4.y, sb4.z, sb4.w};
      float o = offl * abuf[w][jw];
      u32x4_t f;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float x0 = kSV * f16_bits_to_f32(se[2 * i] >> 16) * pe[2 * i];
        const float x1 = kSV * f16_bits_to_f32(se[2 * i + 1] >> 16) * pe[2 * i + 1];
        const uint32_t hi = pk_bf16(x0, x1);
        const float h0 = __uint_as_float(hi << 16), h1 = __uint_as_float(hi & 0xffff0000u);
        const uint32_t lo = pk_bf16(x0 - h0, x1 - h1);
        f[i] = pw ? lo : hi;
        const float mn0 = f16_bits_to_f32(se[2 * i] & 0xffffu), mn1 = f16_bits_to_f32(se[2 * i + 1] & 0xffffu);
        if (pw == 0) {
          o = BITS == 8 ? fmaf(pe[2 * i], mn0, o) : fmaf(pe[2 * i], mn0, o - h0);
          o = BITS == 8 ? fmaf(pe[2 * i + 1], mn1, o) : fmaf(pe[2 * i + 1], mn1, o - h1);
        } else if (BITS != 8) {
          o -= __uint_as_float(lo << 16) + __uint_as_float(lo & 0xffff0000u);
        }
      }
      offl = o;
      AV = as_bf16x8(f);
    }
    uint32_t vlo[8], vhi[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) vchunk<BITS>(vw0[e], vw1[e], vsh, vlo[e], vhi[e]);
#pragma unroll
    for (int nt = 0; nt < 8; ++nt) accV[nt] = mfma16(AV, vfrag<BITS>(vlo, vhi, nt, one), accV[nt]);
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    __builtin_amdgcn_wave_barrier();
  };
  int t0 = t_begin + 32 * w;
  for (; t0 + 32 <= t_endq; t0 += 128) step(t0, std::true_type{});
  if (t0 < t_endq) step(t0, std::false_type{});

  // raw positions [max(tq, t_begin), t_end) of this split (staged tile tokens, at most 15; the
  // KIVI window, at most win + 31), in chunks of 16: scores with the raw query (macc still holds
  // q), a running maximum and sum per query, raw value sums rescaled as the maximum moves
  if constexpr (RAW) {
    const int ringsz = KIVI ? a.win + 32 : TB;
    const int r0 = max(tq, t_begin), nr = max(0, t_end - r0);
    const size_t slc = (size_t(l) * a.kc.B + b) * a.kc.H + h;
    if (threadIdx.x < RJ) {
      rml[0][threadIdx.x] = -INFINITY;
      rml[1][threadIdx.x] = 0.0f;
    }
    for (int idx = threadIdx.x; idx < RJ * kD; idx += kAThreads) (&accr[0][0])[idx] = 0.0f;
    for (int c0 = 0; c0 < nr; c0 += 16) {
      const int nc = min(16, nr - c0);
      __syncthreads();
      if (threadIdx.x < JQ * 16) {
        const int jj = threadIdx.x / 16, r = threadIdx.x % 16;
        float sc = -INFINITY;
        if (jj < nj && r < nc) {
          const uint16_t* kr = a.kc.ring + (slc * ringsz + (r0 + c0 + r) % ringsz) * kD;
          float acc = 0.0f;
          for (int ch = 0; ch < kD; ++ch) acc = fmaf(macc[jj][ch], bf16_to_f32(kr[ch]), acc);
          sc = a.scale * acc;
        }
        rs[jj][r] = sc;
      }
      __syncthreads();
      if (threadIdx.x < JQ) {
        const int jj = threadIdx.x;
        const float mo = rml[0][jj];
        float m = mo;
        for (int r = 0; r < nc; ++r) m = fmaxf(m, rs[jj][r]);
        const float f = mo == -INFINITY ? 0.0f : __expf(mo - m);
        float sum = rml[1][jj] * f;
        for (int r = 0; r < nc; ++r) {
          const float pr = m == -INFINITY ? 0.0f : __expf(rs[jj][r] - m);
          rs[jj][r] = pr;
          sum += pr;
        }
        rml[0][jj] = m;
        rml[1][jj] = sum;
        rfac[jj] = f;
      }
      __syncthreads();
      for (int idx = threadIdx.x; idx < JQ * kD; idx += kAThreads) {
        const int jj = idx / kD, ch = idx % kD;
        float acc = accr[jj][ch] * rfac[jj];
        for (int r = 0; r < nc; ++r)
          acc = fmaf(rs[jj][r], bf16_to_f32(a.vc.ring[(slc * ringsz + (r0 + c0 + r) % ringsz) * kD + ch]), acc);
        accr[jj][ch] = acc;
      }
    }
  }

  // 3. per-wave results: maximum and sum per query, gauge-space value sums
  float lsum[NQL];
#pragma unroll
  for (int qi = 0; qi < NQL; ++qi) lsum[qi] = row16_sum(lp[qi]);
  offs[w][n][gq] = offl;
  if (n == 0) {
#pragma unroll
    for (int qi = 0; qi < NQL; ++qi) {
      const int j = NBLK == 2 ? gq : 2 * gq + qi;
      ml[w][0][j] = mrun[qi];
      ml[w][1][j] = lsum[qi];
    }
  }
  for (int idx = threadIdx.x; idx < JQ * kD; idx += kAThreads) (&macc[0][0])[idx] = 0.0f;
  __syncthreads();
  // merge the four waves: factors exp(m_w - M) per query
  float fq[NQL], offq[NQL][NBLK];
#pragma unroll
  for (int qi = 0; qi < NQL; ++qi) {
    const int j = NBLK == 2 ? gq : 2 * gq + qi;
    float M = RAW ? rml[0][j < RJ ? j : 0] : -INFINITY;
    for (int v = 0; v < 4; ++v) M = fmaxf(M, ml[v][0][j]);
    fq[qi] = mrun[qi] == -INFINITY ? 0.0f : __expf(mrun[qi] - M);
#pragma unroll
    for (int k = 0; k < NBLK; ++k) {
      float o = 0.0f;
      const int r0 = j * 2 * NBLK + 2 * k;  // rows (j, k, hi) and (j, k, lo)
      for (int g4 = 0; g4 < 4; ++g4) o += offs[w][r0][g4] + offs[w][r0 + 1][g4];
      offq[qi][k] = o;
    }
  }
  for (int v = 0; v < 4; ++v) {
    if (w == v) {
#pragma unroll
      for (int nt = 0; nt < 8; ++nt) {
        const int ch = 8 * n + nt;
        if constexpr (NBLK == 2) {
          const bool hiblk = ch >= NB;
          const float val = (hiblk ? accV[nt][2] + accV[nt][3] : accV[nt][0] + accV[nt][1]) +
                            (hiblk ? offq[0][1] : offq[0][0]);
          macc[gq][ch] += fq[0] * val;
        } else {
          macc[2 * gq][ch] += fq[0] * (accV[nt][0] + accV[nt][1] + offq[0][0]);
          macc[2 * gq + 1][ch] += fq[1] * (accV[nt][2] + accV[nt][3] + offq[1][0]);
        }
      }
    }
    __syncthreads();
  }
  if (threadIdx.x < JQ) {
    const int jj = threadIdx.x;
    float M = RAW ? rml[0][jj < RJ ? jj : 0] : -INFINITY, L = 0.0f;
    for (int v = 0; v < 4; ++v) M = fmaxf(M, ml[v][0][jj]);
    for (int v = 0; v < 4; ++v) {
      const float mv = ml[v][0][jj];
      if (mv != -INFINITY) L += ml[v][1][jj] * __expf(mv - M);
    }
    if constexpr (RAW) {
      const float mr = rml[0][jj < RJ ? jj : 0];
      if (mr != -INFINITY) L += rml[1][jj < RJ ? jj : 0] * __expf(mr - M);
    }
    mm[0][jj] = M;
    mm[1][jj] = L;
  }
  __syncthreads();
  if constexpr (RAW) {  // raw value sums to the common maximum
    for (int idx = threadIdx.x; idx < JQ * kD; idx += kAThreads) {
      const int jj = idx / kD, ch = idx % kD;
      const float mr = rml[0][jj];
      accr[jj][ch] = mr == -INFINITY ? 0.0f : accr[jj][ch] * __expf(mr - mm[0][jj]);
    }
    __syncthreads();
  }
  if (a.nsplit == 1) {
    finalize_rows(a, G, &macc[0][0], RAW ? &accr[0][0] : nullptr, mm[1], nj, lv, b, h, hq0);
    return;
  }
  const size_t pstride = size_t(2 + 2 * kD);
  for (int jj = 0; jj < nj; ++jj) {
    float* P = a.part + ((((size_t(lv) * B + b) * a.Hq + hq0 + jj) * a.nsplit) + sp) * pstride;
    for (int idx = threadIdx.x; idx < 2 + 2 * kD; idx += kAThreads) {
      float v;
      if (idx == 0) v = mm[0][jj];
      else if (idx == 1) v = mm[1][jj];
      else if (idx < 2 + kD) v = macc[jj][idx - 2];
      else v = RAW ? accr[jj < RJ ? jj : 0][(idx - 2 - kD) % (RAW ? kD : 1)] : 0.0f;
      P[idx] = v;
    }
  }
}

template <int BITS>
const void* att_mfma_fn(int nblk, int bt, bool kivi) {
  if (kivi) return (const void*)att_mfma<BITS, 2, 1, true>;
  if (bt > 1) return nblk == 2 ? (const void*)att_mfma<BITS, 2, 16> : (const void*)att_mfma<BITS, 1, 16>;
  return nblk == 2 ? (const void*)att_mfma<BITS, 2, 1> : (const void*)att_mfma<BITS, 1, 1>;
}

const void* att_mfma_kernel(int bits, int nblk, int bt, bool kivi) {
  switch (bits) {
    case 2: return att_mfma_fn<2>(nblk, bt, kivi);
    case 3: return att_mfma_fn<3>(nblk, bt, kivi);
    case 4: return att_mfma_fn<4>(nblk, bt, kivi);
    case 6: return att_mfma_fn<6>(nblk, bt, kivi);
    default: return att_mfma_fn<8>(nblk, bt, kivi);
  }
}

hipError_t set_smem(const void* fn, size_t bytes) {
  if (bytes <= 65536) return hipSuccess;
  return hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
}

}  // namespace

AttendPlan attend_plan(int nl, int B, int H, int Hq, int d, int span) {
  AttendPlan p;
  const int grp = Hq / H;
  p.nqc = (grp + kJQ - 1) / kJQ;
  const int64_t rows = int64_t(nl) * B * H * p.nqc;  // workgroups per split
  // enough splits for about 2048 workgroups, each split at least 256 positions
  const int64_t want = (2048 + rows - 1) / rows;
  const int64_t most = (int64_t(span) + 255) / 256;
  int ns = int(std::max<int64_t>(1, std::min(want, most)));
  int chunk = (span + ns - 1) / ns;
  chunk = std::max(kATile, (chunk + kATile - 1) / kATile * kATile);
  ns = std::max(1, (span + chunk - 1) / chunk);
  p.nsplit = ns;
  p.chunk = chunk;
  p.ws_bytes = ns > 1 ? size_t(nl) * B * Hq * ns * (2 + 2 * size_t(d)) * sizeof(float) : 0;
  return p;
}

bool attend_mfma_supported(const AttendDev& a, const CodecDev& c) {
  const bool bits = c.bits == 2 || c.bits == 3 || c.bits == 4 || c.bits == 6 || c.bits == 8;
  // KIVI: 32-position key groups, 64-channel value blocks, contiguous caches
  if (c.backend == CG_BACKEND_KIVI) return a.q.d == kD && c.kg == 32 && c.kvc == 64 && !a.pt.pages && bits;
  // tiles of 16 tokens on contiguous caches (paged caches take per-token blocks only)
  return c.backend == CG_BACKEND_BLOCK_UNIFORM && (c.bt == 1 || (c.bt == 16 && !a.pt.pages)) && a.q.d == kD &&
         (c.n == 64 || c.n == 128) && bits;
}

hipError_t launch_attend(const AttendDev& a, const GaugeDev& G, const CodecDev& c, bool force_generic,
                         hipStream_t st) {
  const int d = a.q.d;
  const int nrow = a.q.L * a.q.B * a.kc.H * a.nqc;
  if (nrow == 0) return hipSuccess;
  hipError_t e;
  if (!force_generic && attend_mfma_supported(a, c)) {
    // the matrix-core kernel takes 8 / NBLK query heads per workgroup (NBLK value blocks per row)
    const bool kivi = c.backend == CG_BACKEND_KIVI;
    const int nblk = kD / (kivi ? c.kvc : c.n), jq = 8 / nblk;
    AttendDev af = a;
    af.nqc = (a.grp + jq - 1) / jq;
    af.win = kivi ? c.win : 0;
    const int nrow_f = a.q.L * a.q.B * a.kc.H * af.nqc;
    GaugeDev g2 = G;
    void* args[] = {&af, &g2};
    e = hipLaunchKernel(att_mfma_kernel(c.bits, nblk, c.bt, kivi), dim3(a.nsplit, nrow_f), dim3(kAThreads), args, 0,
                        st);
    if (e != hipSuccess) return e;
  } else {
    const size_t smem = (size_t(2) * kJQ * d + size_t(kGTile) * (d + 4) + kJQ * kGTile + 3 * kJQ) * sizeof(float);
    e = set_smem((const void*)att_generic, smem);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(att_generic, dim3(a.nsplit, nrow), dim3(kAThreads), smem, st, a, G, c);
  }
  e = hipGetLastError();
  if (e != hipSuccess || a.nsplit == 1) return e;
  const size_t smem2 = (size_t(2) * kJQ * d + 2 * kJQ) * sizeof(float);
  hipLaunchKernelGGL(att_combine, dim3(nrow), dim3(kAThreads), smem2, st, a, G);
  return hipGetLastError();
}

// ------------------------------------------------------------------------------------------
// scratch of kv_attend_noalloc: the split rows' partial results in a file-scope device array
// (one per device the library runs on, held until the process ends).  Host code never passes
// `scratch` itself to a kernel: its device address comes from hipGetSymbolAddress, once per
// device, with that device current.
// ------------------------------------------------------------------------------------------
constexpr size_t kAttendScratchBytes = CG_ATTEND_NOALLOC_SCRATCH_BYTES;
constexpr int kMaxDevices = 64;
static __device__ __align__(256) unsigned char scratch[kAttendScratchBytes];

size_t attend_scratch_bytes() { return kAttendScratchBytes; }

hipError_t attend_scratch(void** ptr) {
  static std::mutex mu;
  static void* addr[kMaxDevices] = {};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    addr[dev] = p;
  }
  *ptr = addr[dev];
  return hipSuccess;
}

}  // namespace cg
