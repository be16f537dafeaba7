// Decode-phase attention over the compressed caches, with the inverse gauge folded into the
// attention consumer instead of materialising Xhat (the deployment route the paper points to
// when it notes that recovery can be folded into downstream operations, section 3 and the
// discussion of its timings).
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

#include "cg_internal.h"
#include "cg_device.h"

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
  if (r.held < 0 || r.held > a.kc.T_cap) r.held = 0;
  if (c.backend == CG_BACKEND_KIVI) r.tq = r.held < c.win ? 0 : ((r.held - c.win) / c.kg) * c.kg;
  else if (c.backend == CG_BACKEND_BLOCK_UNIFORM && c.bt > 1) r.tq = (r.held / c.bt) * c.bt;
  else r.tq = r.held;
  return r;
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
    x += accr[jj * d + i];
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
// Wave w takes the 64-position steps w, w + 4, ... of the split.  Scores: lane = position, a
// binary32 FMA chain over the channels of the dequantised key (gauge-space query for quantised
// positions, the raw query for raw ones).  Values: lane = channel, the running accumulators of
// every query head are rescaled by exp(m_old - m_new) and take p_t zhat^V_t (quantised) or
// p_t x^V_t (raw) for every position of the step.
__global__ __launch_bounds__(kAThreads) void att_generic(AttendDev a, GaugeDev G, CodecDev c) {
  extern __shared__ float sm[];
  const int d = a.q.d, H = a.kc.H, B = a.q.B;
  float* qg = sm;                      // [kJQ][d] scale * G_K q
  float* qr = qg + kJQ * d;            // [kJQ][d] scale * q
  float* pw = qr + kJQ * d;            // [4][kJQ][64] probabilities of a step
  float* macc = pw + 4 * kJQ * kATile;  // [kJQ][d] merged gauge-space accumulator
  float* maccr = macc + kJQ * d;       // [kJQ][d] merged raw accumulator
  float* ml = maccr + kJQ * d;         // [4][2][kJQ] per-wave max and sum, then [2][kJQ] merged

  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int sp = blockIdx.x;
  int sv = blockIdx.y;
  const int qc = sv % a.nqc;
  sv /= a.nqc;
  const int h = sv % H, b = (sv / H) % B, lv = sv / (H * B);
  const int l = lv + a.l0;
  const int j0 = qc * kJQ, nj = min(kJQ, a.grp - j0);
  const int hq0 = h * a.grp + j0;  // first query head of this workgroup
  const size_t slc = (size_t(l) * a.kc.B + b) * H + h;

  if (threadIdx.x == 0 && a.lens && sp == 0 && qc == 0 && h == 0 && lv == 0) {
    const int n = a.lens[b];
    if ((n < 0 || n > a.kc.T_cap) && a.err) atomicOr(a.err, CG_FLAG_POS_RANGE);
  }
  const RowSpan rs = row_span(a, c, b);
  const int t_begin = sp * a.chunk, t_end = min(rs.held, t_begin + a.chunk);

  // 1. queries: raw (scaled) and gauged (z_i = sum_j G_K[i][j] q_j, scaled)
  for (int idx = threadIdx.x; idx < kJQ * d; idx += kAThreads) {
    const int jj = idx / d, ch = idx - jj * d;
    float v = 0.0f;
    if (jj < nj) {
      const size_t off = size_t(lv) * a.q.sl + size_t(b) * a.q.sb + size_t(hq0 + jj) * a.q.sh + ch;
      v = a.q.bf16 ? bf16_to_f32(((const uint16_t*)a.q.ptr)[off]) : ((const float*)a.q.ptr)[off];
    }
    qr[idx] = v;
  }
  __syncthreads();
  {
    const int g = G.g;
    for (int idx = threadIdx.x; idx < kJQ * d; idx += kAThreads) {
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
  for (int idx = threadIdx.x; idx < kJQ * d; idx += kAThreads) qr[idx] *= a.scale;
  __syncthreads();

  // 2. the wave's steps
  constexpr int kCh = 4;  // channels per lane (d <= 256)
  float m[kJQ], ls[kJQ], acc[kJQ][kCh], accr[kJQ][kCh];
#pragma unroll
  for (int jj = 0; jj < kJQ; ++jj) {
    m[jj] = -INFINITY;
    ls[jj] = 0.0f;
#pragma unroll
    for (int k = 0; k < kCh; ++k) acc[jj][k] = accr[jj][k] = 0.0f;
  }
  float* pwv = pw + w * kJQ * kATile;
  for (int t0 = t_begin + kATile * w; t0 < t_end; t0 += 4 * kATile) {
    const int p = t0 + lane;
    const bool valid = p < t_end;
    float s[kJQ];
#pragma unroll
    for (int jj = 0; jj < kJQ; ++jj) s[jj] = 0.0f;
    if (valid) {
      const bool raw = p >= rs.tq;
      const float* qs = raw ? qr : qg;
      for (int ch = 0; ch < d; ++ch) {
        const float z = raw ? raw_at(a.kc, c, slc, p, ch, d) : zhat_at(a.kc, c, 0, slc, p, ch, d);
#pragma unroll
        for (int jj = 0; jj < kJQ; ++jj) s[jj] = fmaf(qs[jj * d + ch], z, s[jj]);
      }
    }
    float alpha[kJQ];
#pragma unroll
    for (int jj = 0; jj < kJQ; ++jj) {
      const float mx = wave_max(valid ? s[jj] : -INFINITY);
      const float mnew = fmaxf(m[jj], mx);
      alpha[jj] = __expf(m[jj] - mnew);  // exp(-inf) = 0 on the first step
      const float pv = valid ? __expf(s[jj] - mnew) : 0.0f;
      ls[jj] = ls[jj] * alpha[jj] + wave_sum(pv);
      m[jj] = mnew;
      pwv[jj * kATile + lane] = pv;
    }
    // the step's probabilities are read across lanes: order the LDS writes before the reads
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    __builtin_amdgcn_wave_barrier();
#pragma unroll
    for (int k = 0; k < kCh; ++k) {
#pragma unroll
      for (int jj = 0; jj < kJQ; ++jj) {
        acc[jj][k] *= alpha[jj];
        accr[jj][k] *= alpha[jj];
      }
    }
    const int nt = min(kATile, t_end - t0);
    for (int tt = 0; tt < nt; ++tt) {
      const int pp = t0 + tt;
      const bool raw = pp >= rs.tq;
#pragma unroll
      for (int k = 0; k < kCh; ++k) {
        const int ch = lane + 64 * k;
        if (ch < d) {
          const float z = raw ? raw_at(a.vc, c, slc, pp, ch, d) : zhat_at(a.vc, c, 1, slc, pp, ch, d);
#pragma unroll
          for (int jj = 0; jj < kJQ; ++jj) {
            const float pv = pwv[jj * kATile + tt];
            if (raw) accr[jj][k] = fmaf(pv, z, accr[jj][k]);
            else acc[jj][k] = fmaf(pv, z, acc[jj][k]);
          }
        }
      }
    }
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    __builtin_amdgcn_wave_barrier();
  }

  // 3. merge the four waves: M = max m_w, each wave's terms scaled by exp(m_w - M)
  if (lane == 0) {
#pragma unroll
    for (int jj = 0; jj < kJQ; ++jj) {
      ml[(w * 2 + 0) * kJQ + jj] = m[jj];
      ml[(w * 2 + 1) * kJQ + jj] = ls[jj];
    }
  }
  for (int idx = threadIdx.x; idx < 2 * kJQ * d; idx += kAThreads) macc[idx] = 0.0f;
  __syncthreads();
  float f[kJQ];
#pragma unroll
  for (int jj = 0; jj < kJQ; ++jj) {
    float M = -INFINITY;
    for (int v = 0; v < 4; ++v) M = fmaxf(M, ml[(v * 2) * kJQ + jj]);
    f[jj] = m[jj] == -INFINITY ? 0.0f : __expf(m[jj] - M);
  }
  for (int v = 0; v < 4; ++v) {
    if (w == v) {
#pragma unroll
      for (int k = 0; k < kCh; ++k) {
        const int ch = lane + 64 * k;
        if (ch < d) {
#pragma unroll
          for (int jj = 0; jj < kJQ; ++jj) {
            macc[jj * d + ch] += f[jj] * acc[jj][k];
            maccr[jj * d + ch] += f[jj] * accr[jj][k];
          }
        }
      }
    }
    __syncthreads();
  }
  float* mm = ml + 8 * kJQ;  // merged [2][kJQ]
  if (threadIdx.x < kJQ) {
    const int jj = threadIdx.x;
    float M = -INFINITY, L = 0.0f;
    for (int v = 0; v < 4; ++v) M = fmaxf(M, ml[(v * 2) * kJQ + jj]);
    for (int v = 0; v < 4; ++v) {
      const float mv = ml[(v * 2) * kJQ + jj];
      if (mv != -INFINITY) L += ml[(v * 2 + 1) * kJQ + jj] * __expf(mv - M);
    }
    mm[jj] = M;
    mm[kJQ + jj] = L;
  }
  __syncthreads();
  if (a.nsplit == 1) {
    finalize_rows(a, G, macc, maccr, mm + kJQ, nj, lv, b, h, hq0);
    return;
  }
  // partial results of this split
  const size_t pstride = size_t(2 + 2 * d);
  for (int jj = 0; jj < nj; ++jj) {
    float* P = a.part + ((((size_t(lv) * B + b) * a.Hq + hq0 + jj) * a.nsplit) + sp) * pstride;
    for (int idx = threadIdx.x; idx < 2 + 2 * d; idx += kAThreads) {
      float v;
      if (idx == 0) v = mm[jj];
      else if (idx == 1) v = mm[kJQ + jj];
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

hipError_t launch_attend(const AttendDev& a, const GaugeDev& G, const CodecDev& c, bool force_generic,
                         hipStream_t st) {
  (void)force_generic;
  const int d = a.q.d;
  const int nrow = a.q.L * a.q.B * a.kc.H * a.nqc;
  if (nrow == 0) return hipSuccess;
  const size_t smem = (size_t(4) * kJQ * d + 4 * kJQ * kATile + 10 * kJQ) * sizeof(float);
  hipError_t e = set_smem((const void*)att_generic, smem);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(att_generic, dim3(a.nsplit, nrow), dim3(kAThreads), smem, st, a, G, c);
  e = hipGetLastError();
  if (e != hipSuccess || a.nsplit == 1) return e;
  const size_t smem2 = (size_t(2) * kJQ * d + 2 * kJQ) * sizeof(float);
  hipLaunchKernelGGL(att_combine, dim3(nrow), dim3(kAThreads), smem2, st, a, G);
  return hipGetLastError();
}

}  // namespace cg
