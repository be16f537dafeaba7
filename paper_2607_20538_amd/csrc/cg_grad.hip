// Gradient of the gauge training objective with respect to the gauge generators (sections 4.1
// and 4.2): G = exp(S), S = A - A^T, per (layer, cache type, head, group), and per layer
// L_train = lambda_f L_freq + lambda_r L_rate of X' = G X cut into Tb-token blocks, each Tb x d
// block through the orthonormal 2-D DCT, U = C_Tb Z C_d^T.
//
// With M = C_d G (G block-diagonal over the head's groups) a block is U = C_Tb W, W = X M^T.
//   dL/dU = lambda_f 2 U (rho - L_freq) / D + lambda_r sign(U) / (N (tau + |U|))
//           (D = sum E + eps, N the layer's coefficient count, L_freq and sum E from the
//           forward statistics of the same launch);
//   dL/dW = C_Tb^T dL/dU;   dL/dM = sum over blocks of (dL/dW)^T X;   dL/dG = C_d^T dL/dM,
//           restricted to the gauge's diagonal blocks;
//   dL/dS = L(S^T, dL/dG), the adjoint of the Frechet derivative of exp at S, the top-right block
//           of exp([[S^T, dL/dG], [0, S^T]]);   dL/dA = dL/dS - (dL/dS)^T.
//
// Kernels: grad_prep forms M in binary32 per (layer, head) (binary64 sums); grad_data runs the
// blocks of a range of tokens of one (layer, batch row, head) on the VALU through LDS: X and M
// in binary32, W, U, dL/dU and dL/dW in binary64 (the binary32 products accumulate exactly),
// and accumulates its part of dL/dM in binary64 registers (a (d/16) x (d/16) tile per thread),
// written as one partial per workgroup; grad_data_mfma does the same for d = 128 with 16-token
// blocks on the binary64 matrix cores; grad_reduce sums the partials in a fixed order
// (deterministic); grad_frechet forms dL/dG and the Frechet adjoint per gauge block in binary64
// (power series of the scaled block matrix by the Paterson-Stockmeyer scheme, then squaring),
// and grad_frechet16 does the same for groups of at most 16 channels in one wave, in LDS.
// Binary64 through the data pass matters: dL/dA is the antisymmetric part of dL/dS, which for
// smooth objectives is much smaller than the terms that cancel in it (about 40x on random
// Llama-shaped data), so binary32 sums over a block's d channels would reach the result.
#include <algorithm>
#include <type_traits>

#include "cg_internal.h"
#include "cg_device.h"

namespace cg {

namespace {

constexpr int kGradThreads = 256;
constexpr int kFrechetTerms = 16;  // series terms of exp(W / 2^s) with |W / 2^s|_1 <= 1/2
// 1 / k!, by successive binary64 divisions (evaluated by the compiler)
constexpr double inv_fact(int k) {
  double r = 1.0;
  for (int i = 2; i <= k; ++i) r /= i;
  return r;
}

// cos(pi k / (2 d)) for k < 4 d, by the workgroup into LDS: the orthonormal DCT-II entry
// C_d[v][c] = sqrt((v ? 2 : 1) / d) cos(pi (2 c + 1) v / (2 d)) is that table at ((2 c + 1) v) mod 4 d
// (the argument is a multiple of 1 / (2 d), exact in binary64, and the cosine has period 2 pi).
// Along a row (v fixed) the index advances by 2 v, along a column (c fixed) by 2 c + 1, both
// below 2 d, so loops step it with one conditional wrap instead of a division.
constexpr int kMaxD = 128;
__device__ void dct_table(double* tab, int d) {
  for (int k = int(threadIdx.x); k < 4 * d; k += int(blockDim.x)) tab[k] = cospi(double(k) / (2.0 * d));
  __syncthreads();
}
__device__ __forceinline__ int dct_step(int k, int step, int d) {
  k += step;
  return k >= 4 * d ? k - 4 * d : k;
}

// M = C_d G_{l,s,h} per (l, h), binary64 sums rounded to binary32: [L][H][d][d].  Thread gi of a
// head computes column c = gi % d of the rows v = gi / d + (d / 8) q, q < 8, so each entry of G
// it loads serves eight sums (each over a in order).
constexpr int kPrepRows = 8;
__global__ __launch_bounds__(256) void grad_prep(int s, GaugeDev G, int H, int d, float* M) {
  __shared__ double tab[4 * kMaxD];
  dct_table(tab, d);
  const int lh = blockIdx.y, l = lh / H, h = lh - l * H;
  const int g = G.g, vs = d / kPrepRows;
  const double n0 = sqrt(1.0 / d), n1 = sqrt(2.0 / d);
  const int gi = blockIdx.x * blockDim.x + threadIdx.x;
  if (gi >= d * vs) return;
  const int c = gi % d, vb = gi / d, r = c / g, j = c - r * g;
  const float* Gc = G.f32 + (((size_t(l) * 2 + s) * G.H + h) * G.R + r) * g * g + j;
  double acc[kPrepRows], nv[kPrepRows];
  int k[kPrepRows];
#pragma unroll
  for (int q = 0; q < kPrepRows; ++q) {
    const int v = vb + vs * q;
    nv[q] = v == 0 ? n0 : n1;
    k[q] = ((2 * r * g + 1) * v) % (4 * d);  // entry (v, r g + a) for a = 0
    acc[q] = 0.0;
  }
  for (int a = 0; a < g; ++a) {
    const double gv = double(Gc[size_t(a) * g]);
#pragma unroll
    for (int q = 0; q < kPrepRows; ++q) {
      acc[q] = fma(nv[q] * tab[k[q]], gv, acc[q]);
      k[q] = dct_step(k[q], 2 * (vb + vs * q), d);
    }
  }
#pragma unroll
  for (int q = 0; q < kPrepRows; ++q) M[size_t(lh) * d * d + size_t(vb + vs * q) * d + c] = float(acc[q]);
}

struct GradArgs {
  ViewDev X;
  const float* M;        // [L][H][d][d]
  const double* stats;   // [L][4] from the forward statistics
  double* part;          // [L][H][B * chunks][d][d] partial dL/dM
  int Tb, nblk, chunks, blocks_per_wg;
  float inv_tau, tau, lam_f, lam_r;
  double inv_count;      // 1 / (coefficients per layer)
};

// One workgroup per (layer, batch row, head, chunk of blocks); TD = d / 16: thread (ty, tx) owns
// rows v in [TD ty, TD ty + TD) and columns k in [TD tx, TD tx + TD) of dL/dM.
template <int TD>
__global__ __launch_bounds__(kGradThreads) void grad_data(GradArgs a) {
  extern __shared__ double smd[];
  const int d = 16 * TD, dp = d + 1, Tb = a.Tb;
  double* ws = smd;                                  // W, then dL/dW [Tb][dp]
  double* us = ws + Tb * dp;                         // U, then dL/dU [Tb][dp]
  float* ms = reinterpret_cast<float*>(us + Tb * dp);  // M rows [d][dp]
  float* xs = ms + d * dp;                           // block of X [Tb][dp]
  float* ct = xs + Tb * dp;                          // C_Tb [Tb][Tb]
  const ViewDev& X = a.X;
  const int wg = blockIdx.x, chunk = wg % a.chunks, sl = wg / a.chunks;
  const int h = sl % X.H, b = (sl / X.H) % X.B, l = sl / (X.H * X.B);
  const int tid = int(threadIdx.x), ty = tid >> 4, tx = tid & 15;
  const int k0 = chunk * a.blocks_per_wg, k1 = min(a.nblk, k0 + a.blocks_per_wg);

  const float* Mg = a.M + (size_t(l) * X.H + h) * d * d;
  for (int idx = tid; idx < d * d; idx += kGradThreads) ms[(idx / d) * dp + idx % d] = Mg[idx];
  for (int idx = tid; idx < Tb * Tb; idx += kGradThreads) {
    const int u = idx / Tb, t = idx - u * Tb;
    ct[idx] = float(sqrt((u == 0 ? 1.0 : 2.0) / Tb) * cospi((2.0 * t + 1.0) * u / (2.0 * Tb)));
  }
  const double lf = a.stats[4 * l + 0], D = a.stats[4 * l + 3] + 1e-12;
  const double cf = 2.0 * a.lam_f / D, cr = a.lam_r * a.inv_count, tau = a.tau;
  double acc[TD][TD];
#pragma unroll
  for (int i = 0; i < TD; ++i)
#pragma unroll
    for (int j = 0; j < TD; ++j) acc[i][j] = 0.0;
  const size_t xbase = size_t(l) * X.sl + size_t(b) * X.sb + size_t(h) * X.sh;

  for (int blk = k0; blk < k1; ++blk) {
    __syncthreads();  // the previous block's buffers are read (and, at the start, M and C_Tb written)
    for (int idx = tid; idx < Tb * d; idx += kGradThreads) {
      const int t = idx / d, c = idx - t * d;
      const size_t off = xbase + size_t(blk * Tb + t) * X.st + c;
      xs[t * dp + c] = X.bf16 ? bf16_to_f32(((const uint16_t*)X.ptr)[off]) : ((const float*)X.ptr)[off];
    }
    __syncthreads();
    // W = X M^T: 2 tokens x 4 frequencies per thread and step
    for (int tile = tid; tile < (Tb / 2) * (d / 4); tile += kGradThreads) {
      const int t0 = 2 * (tile / (d / 4)), v0 = 4 * (tile % (d / 4));
      double w[2][4] = {};
      for (int k = 0; k < d; ++k) {
        const double x0 = xs[t0 * dp + k], x1 = xs[(t0 + 1) * dp + k];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const double m = ms[(v0 + j) * dp + k];
          w[0][j] = fma(x0, m, w[0][j]);
          w[1][j] = fma(x1, m, w[1][j]);
        }
      }
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        ws[t0 * dp + v0 + j] = w[0][j];
        ws[(t0 + 1) * dp + v0 + j] = w[1][j];
      }
    }
    __syncthreads();
    // U = C_Tb W, then dL/dU in place
    for (int idx = tid; idx < Tb * d; idx += kGradThreads) {
      const int u = idx / d, v = idx - u * d;
      double U = 0.0;
      for (int t = 0; t < Tb; ++t) U = fma(double(ct[u * Tb + t]), ws[t * dp + v], U);
      const double fu = double(u) / (Tb - 1), fv = double(v) / (d - 1);
      const double rho = sqrt(fu * fu + fv * fv) * 0.70710678118654752;
      const double sg = U > 0.0 ? 1.0 : (U < 0.0 ? -1.0 : 0.0);
      us[u * dp + v] = cf * U * (rho - lf) + cr * sg / (tau + fabs(U));
    }
    __syncthreads();
    // dL/dW = C_Tb^T dL/dU
    for (int idx = tid; idx < Tb * d; idx += kGradThreads) {
      const int t = idx / d, v = idx - t * d;
      double gw = 0.0;
      for (int u = 0; u < Tb; ++u) gw = fma(double(ct[u * Tb + t]), us[u * dp + v], gw);
      ws[t * dp + v] = gw;
    }
    __syncthreads();
    // dL/dM += (dL/dW)^T X over the block's tokens
    for (int t = 0; t < Tb; ++t) {
      double gv[TD], xv[TD];
#pragma unroll
      for (int i = 0; i < TD; ++i) {
        gv[i] = ws[t * dp + TD * ty + i];
        xv[i] = xs[t * dp + TD * tx + i];
      }
#pragma unroll
      for (int i = 0; i < TD; ++i)
#pragma unroll
        for (int j = 0; j < TD; ++j) acc[i][j] = fma(gv[i], xv[j], acc[i][j]);
    }
  }
  double* out = a.part + ((size_t(l) * X.H + h) * (size_t(X.B) * a.chunks) + size_t(b) * a.chunks + chunk) * d * d;
#pragma unroll
  for (int i = 0; i < TD; ++i)
#pragma unroll
    for (int j = 0; j < TD; ++j) out[(TD * ty + i) * d + TD * tx + j] = acc[i][j];
}

typedef double f64x4_t __attribute__((ext_vector_type(4)));

// The data pass on the binary64 matrix cores for d = 128, Tb = 16 (v_mfma_f64_16x16x4f64: lane l
// supplies A[l % 16][l / 16] and B[l / 16][l % 16] of each 16 x 4 by 4 x 16 step and holds
// D[4 v + l / 16][l % 16], v < 4), by 512-thread workgroups: wave w takes frequencies
// [16 w, 16 w + 16) of W = X M^T, one 16 x 16 tile over K = 128 channels (A = the block of X from
// LDS, B = the wave's 16 rows of M, held in registers; both exact in binary64); then U = C_Tb W and
// dL/dW = C_Tb^T dL/dU with constant DCT fragments as A and the previous result as B (item s of a
// 16 x 16 result is the B fragment of K-step s); then dL/dM rows [16 w, 16 w + 16) += (dL/dW)^T X
// over the block's tokens, the items of dL/dW serving as the A fragments of its transpose.  Eight
// waves keep two per SIMD (a wave's 16 rows of dL/dM take 64 accumulator registers), so one wave's
// matrix-core chain runs while the other's loads and dL/dU arithmetic wait.  The block of X is
// converted to binary64 once, as it is staged; each thread loads its share of the next block into
// registers while the waves multiply the current one.
constexpr int kDataThreads = 512;
template <bool BF16>
__global__ __launch_bounds__(kDataThreads) void grad_data_mfma(GradArgs a) {
  constexpr int d = 128, Tb = 16, XP = 130;  // rows of the staged block padded to 130 doubles
  extern __shared__ double smd2[];
  double* xs = smd2;           // block of X [Tb][XP], binary64
  double* rw = xs + Tb * XP;   // frequency weights [Tb][d]
  const ViewDev& X = a.X;
  const int wg = blockIdx.x, chunk = wg % a.chunks, sl = wg / a.chunks;
  const int h = sl % X.H, b = (sl / X.H) % X.B, l = sl / (X.H * X.B);
  const int tid = int(threadIdx.x), lane = tid & 63, w = tid >> 6, mi = lane & 15, mk = lane >> 4;
  const int n0 = 16 * w;  // this wave's frequencies
  const int k0 = chunk * a.blocks_per_wg, k1 = min(a.nblk, k0 + a.blocks_per_wg);

  // B fragments of W = X M^T: mf[s] = M[n0 + mi][4 s + mk]
  const float* Mg = a.M + ((size_t(l) * X.H + h) * d + n0 + mi) * d + mk;
  double mf[32];
#pragma unroll
  for (int st = 0; st < 32; ++st) mf[st] = double(Mg[4 * st]);
  // DCT fragments: cu[s] = C[mi][4 s + mk] (A of C W), cv[s] = C[4 s + mk][mi] (A of C^T dL/dU)
  double cu[4], cv[4];
#pragma unroll
  for (int st = 0; st < 4; ++st) {
    const int t = 4 * st + mk;
    cu[st] = sqrt((mi == 0 ? 1.0 : 2.0) / Tb) * cospi((2.0 * t + 1.0) * mi / (2.0 * Tb));
    cv[st] = sqrt((t == 0 ? 1.0 : 2.0) / Tb) * cospi((2.0 * mi + 1.0) * t / (2.0 * Tb));
  }
  const double lf = a.stats[4 * l + 0], D = a.stats[4 * l + 3] + 1e-12;
  const double cf = 2.0 * a.lam_f / D, cr = a.lam_r * a.inv_count, tau = a.tau;
  // the L_freq factor of dL/dU per coefficient, the same for every block of the layer:
  // rw[u][v] = 2 lambda_f (rho(u, v) - L_freq) / D
  for (int idx = tid; idx < Tb * d; idx += kDataThreads) {
    const int u = idx >> 7, v = idx & 127;
    const double fu = double(u) / (Tb - 1), fv = double(v) / (d - 1);
    rw[idx] = cf * (sqrt(fu * fu + fv * fv) * 0.70710678118654752 - lf);
  }
  f64x4_t acc[8];
#pragma unroll
  for (int jt = 0; jt < 8; ++jt) acc[jt] = f64x4_t{0.0, 0.0, 0.0, 0.0};
  // this thread's entries of a block of X: tokens tid / 128 + 4 q, channel tid % 128; the
  // pointer steps by one block of tokens per fetch
  typedef std::conditional_t<BF16, uint16_t, float> xt;
  constexpr int XQ = Tb * d / kDataThreads;  // entries of a block of X per thread
  static_assert(kDataThreads % d == 0, "whole token rows per pass");
  const xt* xp = static_cast<const xt*>(X.ptr) + size_t(l) * X.sl + size_t(b) * X.sb + size_t(h) * X.sh +
                 size_t(k0 * Tb + (tid >> 7)) * X.st + (tid & 127);
  const size_t qstride = size_t(kDataThreads / d) * X.st, bstride = size_t(Tb) * X.st;
  // raw entries, converted only when staged, so the loads stay in flight through the block
  xt rx[XQ];
  auto fetch = [&]() {
#pragma unroll
    for (int q = 0; q < XQ; ++q) rx[q] = xp[q * qstride];
    xp += bstride;
  };
  if (k0 < k1) fetch();
  for (int blk = k0; blk < k1; ++blk) {
    __syncthreads();  // the previous block's X is read (and, at the start, rw written)
#pragma unroll
    for (int q = 0; q < XQ; ++q) {
      const int idx = tid + kDataThreads * q;
      float v;
      if constexpr (BF16) v = bf16_to_f32(rx[q]);
      else v = rx[q];
      xs[(idx >> 7) * XP + (idx & 127)] = double(v);
    }
    __syncthreads();
    if (blk + 1 < k1) fetch();
    // W tile: tokens x frequencies n0 .. n0 + 15
    f64x4_t wd = {0.0, 0.0, 0.0, 0.0};
#pragma unroll
    for (int st = 0; st < 32; ++st)
      wd = __builtin_amdgcn_mfma_f64_16x16x4f64(xs[mi * XP + 4 * st + mk], mf[st], wd, 0, 0, 0);
    // U = C_Tb W (token frequency 4 v + mk, frequency n0 + mi)
    f64x4_t ud = {0.0, 0.0, 0.0, 0.0};
#pragma unroll
    for (int st = 0; st < 4; ++st) ud = __builtin_amdgcn_mfma_f64_16x16x4f64(cu[st], wd[st], ud, 0, 0, 0);
    // dL/dU = U rw + lambda_r sign(U) / (N (tau + |U|)); the reciprocal by the hardware's
    // estimate and two Newton steps (each squares the relative error: below 2^-52 after two)
    f64x4_t gu;
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const double U = ud[v], q = tau + fabs(U);
      double r = __builtin_amdgcn_rcp(q);
      r = fma(r, fma(-q, r, 1.0), r);
      r = fma(r, fma(-q, r, 1.0), r);
      const double sg = U > 0.0 ? cr : (U < 0.0 ? -cr : 0.0);
      gu[v] = fma(U, rw[(4 * v + mk) * d + n0 + mi], sg * r);
    }
    // dL/dW = C_Tb^T dL/dU
    f64x4_t gw = {0.0, 0.0, 0.0, 0.0};
#pragma unroll
    for (int st = 0; st < 4; ++st) gw = __builtin_amdgcn_mfma_f64_16x16x4f64(cv[st], gu[st], gw, 0, 0, 0);
    // dL/dM rows n0 .. n0 + 15 += (dL/dW)^T X
#pragma unroll
    for (int jt = 0; jt < 8; ++jt)
#pragma unroll
      for (int st = 0; st < 4; ++st)
        acc[jt] = __builtin_amdgcn_mfma_f64_16x16x4f64(gw[st], xs[(4 * st + mk) * XP + 16 * jt + mi], acc[jt], 0, 0, 0);
  }
  double* out = a.part + ((size_t(l) * X.H + h) * (size_t(X.B) * a.chunks) + size_t(b) * a.chunks + chunk) * d * d;
#pragma unroll
  for (int jt = 0; jt < 8; ++jt)
#pragma unroll
    for (int v = 0; v < 4; ++v) out[size_t(n0 + 4 * v + mk) * d + 16 * jt + mi] = acc[jt][v];
}

// dL/dM per (layer, head): the partials summed in order, binary64
__global__ __launch_bounds__(256) void grad_reduce(const double* part, int nparts, int d, double* dM) {
  const int lh = blockIdx.y;
  const size_t dd = size_t(d) * d;
  for (size_t idx = blockIdx.x * size_t(blockDim.x) + threadIdx.x; idx < dd; idx += size_t(gridDim.x) * blockDim.x) {
    double acc = 0.0;
    for (int p = 0; p < nparts; ++p) acc += part[(size_t(lh) * nparts + p) * dd + idx];
    dM[size_t(lh) * dd + idx] = acc;
  }
}

// C (+)= A B for g x g binary64 matrices in global memory, by the whole workgroup, through 32 x 32
// LDS tiles.  With g a multiple of 32 each of the four waves takes one 16 x 16 quarter of the
// output tile on the matrix cores (v_mfma_f64_16x16x4f64: binary64 products and sums; lane l
// supplies A[l % 16][l / 16] and B[l / 16][l % 16] of each 16 x 4 by 4 x 16 step and holds
// D[4 v + l / 16][l % 16], v < 4); otherwise binary64 FMAs on the VALU, four outputs per thread.
// Callers separate dependent products with barriers.
__device__ void wg_gemm(const double* A, const double* B, double* C, int g, bool acc) {
  static_assert(kGradThreads == 256, "four waves, one output quarter each");
  __shared__ double as[32][33], bs[32][33];
  const int tid = int(threadIdx.x), r = tid >> 3, c4 = (tid & 7) * 4;
  const int lane = tid & 63, w = tid >> 6, qi = (w >> 1) * 16, qj = (w & 1) * 16;
  const int mi = lane & 15, mk = lane >> 4;
  const bool mf = (g & 31) == 0;
  const int nt = (g + 31) / 32;
  for (int tile = 0; tile < nt * nt; ++tile) {
    const int i0 = 32 * (tile / nt), j0 = 32 * (tile % nt);
    double o[4] = {0.0, 0.0, 0.0, 0.0};
    f64x4_t dq = {0.0, 0.0, 0.0, 0.0};
    for (int k0 = 0; k0 < g; k0 += 32) {
      __syncthreads();
      for (int idx = tid; idx < 32 * 32; idx += kGradThreads) {
        const int rr = idx >> 5, cc = idx & 31;
        as[rr][cc] = (i0 + rr < g && k0 + cc < g) ? A[size_t(i0 + rr) * g + k0 + cc] : 0.0;
        bs[rr][cc] = (k0 + rr < g && j0 + cc < g) ? B[size_t(k0 + rr) * g + j0 + cc] : 0.0;
      }
      __syncthreads();
      if (mf) {
#pragma unroll
        for (int kk = 0; kk < 32; kk += 4)
          dq = __builtin_amdgcn_mfma_f64_16x16x4f64(as[qi + mi][kk + mk], bs[kk + mk][qj + mi], dq, 0, 0, 0);
      } else {
#pragma unroll 8
        for (int k = 0; k < 32; ++k) {
          const double av = as[r][k];
#pragma unroll
          for (int q = 0; q < 4; ++q) o[q] = fma(av, bs[k][c4 + q], o[q]);
        }
      }
    }
    if (mf) {
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        double* p = C + size_t(i0 + qi + 4 * v + mk) * g + j0 + qj + mi;
        *p = acc ? *p + dq[v] : dq[v];
      }
    } else if (i0 + r < g) {
#pragma unroll
      for (int q = 0; q < 4; ++q)
        if (j0 + c4 + q < g) {
          double* p = C + size_t(i0 + r) * g + j0 + c4 + q;
          *p = acc ? *p + o[q] : o[q];
        }
    }
  }
  __syncthreads();
}

// C (+)= A B for g a multiple of 64: 64 x 64 output tiles, each wave a 32 x 32 quarter of four
// 16 x 16 matrix-core tiles (lanes as in wg_gemm), 32-wide K chunks through LDS.  Each thread
// loads its share of the next chunk (the next tile's first one after a tile's last) into
// registers while the waves multiply the current one, so the global loads' latency overlaps 32
// products per wave (a second register stage spills).  Callers separate dependent products with barriers; C is neither A nor B.
__device__ void wg_gemm64(const double* A, const double* B, double* C, int g, bool acc) {
  static_assert(kGradThreads == 256, "four waves, one output quarter each");
  __shared__ double as[64][33], bs[32][65];
  const int tid = int(threadIdx.x), lane = tid & 63, w = tid >> 6;
  const int qi = (w >> 1) * 32, qj = (w & 1) * 32, mi = lane & 15, mk = lane >> 4;
  const int nt = g / 64, nk = g / 32, niter = nt * nt * nk;
  double ra[8], rb[8];
  auto fetch = [&](int it) {
    const int tile = it / nk, k0 = 32 * (it % nk), i0 = 64 * (tile / nt), j0 = 64 * (tile % nt);
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const int idx = tid + kGradThreads * q;
      ra[q] = A[size_t(i0 + (idx >> 5)) * g + k0 + (idx & 31)];
      rb[q] = B[size_t(k0 + (idx >> 6)) * g + j0 + (idx & 63)];
    }
  };
  f64x4_t dq[2][2];
  fetch(0);
  for (int it = 0; it < niter; ++it) {
    const int tile = it / nk, kc = it % nk, i0 = 64 * (tile / nt), j0 = 64 * (tile % nt);
    if (kc == 0) {
#pragma unroll
      for (int ti = 0; ti < 2; ++ti)
#pragma unroll
        for (int tj = 0; tj < 2; ++tj) dq[ti][tj] = f64x4_t{0.0, 0.0, 0.0, 0.0};
    }
    __syncthreads();  // the previous chunk's reads are done
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const int idx = tid + kGradThreads * q;
      as[idx >> 5][idx & 31] = ra[q];
      bs[idx >> 6][idx & 63] = rb[q];
    }
    __syncthreads();
    if (it + 1 < niter) fetch(it + 1);
#pragma unroll
    for (int kk = 0; kk < 32; kk += 4) {
      const double a0 = as[qi + mi][kk + mk], a1 = as[qi + 16 + mi][kk + mk];
      const double b0 = bs[kk + mk][qj + mi], b1 = bs[kk + mk][qj + 16 + mi];
      dq[0][0] = __builtin_amdgcn_mfma_f64_16x16x4f64(a0, b0, dq[0][0], 0, 0, 0);
      dq[0][1] = __builtin_amdgcn_mfma_f64_16x16x4f64(a0, b1, dq[0][1], 0, 0, 0);
      dq[1][0] = __builtin_amdgcn_mfma_f64_16x16x4f64(a1, b0, dq[1][0], 0, 0, 0);
      dq[1][1] = __builtin_amdgcn_mfma_f64_16x16x4f64(a1, b1, dq[1][1], 0, 0, 0);
    }
    if (kc == nk - 1) {
#pragma unroll
      for (int ti = 0; ti < 2; ++ti)
#pragma unroll
        for (int tj = 0; tj < 2; ++tj)
#pragma unroll
          for (int v = 0; v < 4; ++v) {
            double* p = C + size_t(i0 + qi + 16 * ti + 4 * v + mk) * g + j0 + qj + 16 * tj + mi;
            *p = acc ? *p + dq[ti][tj][v] : dq[ti][tj][v];
          }
    }
  }
  __syncthreads();
}

// C = A1 B1 (+ A2 B2 when A2 is not null) for g = 128 by a 1024-thread workgroup: wave w (of 16)
// takes the 32 x 32 output quarter at (32 (w / 4), 32 (w % 4)) as four 16 x 16 matrix-core tiles
// (lanes as in wg_gemm); the 128 x 32 chunks of A and the 32 x 128 chunks of B of each K step sit
// in LDS, and each thread loads its entries of the next chunks into registers while the waves
// multiply.  Sixteen waves per CU (four per SIMD) hide the latencies one wave per SIMD leaves
// exposed; the second product in the same pass reads no partial C back (the work matrices live
// in HBM, so the kernel's time follows their traffic).
constexpr int kWideThreads = 1024;
struct Gemm128Lds {
  double as[2][128][33], bs[2][32][129];  // the K step's chunks of A1, A2 and B1, B2
};
template <bool TWO>
__device__ void wg_gemm128(Gemm128Lds& L, const double* A1, const double* B1, const double* A2, const double* B2,
                           double* C) {
  auto& as = L.as;
  auto& bs = L.bs;
  constexpr bool two = TWO;
  const int tid = int(threadIdx.x), lane = tid & 63, w = tid >> 6;
  const int qi = (w >> 2) * 32, qj = (w & 3) * 32, mi = lane & 15, mk = lane >> 4;
  double ra[TWO ? 2 : 1][4], rb[TWO ? 2 : 1][4];
  auto fetch = [&](int k0) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int idx = tid + kWideThreads * q;
      // 32-bit offsets from uniform bases
      ra[0][q] = A1[(idx >> 5) * 128 + k0 + (idx & 31)];
      rb[0][q] = B1[(k0 + (idx >> 7)) * 128 + (idx & 127)];
      if constexpr (two) {
        ra[1][q] = A2[(idx >> 5) * 128 + k0 + (idx & 31)];
        rb[1][q] = B2[(k0 + (idx >> 7)) * 128 + (idx & 127)];
      }
    }
  };
  f64x4_t dq[2][2];
#pragma unroll
  for (int ti = 0; ti < 2; ++ti)
#pragma unroll
    for (int tj = 0; tj < 2; ++tj) dq[ti][tj] = f64x4_t{0.0, 0.0, 0.0, 0.0};
  fetch(0);
#pragma unroll 1
  for (int kc = 0; kc < 4; ++kc) {
    __syncthreads();  // the previous chunk's reads are done
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int idx = tid + kWideThreads * q;
      as[0][idx >> 5][idx & 31] = ra[0][q];
      bs[0][idx >> 7][idx & 127] = rb[0][q];
      if constexpr (two) {
        as[1][idx >> 5][idx & 31] = ra[1][q];
        bs[1][idx >> 7][idx & 127] = rb[1][q];
      }
    }
    __syncthreads();
    if (kc < 3) fetch(32 * (kc + 1));
#pragma unroll 1
    for (int pr = 0; pr < (two ? 2 : 1); ++pr) {
#pragma unroll
      for (int kk = 0; kk < 32; kk += 4) {
        const double a0 = as[pr][qi + mi][kk + mk], a1 = as[pr][qi + 16 + mi][kk + mk];
        const double b0 = bs[pr][kk + mk][qj + mi], b1 = bs[pr][kk + mk][qj + 16 + mi];
        dq[0][0] = __builtin_amdgcn_mfma_f64_16x16x4f64(a0, b0, dq[0][0], 0, 0, 0);
        dq[0][1] = __builtin_amdgcn_mfma_f64_16x16x4f64(a0, b1, dq[0][1], 0, 0, 0);
        dq[1][0] = __builtin_amdgcn_mfma_f64_16x16x4f64(a1, b0, dq[1][0], 0, 0, 0);
        dq[1][1] = __builtin_amdgcn_mfma_f64_16x16x4f64(a1, b1, dq[1][1], 0, 0, 0);
      }
    }
  }
#pragma unroll
  for (int ti = 0; ti < 2; ++ti)
#pragma unroll
    for (int tj = 0; tj < 2; ++tj)
#pragma unroll
      for (int v = 0; v < 4; ++v) C[(qi + 16 * ti + 4 * v + mk) * 128 + qj + 16 * tj + mi] = dq[ti][tj][v];
  __syncthreads();
}

// Products of the Frechet kernel by gauge width: kFrechet128 (g = 128, 1024 threads),
// kFrechet64 (g a multiple of 64, 64 x 64 tiles), kFrechetSmall (wg_gemm's 32 x 32 tiles; a
// separate instantiation, so that small groups keep the register budget that lets several blocks
// share a CU).
enum { kFrechetSmall = 0, kFrechet64 = 1, kFrechet128 = 2 };
template <int MODE>
constexpr int frechet_threads() { return MODE == kFrechet128 ? kWideThreads : kGradThreads; }
template <int MODE>
__device__ void wg_product(const double* A, const double* B, double* C, int g, bool acc) {
  if constexpr (MODE == kFrechet64) wg_gemm64(A, B, C, g, acc);
  else wg_gemm(A, B, C, g, acc);
}

// 1-norm (largest column sum of |.|) of a g x g matrix, by the whole workgroup of NT threads
template <int NT>
__device__ double wg_norm1(const double* Mx, int g, double* red) {
  double best = 0.0;
  for (int j = int(threadIdx.x); j < g; j += NT) {
    double s = 0.0;
    for (int i = 0; i < g; ++i) s += fabs(Mx[size_t(i) * g + j]);
    best = fmax(best, s);
  }
  red[threadIdx.x] = best;
  __syncthreads();
  for (int o = NT / 2; o > 0; o >>= 1) {
    if (int(threadIdx.x) < o) red[threadIdx.x] = fmax(red[threadIdx.x], red[threadIdx.x + o]);
    __syncthreads();
  }
  const double v = red[0];
  __syncthreads();
  return v;
}

// One workgroup per gauge block (l, h, r): dL/dG from dL/dM, then the Frechet adjoint and
// dL/dA.  work: twelve g x g binary64 matrices per block.
template <int MODE>
__global__ __launch_bounds__(frechet_threads<MODE>()) void grad_frechet(const double* dM, const float* A, int s, int H, int R, int g,
                                                             int d, double* work, double* grad) {
  constexpr int NT = frechet_threads<MODE>();
  __shared__ double red[NT];
  __shared__ double tab[4 * kMaxD];
  __shared__ std::conditional_t<MODE == kFrechet128, Gemm128Lds, char> glds_store;
  auto* glds = &glds_store;
  dct_table(tab, d);
  const int blk = blockIdx.x, r = blk % R, lh = blk / R, h = lh % H, l = lh / H;
  const size_t gg = size_t(g) * g;
  const double n0 = sqrt(1.0 / d), n1 = sqrt(2.0 / d);
  double* Mm = work + size_t(blk) * 12 * gg;  // W = [[Mm, Es], [0, Mm]], then its powers 2..4
  double* Es = Mm + gg;
  double* S2 = Es + gg;
  double* D2 = S2 + gg;
  double* S3 = D2 + gg;
  double* D3 = S3 + gg;
  double* S4 = D3 + gg;
  double* D4 = S4 + gg;
  double* P1 = D4 + gg;  // the running polynomial [[P1, P2], [0, P1]]
  double* P2 = P1 + gg;
  double* T1 = P2 + gg;
  double* T2 = T1 + gg;
  const double* dMl = dM + size_t(lh) * d * d;
  const float* Ab = A + ((((size_t(l) * 2 + s) * H + h) * R + r) * gg);
  // dL/dG = C_d^T dL/dM on the block (entry (c, k) sums over v in order) and S^T = A^T - A
  constexpr int QW = 16;  // most outputs per thread on the shared-load path (g^2 / NT: 16 at g = 128 and 64)
  if (MODE == kFrechet128 && g == d) {
    // one group per head: dL/dG = C_d^T dL/dM as one product, C_d^T staged in T1 from the table
    for (int idx = int(threadIdx.x); idx < int(gg); idx += NT) {
      const int c = idx / g, v = idx - c * g;
      T1[idx] = (v == 0 ? n0 : n1) * tab[((2 * c + 1) * v) % (4 * d)];
      Mm[idx] = double(Ab[size_t(v) * g + c]) - double(Ab[idx]);  // S^T = A^T - A
    }
    __syncthreads();
    if constexpr (MODE == kFrechet128) wg_gemm128<false>(*glds, T1, dMl, nullptr, nullptr, Es);
  } else if (NT % g == 0 && int(gg) / NT <= QW) {
    // thread tid: column k = tid % g of rows c = tid / g + (NT / g) q, so one load of
    // dL/dM[v][r g + k] serves all of them
    const int k = int(threadIdx.x) % g, c0 = int(threadIdx.x) / g, cs = NT / g, nq = int(gg) / NT;
    double acc[QW];
    int ti[QW], stp[QW];
#pragma unroll
    for (int q = 0; q < QW; ++q) {
      stp[q] = 2 * (r * g + c0 + cs * q) + 1;  // column r g + c of C_d, rows v = 0, 1, ...
      ti[q] = stp[q];
      acc[q] = 0.0;
    }
    const double m0 = dMl[r * g + k];
#pragma unroll
    for (int q = 0; q < QW; ++q) acc[q] = n0 * m0;  // the table's entry 0 is cos 0 = 1
    for (int v = 1; v < d; ++v) {
      const double m = dMl[size_t(v) * d + r * g + k];
#pragma unroll
      for (int q = 0; q < QW; ++q) {
        if (q < nq) acc[q] = fma(n1 * tab[ti[q]], m, acc[q]);
        ti[q] = dct_step(ti[q], stp[q], d);
      }
    }
#pragma unroll
    for (int q = 0; q < QW; ++q)
      if (q < nq) {
        const int c = c0 + cs * q, idx = c * g + k;
        Es[idx] = acc[q];                                          // dL/dG
        Mm[idx] = double(Ab[size_t(k) * g + c]) - double(Ab[idx]);  // S^T = A^T - A
      }
  } else {
#pragma nounroll
    for (int idx = int(threadIdx.x); idx < int(gg); idx += NT) {
      const int c = idx / g, k = idx - c * g;
      const int step = 2 * (r * g + c) + 1;
      double acc = n0 * dMl[r * g + k];
      for (int v = 1, ti = step; v < d; ++v, ti = dct_step(ti, step, d))
        acc = fma(n1 * tab[ti], dMl[size_t(v) * d + r * g + k], acc);
      Es[idx] = acc;
      Mm[idx] = double(Ab[size_t(k) * g + c]) - double(Ab[idx]);
    }
  }
  __syncthreads();
  const double e = wg_norm1<NT>(Es, g, red);
  double* out = grad + size_t(blk) * gg;
  if (!(e > 0.0)) {
#pragma nounroll
    for (int idx = int(threadIdx.x); idx < int(gg); idx += NT) out[idx] = 0.0;
    return;
  }
  // W = [[S^T, E / e], [0, S^T]] halved sq times until its 1-norm (at most |S^T|_1 + 1) is <= 1/2
  double nw = wg_norm1<NT>(Mm, g, red) + 1.0;
  if (!isfinite(nw) || !isfinite(e)) {  // non-finite generators or statistics: no scaling ends
#pragma nounroll
    for (int idx = int(threadIdx.x); idx < int(gg); idx += NT) out[idx] = __builtin_nan("");
    return;
  }
  int sq = 0;
  while (nw > 0.5) {
    nw *= 0.5;
    ++sq;
  }
  const double fm = ldexp(1.0, -sq), fe = fm / e;
#pragma nounroll
  for (int idx = int(threadIdx.x); idx < int(gg); idx += NT) {
    Mm[idx] *= fm;
    Es[idx] *= fe;
  }
  __syncthreads();
  // exp(W) ~= sum_{k <= 16} W^k / k! (Paterson-Stockmeyer): with B_j = sum_{i < 4} W^i / (4j + i)!,
  // p = B_0 + W^4 (B_1 + W^4 (B_2 + W^4 (B_3 + W^4 / 16!))), then p squared sq times.  Matrices of
  // the form [[X, Y], [0, X]] (powers of W, polynomials in W) are held as their two g x g parts; a
  // product of two is [[X X', X Y' + Y X'], [0, X X']], three g x g products.  Steps: W^2, W^3,
  // W^4 (0-2), three products by W^4 (3-5), each followed by adding B_j, then the squarings.  One
  // call site of the product keeps a single inlined copy of it (and its register budget).
  static_assert(kFrechetTerms == 16, "four groups of four terms and W^16");
  // P = B_j + c (Ts, Td): after a product by W^4 (c = 1), or for j = 3 from W^4 itself (c = 1 / 16!)
  auto add_b = [&](int j, const double* Ts, const double* Td, double c) {
    const double c0 = j == 3 ? inv_fact(12) : (j == 2 ? inv_fact(8) : (j == 1 ? inv_fact(4) : 1.0));
    const double c1 = j == 3 ? inv_fact(13) : (j == 2 ? inv_fact(9) : (j == 1 ? inv_fact(5) : 1.0));
    const double c2 = j == 3 ? inv_fact(14) : (j == 2 ? inv_fact(10) : (j == 1 ? inv_fact(6) : inv_fact(2)));
    const double c3 = j == 3 ? inv_fact(15) : (j == 2 ? inv_fact(11) : (j == 1 ? inv_fact(7) : inv_fact(3)));
#pragma nounroll
    for (int idx = int(threadIdx.x); idx < int(gg); idx += NT) {
      const double id = (idx / g == idx % g) ? c0 : 0.0;
      P1[idx] = id + c1 * Mm[idx] + c2 * S2[idx] + c3 * S3[idx] + c * Ts[idx];
      P2[idx] = c1 * Es[idx] + c2 * D2[idx] + c3 * D3[idx] + c * Td[idx];
    }
    __syncthreads();
  };
  // the running polynomial and the product's target swap after each squaring instead of copying
  double *Pc1 = P1, *Pc2 = P2, *Tc1 = T1, *Tc2 = T2;
  for (int step = 0; step < 6 + sq; ++step) {
    const double *Xs, *Xd, *Ys, *Yd;
    double *Cs, *Cd;
    if (step == 0) { Xs = Mm; Xd = Es; Ys = Mm; Yd = Es; Cs = S2; Cd = D2; }
    else if (step == 1) { Xs = S2; Xd = D2; Ys = Mm; Yd = Es; Cs = S3; Cd = D3; }
    else if (step == 2) { Xs = S2; Xd = D2; Ys = S2; Yd = D2; Cs = S4; Cd = D4; }
    else if (step < 6) { Xs = S4; Xd = D4; Ys = P1; Yd = P2; Cs = T1; Cd = T2; }
    else { Xs = Pc1; Xd = Pc2; Ys = Pc1; Yd = Pc2; Cs = Tc1; Cd = Tc2; }
    if (step == 3) add_b(3, S4, D4, inv_fact(16));
    if constexpr (MODE == kFrechet128) {
      // Cs = Xs Ys, then Cd = Xs Yd + Xd Ys in one pass
      wg_gemm128<false>(*glds, Xs, Ys, nullptr, nullptr, Cs);
      wg_gemm128<true>(*glds, Xs, Yd, Xd, Ys, Cd);
    } else {
#pragma unroll 1
      for (int q = 0; q < 3; ++q)  // Cs = Xs Ys, Cd = Xs Yd + Xd Ys
        wg_product<MODE>(q == 2 ? Xd : Xs, q == 0 ? Ys : (q == 1 ? Yd : Ys), q == 0 ? Cs : Cd, g, q == 2);
    }
    if (step >= 3 && step < 6) {
      add_b(5 - step, T1, T2, 1.0);
    } else if (step >= 6) {
      double* t = Pc1; Pc1 = Tc1; Tc1 = t;
      t = Pc2; Pc2 = Tc2; Tc2 = t;
    }
  }
  // dL/dS = e P2, dL/dA = dL/dS - (dL/dS)^T
#pragma nounroll
  for (int idx = int(threadIdx.x); idx < int(gg); idx += NT) {
    const int i = idx / g, j = idx - i * g;
    out[idx] = e * (Pc2[idx] - Pc2[size_t(j) * g + i]);
  }
}

// The same Frechet step for g <= 16: one wave per gauge block, every matrix in LDS, zero-padded to
// 16 x 16 (rows padded to 17 doubles against bank conflicts), each product four
// v_mfma_f64_16x16x4f64 steps (lanes as in wg_gemm).  Products of zero-padded matrices are zero
// outside the g x g part and the identity is placed on that part only, so the padding stays zero
// and the g x g part follows grad_frechet step for step (norms, scaling, series, squarings),
// without the global work area or the workgroup-wide tiles a 16 x 16 product does not fill.
constexpr int kF16 = 16, kF16P = 17;
__global__ __launch_bounds__(64) void grad_frechet16(const double* dM, const float* A, int s, int H, int R, int g, int d,
                                                     double* grad) {
  __shared__ double tab[4 * kMaxD];
  __shared__ double mt[12][kF16 * kF16P];
  dct_table(tab, d);
  const int lane = int(threadIdx.x), mi = lane & 15, mk = lane >> 4;
  const int blk = blockIdx.x, r = blk % R, lh = blk / R, h = lh % H, l = lh / H;
  const int gg = g * g;
  const double n0 = sqrt(1.0 / d), n1 = sqrt(2.0 / d);
  double *Mm = mt[0], *Es = mt[1], *S2 = mt[2], *D2 = mt[3], *S3 = mt[4], *D3 = mt[5];
  double *S4 = mt[6], *D4 = mt[7], *P1 = mt[8], *P2 = mt[9], *T1 = mt[10], *T2 = mt[11];
  auto at = [](int i, int j) { return i * kF16P + j; };
  const double* dMl = dM + size_t(lh) * d * d;
  const float* Ab = A + ((((size_t(l) * 2 + s) * H + h) * R + r) * size_t(gg));
  // dL/dG = C_d^T dL/dM on the block and S^T = A^T - A, zero outside g x g: lane holds column
  // k = lane % 16 of rows c = lane / 16 + 4 q, so one load of dL/dM[v][r g + k] serves its four
  // entries (each summed over v in order)
  {
    const int k = lane & 15, c0 = lane >> 4;
    const bool kin = k < g;
    double acc[4];
    int ti[4], stp[4];
    const double m0 = kin ? dMl[r * g + k] : 0.0;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      stp[q] = 2 * (r * g + c0 + 4 * q) + 1;  // column r g + c of C_d, rows v = 0, 1, ...
      ti[q] = stp[q];
      acc[q] = n0 * m0;                        // the table's entry 0 is cos 0 = 1
    }
    for (int v = 1; v < d; ++v) {
      const double m = kin ? dMl[size_t(v) * d + r * g + k] : 0.0;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        acc[q] = fma(n1 * tab[ti[q]], m, acc[q]);
        ti[q] = dct_step(ti[q], stp[q], d);
      }
    }
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int c = c0 + 4 * q;
      const bool in = kin && c < g;
      Es[at(c, k)] = in ? acc[q] : 0.0;
      Mm[at(c, k)] = in ? double(Ab[k * g + c]) - double(Ab[c * g + k]) : 0.0;
    }
  }
  __syncthreads();
  // 1-norm: lane j < 16 sums column j in row order, then the largest over the wave
  auto norm1 = [&](const double* X) {
    double sum = 0.0;
    if (lane < kF16)
      for (int i = 0; i < kF16; ++i) sum += fabs(X[at(i, lane)]);
    for (int o = 32; o > 0; o >>= 1) sum = fmax(sum, __shfl_xor(sum, o));
    return sum;
  };
  const double e = norm1(Es);
  double* out = grad + size_t(blk) * gg;
  if (!(e > 0.0)) {
    for (int idx = lane; idx < gg; idx += 64) out[idx] = 0.0;
    return;
  }
  double nw = norm1(Mm) + 1.0;
  if (!isfinite(nw) || !isfinite(e)) {
    for (int idx = lane; idx < gg; idx += 64) out[idx] = __builtin_nan("");
    return;
  }
  int sq = 0;
  while (nw > 0.5) {
    nw *= 0.5;
    ++sq;
  }
  const double fm = ldexp(1.0, -sq), fe = fm / e;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int idx = lane + 64 * q, o = at(idx >> 4, idx & 15);
    Mm[o] *= fm;
    Es[o] *= fe;
  }
  __syncthreads();
  // C (+)= X Y, 16 x 16
  auto prod = [&](const double* X, const double* Y, double* C, bool acc) {
    f64x4_t dq = {0.0, 0.0, 0.0, 0.0};
#pragma unroll
    for (int st = 0; st < 4; ++st)
      dq = __builtin_amdgcn_mfma_f64_16x16x4f64(X[at(mi, 4 * st + mk)], Y[at(4 * st + mk, mi)], dq, 0, 0, 0);
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      double* p = C + at(4 * v + mk, mi);
      *p = acc ? *p + dq[v] : dq[v];
    }
    __syncthreads();
  };
  // [[Cs, Cd], [0, Cs]] = [[Xs, Xd], [0, Xs]] [[Ys, Yd], [0, Ys]]
  auto blk_prod = [&](const double* Xs, const double* Xd, const double* Ys, const double* Yd, double* Cs, double* Cd) {
    prod(Xs, Ys, Cs, false);
    prod(Xs, Yd, Cd, false);
    prod(Xd, Ys, Cd, true);
  };
  // P = B_j + c (Ts, Td), as in grad_frechet, the identity on the g x g part only
  auto add_b = [&](int j, const double* Ts, const double* Td, double c) {
    const double c0 = j == 3 ? inv_fact(12) : (j == 2 ? inv_fact(8) : (j == 1 ? inv_fact(4) : 1.0));
    const double c1 = j == 3 ? inv_fact(13) : (j == 2 ? inv_fact(9) : (j == 1 ? inv_fact(5) : 1.0));
    const double c2 = j == 3 ? inv_fact(14) : (j == 2 ? inv_fact(10) : (j == 1 ? inv_fact(6) : inv_fact(2)));
    const double c3 = j == 3 ? inv_fact(15) : (j == 2 ? inv_fact(11) : (j == 1 ? inv_fact(7) : inv_fact(3)));
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int idx = lane + 64 * q, i = idx >> 4, jj = idx & 15, o = at(i, jj);
      const double id = (i == jj && i < g) ? c0 : 0.0;
      P1[o] = id + c1 * Mm[o] + c2 * S2[o] + c3 * S3[o] + c * Ts[o];
      P2[o] = c1 * Es[o] + c2 * D2[o] + c3 * D3[o] + c * Td[o];
    }
    __syncthreads();
  };
  blk_prod(Mm, Es, Mm, Es, S2, D2);
  blk_prod(S2, D2, Mm, Es, S3, D3);
  blk_prod(S2, D2, S2, D2, S4, D4);
  add_b(3, S4, D4, inv_fact(16));
#pragma unroll 1
  for (int j = 2; j >= 0; --j) {
    blk_prod(S4, D4, P1, P2, T1, T2);
    add_b(j, T1, T2, 1.0);
  }
#pragma unroll 1
  for (int q = 0; q < sq; ++q) {
    blk_prod(P1, P2, P1, P2, T1, T2);
#pragma unroll
    for (int qq = 0; qq < 4; ++qq) {
      const int idx = lane + 64 * qq, o = at(idx >> 4, idx & 15);
      P1[o] = T1[o];
      P2[o] = T2[o];
    }
    __syncthreads();
  }
  // dL/dS = e P2, dL/dA = dL/dS - (dL/dS)^T
  for (int idx = lane; idx < gg; idx += 64) {
    const int i = idx / g, j = idx - i * g;
    out[idx] = e * (P2[at(i, j)] - P2[at(j, i)]);
  }
}

template <int TD>
hipError_t launch_data(const GradArgs& a, int nwg, size_t smem, hipStream_t st) {
  hipError_t e;
  if (smem > 65536 &&
      (e = hipFuncSetAttribute((const void*)grad_data<TD>, hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem)) !=
          hipSuccess)
    return e;
  hipLaunchKernelGGL(grad_data<TD>, dim3(nwg), dim3(kGradThreads), smem, st, a);
  return hipGetLastError();
}

}  // namespace

GradLayout grad_layout(const cg_gauge_shape& s, int B, int T, int Tb) {
  GradLayout o;
  const int nblk = Tb > 0 ? T / Tb : 0;
  // about 1024 workgroups over the (layer, batch row, head) slices, at least 4 blocks each
  const int nslices = s.L * B * s.H;
  int chunks = std::max(1, (1024 + nslices - 1) / std::max(nslices, 1));
  chunks = std::min(chunks, std::max(1, nblk / 4));
  o.blocks_per_wg = nblk > 0 ? (nblk + chunks - 1) / chunks : 1;
  o.chunks = nblk > 0 ? (nblk + o.blocks_per_wg - 1) / o.blocks_per_wg : 1;
  const size_t dd = size_t(s.d) * s.d, gg = size_t(s.g) * s.g;
  const size_t nlh = size_t(s.L) * s.H;
  size_t off = align256(spec_layout(s, Tb).total);
  o.off_m = off;
  off = align256(off + nlh * dd * 4);
  o.off_part = off;
  off = align256(off + nlh * size_t(B) * o.chunks * dd * 8);
  o.off_dm = off;
  off = align256(off + nlh * dd * 8);
  o.off_work = off;
  off = align256(off + nlh * (s.d / s.g) * 12 * gg * 8);
  o.total = off;
  return o;
}

hipError_t launch_gauge_grad(int s, const ViewDev& X, const GaugeDev& G, const float* A, int Tb, float tau, float lam_f,
                             float lam_r, void* ws, double* stats, double* grad, bool force_generic, hipStream_t st) {
  const cg_gauge_shape shp{X.L, X.H, X.d, G.g};
  hipError_t e = launch_spectral(s, X, G, Tb, tau, ws, stats, nullptr, force_generic, st);
  if (e != hipSuccess) return e;
  const GradLayout lay = grad_layout(shp, X.B, X.T, Tb);
  char* base = static_cast<char*>(ws);
  float* M = reinterpret_cast<float*>(base + lay.off_m);
  double* part = reinterpret_cast<double*>(base + lay.off_part);
  double* dM = reinterpret_cast<double*>(base + lay.off_dm);
  double* work = reinterpret_cast<double*>(base + lay.off_work);
  const int d = X.d, R = d / G.g, nblk = X.T / Tb;
  hipLaunchKernelGGL(grad_prep, dim3((d * (d / kPrepRows) + 255) / 256, X.L * X.H), dim3(256), 0, st, s, G, X.H, d, M);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  GradArgs a{};
  a.X = X;
  a.M = M;
  a.stats = stats;
  a.part = part;
  a.Tb = Tb;
  a.nblk = nblk;
  a.chunks = lay.chunks;
  a.blocks_per_wg = lay.blocks_per_wg;
  a.tau = tau;
  a.inv_tau = 1.0f / tau;
  a.lam_f = lam_f;
  a.lam_r = lam_r;
  const double count = double(X.B) * X.H * nblk * Tb * d;
  a.inv_count = count > 0 ? 1.0 / count : 0.0;
  const int nwg = X.L * X.B * X.H * lay.chunks;
  const size_t smem = size_t(2) * Tb * (d + 1) * sizeof(double) +
                      (size_t(d) * (d + 1) + size_t(Tb) * (d + 1) + size_t(Tb) * Tb) * sizeof(float);
  if (nblk > 0 && d == 128 && Tb == 16 && !force_generic) {
    const size_t smf = (size_t(16) * 130 + size_t(16) * 128) * sizeof(double);
    const void* fn = X.bf16 ? (const void*)grad_data_mfma<true> : (const void*)grad_data_mfma<false>;
    if ((e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)smf)) != hipSuccess) return e;
    void* args[] = {&a};
    if ((e = hipLaunchKernel(fn, dim3(nwg), dim3(kDataThreads), args, smf, st)) != hipSuccess) return e;
    if ((e = hipGetLastError()) != hipSuccess) return e;
  } else if (nblk > 0) {
    switch (d / 16) {
      case 1: e = launch_data<1>(a, nwg, smem, st); break;
      case 2: e = launch_data<2>(a, nwg, smem, st); break;
      case 3: e = launch_data<3>(a, nwg, smem, st); break;
      case 4: e = launch_data<4>(a, nwg, smem, st); break;
      case 5: e = launch_data<5>(a, nwg, smem, st); break;
      case 6: e = launch_data<6>(a, nwg, smem, st); break;
      case 7: e = launch_data<7>(a, nwg, smem, st); break;
      case 8: e = launch_data<8>(a, nwg, smem, st); break;
      default: return hipErrorInvalidValue;
    }
    if (e != hipSuccess) return e;
  }
  const int nparts = nblk > 0 ? X.B * lay.chunks : 0;
  hipLaunchKernelGGL(grad_reduce, dim3((d * d + 255) / 256, X.L * X.H), dim3(256), 0, st, part, nparts, d, dM);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if (G.g == 128)
    hipLaunchKernelGGL(grad_frechet<kFrechet128>, dim3(X.L * X.H * R), dim3(kWideThreads), 0, st, dM, A, s, X.H, R, G.g,
                       d, work, grad);
  else if (G.g <= kF16)
    hipLaunchKernelGGL(grad_frechet16, dim3(X.L * X.H * R), dim3(64), 0, st, dM, A, s, X.H, R, G.g, d, grad);
  else if (G.g % 64 == 0)
    hipLaunchKernelGGL(grad_frechet<kFrechet64>, dim3(X.L * X.H * R), dim3(kGradThreads), 0, st, dM, A, s, X.H, R, G.g,
                       d, work, grad);
  else
    hipLaunchKernelGGL(grad_frechet<kFrechetSmall>, dim3(X.L * X.H * R), dim3(kGradThreads), 0, st, dM, A, s, X.H, R,
                       G.g, d, work, grad);
  return hipGetLastError();
}

}  // namespace cg
