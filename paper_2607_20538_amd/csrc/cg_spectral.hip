// Codec-facing spectral statistics of the gauge training objective (section 4.2).
//
// For the gauge-transformed cache X' = G X of one cache type, the token axis is cut into
// blocks of Tb tokens and each Tb x d block goes through the orthonormal 2-D DCT-II,
// U = C_Tb Z C_d^T (rows: token frequency u, columns: channel-layout frequency v).  Per layer
// the kernels accumulate the energy map E_uv = sum over blocks of U_uv^2 and the sum of
// log(1 + |U| / tau) over all coefficients; a final kernel forms
//   L_freq = sum E rho / (sum E + eps),  rho(u, v) = sqrt((u/(Tb-1))^2 + (v/(d-1))^2) / sqrt(2),
//   L_rate = mean log(1 + |U| / tau),   concentration = 1 - L_freq.
//
// Matrix-core path (bf16, d = 128, Tb = 16): the channel DCT is folded into the gauge,
// M = C_d G (one dense 128 x 128 matrix per (layer, head), built in binary64 and split into
// two bf16 planes), so one matrix-core chain per 32-token tile gives y = M x = C_d z for the
// tile's tokens.  The chain runs transposed (the tile as the A operand), so a lane holds one
// channel-layout frequency v of 16 tokens; the lane pair exchanges half-waves so that each lane
// holds the 16 tokens of one block, and the token DCT is an in-lane 16-point DCT by even / odd
// splits (120 operations for 16 outputs).  Energies accumulate per lane in binary64 and leave
// by atomic adds at the end of the workgroup; log(1 + |U| / tau) is summed as log2 (the
// hardware's v_log_f32 on an argument >= 1) and scaled by ln 2 once.  The matrix-core chain of
// tile t + 1 is issued before the VALU work of tile t (two accumulators).
//
// General path (any supported d and g, bf16 or binary32 input, Tb in {2, 4, 8, 16, 32}): one
// workgroup per block, gauge, channel DCT and token DCT on the VALU in binary32 through LDS.
#include <algorithm>
#include <cstdlib>
#include <utility>

#include "cg_internal.h"
#include "cg_device.h"
#include "cg_mfma_util.h"

namespace cg {

namespace {

constexpr int kSpecStages = 5;   // LDS ring of the matrix-core path
constexpr int kSpecTb = 16;      // block length of the matrix-core path

__global__ void spec_init(double* acc, size_t nacc, double* lsum, int L, double* cd, int d) {
  const size_t i = blockIdx.x * size_t(blockDim.x) + threadIdx.x;
  if (i < nacc) acc[i] = 0.0;
  if (i < size_t(L)) lsum[i] = 0.0;
  if (i < size_t(d) * d) {
    const int k = int(i / d), n = int(i % d);
    cd[i] = sqrt((k == 0 ? 1.0 : 2.0) / d) * cospi((2.0 * n + 1.0) * k / (2.0 * d));
  }
}

// M = C_d G_{l,s,h} (G block-diagonal over its R groups), products and sums in binary64 from
// the binary32 DCT rows and gauge, rounded to binary32 and split into two bf16 planes.  One
// workgroup of 1024 threads per (l, h) stages C_d (row pitch 129 floats, so that a fragment's 16
// rows fall in 16 banks) and the gauge blocks in LDS; wave w (of 16) takes the 32 x 32 quarter
// of M at (32 (w / 4), 32 (w % 4)) as four 16 x 16 binary64 matrix-core tiles
// (v_mfma_f64_16x16x4f64: lane l supplies A[l % 16][l / 16] and B[l / 16][l % 16] of each step
// and holds D[4 v + l / 16][l % 16]), the K range of a tile limited to the gauge rows its
// columns read (gs is zero outside a column's group).
constexpr int kMprepThreads = 1024;
constexpr int kCdPitch = kD + 1;
typedef double f64x4_t __attribute__((ext_vector_type(4)));
__global__ __launch_bounds__(kMprepThreads) void spec_mprep(int s, GaugeDev G, int H, const double* cd, uint16_t* m0,
                                                   uint16_t* m1) {
  __shared__ float cds[kD * kCdPitch];  // C_d rows
  __shared__ float gs[kD * kD];         // gs[a_global][j]: G_{r}[a][j - r g] for j in group r, a = a_global - r g
  const int lh = blockIdx.x, l = lh / H, h = lh - l * H;
  const int g = G.g;
  for (int idx = threadIdx.x; idx < kD * kD; idx += blockDim.x) {
    const int ag = idx / kD, j = idx - ag * kD, r = j / g;
    cds[ag * kCdPitch + j] = float(cd[idx]);
    const int a = ag - r * g;
    float v = 0.0f;
    if (a >= 0 && a < g) v = G.f32[((((size_t(l) * 2 + s) * G.H + h) * G.R + r) * g + a) * g + (j - r * g)];
    gs[idx] = v;
  }
  __syncthreads();
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, mi = lane & 15, mk = lane >> 4;
  const int qi = (w >> 2) * 32, qj = (w & 3) * 32;
  const int kw = g > 16 ? g : 16;  // K range of a 16-column tile: its group, or the groups it spans
#pragma unroll
  for (int tj = 0; tj < 2; ++tj) {
    const int j0 = qj + 16 * tj, ks = (j0 / kw) * kw;
#pragma unroll
    for (int ti = 0; ti < 2; ++ti) {
      const int i0 = qi + 16 * ti;
      f64x4_t dq = {0.0, 0.0, 0.0, 0.0};
      for (int k = ks; k < ks + kw; k += 4)
        dq = __builtin_amdgcn_mfma_f64_16x16x4f64(double(cds[(i0 + mi) * kCdPitch + k + mk]),
                                                  double(gs[(k + mk) * kD + j0 + mi]), dq, 0, 0, 0);
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const float x = float(dq[v]);
        const uint32_t hi = f32_to_bf16_rne(x);
        const uint32_t lo = f32_to_bf16_rne(x - __uint_as_float(hi << 16));
        const size_t off = (size_t(lh) * kD + i0 + 4 * v + mk) * kD + j0 + mi;
        m0[off] = uint16_t(hi);
        m1[off] = uint16_t(lo);
      }
    }
  }
}

struct SpecArgs {
  const char* x;
  int64_t sl, sb, sh, st;   // element strides of the bf16 view
  int L, B, H;
  const uint16_t* m0;       // planes of M, [L][H][128][128]
  const uint16_t* m1;
  double* acc;              // [L][16][128]
  double* lsum;             // [L]
  float inv_tau;
  int nblk;                 // whole 16-token blocks per slice
  int nslices, chunks, tiles_per_wg;
};

// cos(pi x) at compile time: x reduced to [0, 1), then the Taylor series of cos at pi x
// (|pi x| < pi: the 30 terms below are exact to binary64 rounding)
constexpr double cos_pi(double x) {
  while (x >= 2.0) x -= 2.0;
  double sign = 1.0;
  if (x >= 1.0) {  // cos(pi (x - 1)) = -cos(pi x)
    x -= 1.0;
    sign = -1.0;
  }
  const double th = 3.14159265358979323846 * x, th2 = th * th;
  double term = 1.0, sum = 1.0;
  for (int k = 1; k < 30; ++k) {
    term *= -th2 / double((2 * k - 1) * (2 * k));
    sum += term;
  }
  return sign * sum;
}

// Orthonormal 16-point DCT-II, U[u] = a_u sum_t y[t] cos(pi (2t + 1) u / 32) (a_0 = sqrt(1/16),
// a_u = sqrt(2/16)), by its even / odd splits: with s[t] = y[t] + y[15 - t] and d[t] =
// y[t] - y[15 - t] (t < 8), the odd outputs are an 8 x 8 product with d; with ss[t] = s[t] +
// s[7 - t] and sd[t] = s[t] - s[7 - t] (t < 4), U[4m + 2] and U[4m] are 4 x 4 products with sd
// and ss.  The tables hold a_u times the cosines.
struct Dct16Tables {
  float odd[8][8], e2[4][4], e4[4][4];
};
constexpr Dct16Tables make_dct16() {
  Dct16Tables c{};
  const double a0 = 0.25, a1 = 0.35355339059327376220;  // sqrt(1/16), sqrt(2/16)
  for (int k = 0; k < 8; ++k)
    for (int t = 0; t < 8; ++t) c.odd[k][t] = float(a1 * cos_pi((2.0 * t + 1.0) * (2.0 * k + 1.0) / 32.0));
  for (int m = 0; m < 4; ++m)
    for (int t = 0; t < 4; ++t) {
      c.e2[m][t] = float(a1 * cos_pi((2.0 * t + 1.0) * (2.0 * m + 1.0) / 16.0));
      c.e4[m][t] = float((m == 0 ? a0 : a1) * cos_pi((2.0 * t + 1.0) * m / 8.0));
    }
  return c;
}
constexpr Dct16Tables kDct16 = make_dct16();

__device__ __forceinline__ void dct16(const float (&y)[16], float (&U)[16]) {
  float s[8], d[8], ss[4], sd[4];
#pragma unroll
  for (int t = 0; t < 8; ++t) {
    s[t] = y[t] + y[15 - t];
    d[t] = y[t] - y[15 - t];
  }
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    ss[t] = s[t] + s[7 - t];
    sd[t] = s[t] - s[7 - t];
  }
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    float v = kDct16.odd[k][0] * d[0];
#pragma unroll
    for (int t = 1; t < 8; ++t) v = fmaf(kDct16.odd[k][t], d[t], v);
    U[2 * k + 1] = v;
  }
#pragma unroll
  for (int m = 0; m < 4; ++m) {
    float v2 = kDct16.e2[m][0] * sd[0], v4 = kDct16.e4[m][0] * ss[0];
#pragma unroll
    for (int t = 1; t < 4; ++t) {
      v2 = fmaf(kDct16.e2[m][t], sd[t], v2);
      v4 = fmaf(kDct16.e4[m][t], ss[t], v4);
    }
    U[4 * m + 2] = v2;
    U[4 * m] = v4;
  }
}

__global__ __launch_bounds__(kThreads, 2) void spec_mfma(SpecArgs a) {
  __shared__ __attribute__((aligned(16))) uint8_t xtile[kSpecStages][kTok * kRowBytes];

  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int n = lane & 31, hc = lane >> 5;
  const int logical = xcd_remap(blockIdx.x, gridDim.x);
  const int slice = logical / a.chunks, chunk = logical - slice * a.chunks;
  if (slice >= a.nslices) return;
  const int h = slice % a.H, b = (slice / a.H) % a.B, l = slice / (a.H * a.B);
  const int Tu = a.nblk * kSpecTb;  // tokens in whole blocks
  const int ntiles = (Tu + kTok - 1) / kTok;
  const int tb = chunk * a.tiles_per_wg;
  const int te = min(ntiles, tb + a.tiles_per_wg);
  if (tb >= te) return;
  const char* xs = a.x + 2 * (size_t(l) * a.sl + size_t(b) * a.sb + size_t(h) * a.sh);
  const int64_t tstride = 2 * a.st;

  // rows chA of the planes of M (output channel = channel-layout frequency v)
  const int chA = 32 * w + 16 * ((n >> 2) & 1) + 4 * (n >> 3) + (n & 3);
  bf16x8_t A[2][8];
#pragma unroll
  for (int kk = 0; kk < 8; ++kk) {
    const size_t off = ((size_t(l) * a.H + h) * kD + chA) * kD + 16 * kk + 8 * hc;
    A[0][kk] = as_bf16x8(*(const u32x4_t*)(a.m0 + off));
    A[1][kk] = as_bf16x8(*(const u32x4_t*)(a.m1 + off));
  }
  // LDS-direct tile loads as in the encoder: wave w moves rows 8w .. 8w+7 with two 1 KB
  // instructions; rows past the whole blocks repeat the last used row
  const int wu = __builtin_amdgcn_readfirstlane(w);
  int drow[2];
  const char* dsrc[2];
#pragma unroll
  for (int q = 0; q < 2; ++q) {
    drow[q] = 8 * w + 4 * q + (lane >> 4);
    dsrc[q] = xs + drow[q] * tstride + 16 * swz(drow[q], lane & 15);
  }
  auto issue = [&](int tile) {
    uint8_t* dst = xtile[(tile - tb) % kSpecStages] + 8 * wu * kRowBytes;
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const int tok = min(tile * kTok + drow[q], Tu - 1);
      __builtin_amdgcn_global_load_lds(dsrc[q] + (int64_t(tok) - drow[q]) * tstride,
                                       (__attribute__((address_space(3))) void*)(dst + 4 * q * kRowBytes), 16, 0, 0);
    }
  };
  auto wait_tile = [&](int in_flight) {  // loads of later tiles that may stay outstanding
    switch (in_flight) {
      case 0: __builtin_amdgcn_s_waitcnt(waitcnt_imm(0)); break;
      case 1: __builtin_amdgcn_s_waitcnt(waitcnt_imm(2)); break;
      case 2: __builtin_amdgcn_s_waitcnt(waitcnt_imm(4)); break;
      case 3: __builtin_amdgcn_s_waitcnt(waitcnt_imm(6)); break;
      default: __builtin_amdgcn_s_waitcnt(waitcnt_imm(8)); break;
    }
  };
  int boff[8];
#pragma unroll
  for (int kk = 0; kk < 8; ++kk) boff[kk] = n * kRowBytes + 16 * swz(n, 2 * kk + hc);

  // energy accumulators of the lane's entries (u = 0..15, v = chA): the lane pair (n, 0) and
  // (n, 1) holds the same entries for the tile's two blocks
  // (squares summed in binary32 over at most kFold tiles, then added to the binary64 totals:
  // the terms are positive, so the binary32 partial is within kFold 2^-24 of its value)
  constexpr int kFold = 8;
  double eacc[16];
  float ef[16];
#pragma unroll
  for (int e = 0; e < 16; ++e) {
    eacc[e] = 0.0;
    ef[e] = 0.0f;
  }
  double lacc = 0.0;
  // y^T = x^T M^T of tile t on the matrix cores: the tile is the A operand and the planes of M
  // the B operand, so lane (n, hc) holds channel chA of tokens 8 (e / 4) + 4 hc + e % 4
  auto chain = [&](int t) {
    const uint8_t* src_t = xtile[(t - tb) % kSpecStages];
    f32x16_t acc = {};
#pragma unroll
    for (int kk = 0; kk < 8; ++kk) {
      const bf16x8_t bv = as_bf16x8(*(const u32x4_t*)(src_t + boff[kk]));
      acc = mfma(bv, A[1][kk], acc);
      acc = mfma(bv, A[0][kk], acc);
    }
    return acc;
  };
  // the lane pair exchanges half-waves (v_permlane32_swap) so that lane (n, hc) holds all 16
  // tokens of block hc of the tile, then the token DCT runs in-lane; coefficients of a block past
  // the whole ones count as 0 (no energy, log2 1 = 0)
  auto epilogue = [&](int t, const f32x16_t& acc) {
    float y[16];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(acc[e]), __float_as_uint(acc[e + 8]), false, false);
      y[8 * (e >> 2) + (e & 3)] = __uint_as_float(r[0]);
      y[8 * (e >> 2) + 4 + (e & 3)] = __uint_as_float(r[1]);
    }
    float U[16];
    dct16(y, U);
    const bool valid = 2 * t + hc < a.nblk;
    float ls = 0.0f;
#pragma unroll
    for (int u = 0; u < 16; ++u) {
      const float x = valid ? U[u] : 0.0f;
      ef[u] = fmaf(x, x, ef[u]);
      // log2 of an argument >= 1 (v_log_f32); the sum is scaled by ln 2 once, at the end
      ls += __builtin_amdgcn_logf(fmaf(fabsf(x), a.inv_tau, 1.0f));
    }
    lacc += double(ls);
    if ((t - tb) % kFold == kFold - 1 || t == te - 1) {
#pragma unroll
      for (int u = 0; u < 16; ++u) {
        eacc[u] += double(ef[u]);
        ef[u] = 0.0f;
      }
    }
  };
  // software pipeline: the matrix-core chain of tile t + 1 runs while the VALU works on tile t
  for (int t = tb; t < min(te, tb + kSpecStages - 1); ++t) issue(t);
  wait_tile(min(te - 1, tb + kSpecStages - 2) - tb);
  __builtin_amdgcn_s_barrier();
  f32x16_t accs[2];
  accs[0] = chain(tb);
  auto step = [&](int t, auto parity) {
    constexpr int P = decltype(parity)::value;
    if (t + 1 < te) {
      // tile t + 1 landed in every wave, every wave is done with the buffer tile t - 1 used
      wait_tile(min(te - 1, t + kSpecStages - 2) - (t + 1));
      __builtin_amdgcn_s_barrier();
      if (t + kSpecStages - 1 < te) issue(t + kSpecStages - 1);
      accs[P ^ 1] = chain(t + 1);
    }
    epilogue(t, accs[P]);
  };
  int t = tb;
  for (; t + 1 < te; t += 2) {
    step(t, std::integral_constant<int, 0>());
    step(t + 1, std::integral_constant<int, 1>());
  }
  if (t < te) step(t, std::integral_constant<int, 0>());
  // energy map entries (u, v = chA) and the log sum
  double* accl = a.acc + size_t(l) * kSpecTb * kD + chA;
#pragma unroll
  for (int u = 0; u < 16; ++u) atomicAdd(accl + u * kD, eacc[u]);
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) lacc += __shfl_xor(lacc, off);
  if (lane == 0) atomicAdd(a.lsum + l, lacc * 0.69314718055994530942);  // log2 -> natural log
}

// General path: one workgroup per (slice, block).  xs, zs: [Tb][d + 1] binary32; ct:
// [Tb][Tb] token DCT rows.
__global__ __launch_bounds__(256) void spec_generic(int s, ViewDev X, GaugeDev G, int Tb, float inv_tau,
                                                      const double* cd, double* acc, double* lsum) {
  extern __shared__ float sm[];
  const int d = X.d, dp = d + 1;
  float* xs = sm;
  float* zs = sm + Tb * dp;
  float* ct = zs + Tb * dp;
  __shared__ double red[256];
  const int sv = blockIdx.x, blk = blockIdx.y;
  const int h = sv % X.H, b = (sv / X.H) % X.B, l = sv / (X.H * X.B);
  const size_t xbase = size_t(l) * X.sl + size_t(b) * X.sb + size_t(h) * X.sh + size_t(blk) * Tb * X.st;
  for (int idx = threadIdx.x; idx < Tb * d; idx += blockDim.x) {
    const int t = idx / d, c = idx - t * d;
    const size_t off = xbase + size_t(t) * X.st + c;
    xs[t * dp + c] = X.bf16 ? bf16_to_f32(((const uint16_t*)X.ptr)[off]) : ((const float*)X.ptr)[off];
  }
  for (int idx = threadIdx.x; idx < Tb * Tb; idx += blockDim.x) {
    const int u = idx / Tb, t = idx - u * Tb;
    ct[idx] = float(sqrt((u == 0 ? 1.0 : 2.0) / Tb) * cospi((2.0 * t + 1.0) * u / (2.0 * Tb)));
  }
  __syncthreads();
  // z = G x per token (binary32 gauge)
  const int g = G.g;
  for (int idx = threadIdx.x; idx < Tb * d; idx += blockDim.x) {
    const int t = idx / d, c = idx - t * d, r = c / g, cc = c - r * g;
    const float* Gr = G.f32 + ((((size_t(l) * 2 + s) * G.H + h) * G.R + r) * g + cc) * g;
    float v = 0.0f;
    for (int j = 0; j < g; ++j) v = fmaf(Gr[j], xs[t * dp + r * g + j], v);
    zs[t * dp + c] = v;
  }
  __syncthreads();
  // y = C_d z per token
  for (int idx = threadIdx.x; idx < Tb * d; idx += blockDim.x) {
    const int t = idx / d, v = idx - t * d;
    float y = 0.0f;
    for (int c = 0; c < d; ++c) y = fmaf(float(cd[size_t(v) * d + c]), zs[t * dp + c], y);
    xs[t * dp + v] = y;
  }
  __syncthreads();
  // U = C_Tb y, energy and log terms
  double lpart = 0.0;
  for (int idx = threadIdx.x; idx < Tb * d; idx += blockDim.x) {
    const int u = idx / d, v = idx - u * d;
    float U = 0.0f;
    for (int t = 0; t < Tb; ++t) U = fmaf(ct[u * Tb + t], xs[t * dp + v], U);
    atomicAdd(acc + (size_t(l) * Tb + u) * d + v, double(U) * double(U));
    lpart += double(logf(1.0f + fabsf(U) * inv_tau));
  }
  red[threadIdx.x] = lpart;
  __syncthreads();
  for (int o = 128; o > 0; o >>= 1) {
    if (int(threadIdx.x) < o) red[threadIdx.x] += red[threadIdx.x + o];
    __syncthreads();
  }
  if (threadIdx.x == 0) atomicAdd(lsum + l, red[0]);
}

// One workgroup per layer: the statistics from the accumulated energy map and log sum; the
// map is copied out when `energy` is given.
__global__ __launch_bounds__(256) void spec_final(const double* acc, const double* lsum, int Tb, int d,
                                                    double count, double* stats, double* energy) {
  __shared__ double r0[256], r1[256];
  const int l = blockIdx.x;
  const double* al = acc + size_t(l) * Tb * d;
  double e = 0.0, er = 0.0;
  for (int idx = threadIdx.x; idx < Tb * d; idx += blockDim.x) {
    const int u = idx / d, v = idx - u * d;
    const double fu = double(u) / (Tb - 1), fv = double(v) / (d - 1);
    const double rho = sqrt(fu * fu + fv * fv) / sqrt(2.0);
    e += al[idx];
    er += al[idx] * rho;
    if (energy) energy[size_t(l) * Tb * d + idx] = al[idx];
  }
  r0[threadIdx.x] = e;
  r1[threadIdx.x] = er;
  __syncthreads();
  for (int o = 128; o > 0; o >>= 1) {
    if (int(threadIdx.x) < o) {
      r0[threadIdx.x] += r0[threadIdx.x + o];
      r1[threadIdx.x] += r1[threadIdx.x + o];
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    const double lf = r1[0] / (r0[0] + 1e-12);
    stats[4 * l + 0] = lf;
    stats[4 * l + 1] = count > 0 ? lsum[l] / count : 0.0;
    stats[4 * l + 2] = 1.0 - lf;
    stats[4 * l + 3] = r0[0];
  }
}

int cu_count_spec() {
  static int cus = 0;
  if (!cus) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
      cus = 256;
  }
  return cus;
}

}  // namespace

SpecLayout spec_layout(const cg_gauge_shape& s, int Tb) {
  SpecLayout o;
  size_t off = 0;
  o.off_acc = off;
  off = align256(off + size_t(s.L) * Tb * s.d * 8);
  o.off_lsum = off;
  off = align256(off + size_t(s.L) * 8);
  o.off_cd = off;
  off = align256(off + size_t(s.d) * s.d * 8);
  for (int p = 0; p < 2; ++p) {
    o.off_m[p] = off;
    off = align256(off + (s.d == kD ? size_t(s.L) * s.H * kD * kD * 2 : 0));
  }
  o.total = off;
  return o;
}

hipError_t launch_spectral(int s, const ViewDev& X, const GaugeDev& G, int Tb, float tau, void* ws, double* stats,
                           double* energy, bool force_generic, hipStream_t st) {
  const cg_gauge_shape shp{X.L, X.H, X.d, G.g};
  const SpecLayout lay = spec_layout(shp, Tb);
  char* base = static_cast<char*>(ws);
  double* acc = reinterpret_cast<double*>(base + lay.off_acc);
  double* lsum = reinterpret_cast<double*>(base + lay.off_lsum);
  double* cd = reinterpret_cast<double*>(base + lay.off_cd);
  const size_t nacc = size_t(X.L) * Tb * X.d;
  const size_t ninit = std::max(nacc, size_t(X.d) * X.d);
  hipLaunchKernelGGL(spec_init, dim3((ninit + 255) / 256), dim3(256), 0, st, acc, nacc, lsum, X.L, cd, X.d);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int nblk = X.T / Tb;
  const float inv_tau = 1.0f / tau;
  if (nblk > 0) {
    if (!force_generic && X.bf16 && X.d == kD && Tb == kSpecTb) {
      uint16_t* m0 = reinterpret_cast<uint16_t*>(base + lay.off_m[0]);
      uint16_t* m1 = reinterpret_cast<uint16_t*>(base + lay.off_m[1]);
      hipLaunchKernelGGL(spec_mprep, dim3(X.L * X.H), dim3(kMprepThreads), 0, st, s, G, X.H, cd, m0, m1);
      if ((e = hipGetLastError()) != hipSuccess) return e;
      SpecArgs a{};
      a.x = static_cast<const char*>(X.ptr);
      a.sl = X.sl; a.sb = X.sb; a.sh = X.sh; a.st = X.st;
      a.L = X.L; a.B = X.B; a.H = X.H;
      a.m0 = m0; a.m1 = m1;
      a.acc = acc; a.lsum = lsum;
      a.inv_tau = inv_tau;
      a.nblk = nblk;
      // work split as for the codec kernels: as many workgroups as fit at once
      const int ntiles = (nblk * kSpecTb + kTok - 1) / kTok;
      int occ = 0;
      if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&occ, (const void*)spec_mfma, kThreads, 0) != hipSuccess || occ < 1)
        occ = 2;
      a.nslices = X.L * X.B * X.H;
      int chunks = (occ * cu_count_spec() + a.nslices - 1) / a.nslices;
      chunks = std::min(std::max(chunks, 1), ntiles);
      a.tiles_per_wg = (ntiles + chunks - 1) / chunks;
      // CG_TILES_PER_WG=k fixes the tiles per workgroup, as for the codec kernels, so that small
      // inputs run the multi-tile loop (the software pipeline, the periodic fold of the binary32
      // energy partials) that the resident grid only reaches on large ones
      if (const char* f = getenv("CG_TILES_PER_WG")) {
        const long k = strtol(f, nullptr, 10);
        if (k > 0 && k < (1 << 20)) a.tiles_per_wg = int(std::min<long>(k, std::max(ntiles, 1)));
      }
      a.chunks = (ntiles + a.tiles_per_wg - 1) / a.tiles_per_wg;
      const int nwg = ((a.nslices * a.chunks + 7) / 8) * 8;
      void* args[] = {&a};
      e = hipLaunchKernel((const void*)spec_mfma, dim3(nwg), dim3(kThreads), args, 0, st);
    } else {
      const size_t smem = (size_t(2) * Tb * (X.d + 1) + size_t(Tb) * Tb) * sizeof(float);
      if (smem > 65536 &&
          (e = hipFuncSetAttribute((const void*)spec_generic, hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem)) !=
              hipSuccess)
        return e;
      hipLaunchKernelGGL(spec_generic, dim3(X.L * X.B * X.H, nblk), dim3(256), smem, st, s, X, G, Tb, inv_tau, cd, acc,
                         lsum);
      e = hipGetLastError();
    }
    if (e != hipSuccess) return e;
  }
  const double count = double(X.B) * X.H * nblk * Tb * X.d;
  hipLaunchKernelGGL(spec_final, dim3(X.L), dim3(256), 0, st, acc, lsum, Tb, X.d, count, stats, energy);
  return hipGetLastError();
}

}  // namespace cg
