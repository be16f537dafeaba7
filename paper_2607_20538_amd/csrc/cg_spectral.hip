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
// tile's tokens.  The lane holding token n keeps 16 consecutive frequencies v; the 16 tokens
// of a block are the 16 lanes of one DPP row, and the lane at place u of its row produces
// token frequency u.  The DCT's symmetry C[u][15 - t] = (-1)^u C[u][t] halves the work: each
// lane j first forms w_j = y_j + (-1)^j y_{15-j} (row_mirror), and since the even rotations of
// a row keep lane parity and meet each pair (t, 15 - t) once, U[u] is 8 multiply-adds of
// w rotated by 0, 2, .., 14 lanes (row_ror) with per-lane coefficients.  Energies accumulate
// per lane in binary64 and leave by atomic adds at the end of the workgroup.
//
// General path (any supported d and g, bf16 or binary32 input, Tb in {2, 4, 8, 16, 32}): one
// workgroup per block, gauge, channel DCT and token DCT on the VALU in binary32 through LDS.
#include <algorithm>
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
// workgroup per (l, h) stages C_d and the gauge blocks in LDS; thread t accumulates the 8 x 8
// outputs rows 8 (t / 16) .., columns 8 (t % 16) .. (one gauge group: 8 | g).
__global__ __launch_bounds__(256) void spec_mprep(int s, GaugeDev G, int H, const double* cd, uint16_t* m0,
                                                   uint16_t* m1) {
  __shared__ float cds[kD * kD];   // C_d rows
  __shared__ float gs[kD * kD];    // gs[a_global][j]: G_{r}[a][j - r g] for j in group r, a = a_global - r g
  const int lh = blockIdx.x, l = lh / H, h = lh - l * H;
  const int g = G.g;
  for (int idx = threadIdx.x; idx < kD * kD; idx += blockDim.x) {
    cds[idx] = float(cd[idx]);
    const int ag = idx / kD, j = idx - ag * kD, r = j / g;
    const int a = ag - r * g;
    float v = 0.0f;
    if (a >= 0 && a < g) v = G.f32[((((size_t(l) * 2 + s) * G.H + h) * G.R + r) * g + a) * g + (j - r * g)];
    gs[idx] = v;
  }
  __syncthreads();
  const int i0 = 8 * (threadIdx.x / 16), j0 = 8 * (threadIdx.x % 16), r = j0 / g;
  double acc[8][8];
#pragma unroll
  for (int p = 0; p < 8; ++p)
#pragma unroll
    for (int q = 0; q < 8; ++q) acc[p][q] = 0.0;
  for (int a = r * g; a < r * g + g; ++a) {
    double cv[8], gv[8];
#pragma unroll
    for (int p = 0; p < 8; ++p) cv[p] = double(cds[(i0 + p) * kD + a]);
#pragma unroll
    for (int q = 0; q < 8; ++q) gv[q] = double(gs[a * kD + j0 + q]);
#pragma unroll
    for (int p = 0; p < 8; ++p)
#pragma unroll
      for (int q = 0; q < 8; ++q) acc[p][q] = fma(cv[p], gv[q], acc[p][q]);
  }
#pragma unroll
  for (int p = 0; p < 8; ++p)
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const float v = float(acc[p][q]);
      const uint32_t hi = f32_to_bf16_rne(v);
      const uint32_t lo = f32_to_bf16_rne(v - __uint_as_float(hi << 16));
      const size_t off = (size_t(lh) * kD + i0 + p) * kD + j0 + q;
      m0[off] = uint16_t(hi);
      m1[off] = uint16_t(lo);
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

// rotation of a value by K lanes within its DPP row (K = 0: the value itself)
template <int K>
__device__ __forceinline__ float ror16(float v) {
  if constexpr (K == 0) return v;
  else return dpp_mov<0x120 + K>(v);
}
template <int K>
__device__ __forceinline__ int ror16_i(int v) {
  if constexpr (K == 0) return v;
  else return dpp_mov_i<0x120 + K>(v);
}

// U[u] of the lane at place u of its row from the row's w values (rotations by 2K lanes)
template <int... K>
__device__ __forceinline__ float row_dct(float w, const float (&coef)[8], std::integer_sequence<int, K...>) {
  float u = 0.0f;
  ((u = fmaf(coef[K], ror16<2 * K>(w), u)), ...);
  return u;
}

template <int... K>
__device__ __forceinline__ void row_sources(int i, int (&src)[8], std::integer_sequence<int, K...>) {
  ((src[K] = ror16_i<2 * K>(i)), ...);
}

__global__ __launch_bounds__(kThreads, 3) void spec_mfma(SpecArgs a) {
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
  // token DCT: the lane at place i of its row produces frequency u = i; the w value rotated in
  // from lane j = src[k] stands for token t = min(j, 15 - j), with the sign (-1)^u when j >= 8
  // (w_j then holds (-1)^u times the pair sum of token 15 - j)
  const int i = lane & 15;
  int src[8];
  row_sources(i, src, std::make_integer_sequence<int, 8>());
  float coef[8];
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    const int j = src[k], t = j < 8 ? j : 15 - j;
    const double sg = (j >= 8 && (i & 1)) ? -1.0 : 1.0;
    coef[k] = float(sg * sqrt((i == 0 ? 1.0 : 2.0) / kSpecTb) * cospi((2.0 * t + 1.0) * i / (2.0 * kSpecTb)));
  }
  const float par = (i & 1) ? -1.0f : 1.0f;  // (-1)^j of this lane

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

  double eacc[16];
#pragma unroll
  for (int e = 0; e < 16; ++e) eacc[e] = 0.0;
  double lacc = 0.0;
  for (int t = tb; t < min(te, tb + kSpecStages - 1); ++t) issue(t);
  for (int t = tb; t < te; ++t) {
    // tile t landed in every wave, every wave is done with the buffer tile t - 1 used
    wait_tile(min(te - 1, t + kSpecStages - 2) - t);
    __builtin_amdgcn_s_barrier();
    if (t + kSpecStages - 1 < te) issue(t + kSpecStages - 1);
    const uint8_t* src_t = xtile[(t - tb) % kSpecStages];
    f32x16_t acc = {};
#pragma unroll
    for (int kk = 0; kk < 8; ++kk) {
      const bf16x8_t bv = as_bf16x8(*(const u32x4_t*)(src_t + boff[kk]));
      acc = mfma(A[1][kk], bv, acc);
      acc = mfma(A[0][kk], bv, acc);
    }
    // token DCT of the lane's 16 frequencies v = 32w + 16hc + e over its row's block
    const bool valid = 2 * t + (n >> 4) < a.nblk;
    float ls = 0.0f;
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const float y = acc[e];
      const float w = fmaf(par, dpp_mov<0x140>(y), y);  // row_mirror: y of lane 15 - j
      const float u = row_dct(w, coef, std::make_integer_sequence<int, 8>());
      if (valid) {
        eacc[e] = fma(double(u), double(u), eacc[e]);
        ls += __logf(1.0f + fabsf(u) * a.inv_tau);
      }
    }
    lacc += double(ls);
  }
  // energy map entries (u = i, v = 32w + 16hc + e) and the log sum
  double* accl = a.acc + size_t(l) * kSpecTb * kD + size_t(i) * kD + 32 * w + 16 * hc;
#pragma unroll
  for (int e = 0; e < 16; ++e) atomicAdd(accl + e, eacc[e]);
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) lacc += __shfl_xor(lacc, off);
  if (lane == 0) atomicAdd(a.lsum + l, lacc);
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
      hipLaunchKernelGGL(spec_mprep, dim3(X.L * X.H), dim3(256), 0, st, s, G, X.H, cd, m0, m1);
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
