// Host side of the C ABI: argument validation, gauge construction (gauge_make), buffer
// sizing and dispatch of the encode / decode / rolling-append kernels.
#include <math.h>
#include <climits>
#include <algorithm>
#include <stdlib.h>
#include <string.h>

#include <atomic>
#include <thread>
#include <vector>

#include "cg_internal.h"

using namespace cg;

namespace {

// ------------------------------------------------------------------------------------------
// gauge construction on the host, binary64
// ------------------------------------------------------------------------------------------

// Philox4x32-10 block function (Salmon et al., SC 2011).
void philox4x32_10(uint32_t c[4], uint32_t k0, uint32_t k1) {
  const uint32_t M0 = 0xD2511F53u, M1 = 0xCD9E8D57u, W0 = 0x9E3779B9u, W1 = 0xBB67AE85u;
  for (int i = 0; i < 10; ++i) {
    const uint64_t a = uint64_t(M0) * c[0], b = uint64_t(M1) * c[2];
    const uint32_t x0 = uint32_t(b >> 32) ^ c[1] ^ k0;
    const uint32_t x2 = uint32_t(a >> 32) ^ c[3] ^ k1;
    c[1] = uint32_t(b);
    c[3] = uint32_t(a);
    c[0] = x0;
    c[2] = x2;
    k0 += W0;
    k1 += W1;
  }
}

// g*g standard normals of stream `index`: counter (block, 0, index_lo, index_hi), key = seed;
// each Philox output (w0..w3) yields two Box-Muller pairs (w0, w1), (w2, w3) with
// u1 = (w + 1) 2^-32, u2 = w 2^-32, giving r cos(2 pi u2), r sin(2 pi u2).
void normals(uint64_t seed, uint64_t index, size_t count, double* out) {
  const double two32 = 4294967296.0;
  for (size_t blk = 0; blk * 4 < count; ++blk) {
    uint32_t c[4] = {uint32_t(blk), 0u, uint32_t(index), uint32_t(index >> 32)};
    philox4x32_10(c, uint32_t(seed), uint32_t(seed >> 32));
    for (int pr = 0; pr < 2; ++pr) {
      const double u1 = (double(c[2 * pr]) + 1.0) / two32;
      const double u2 = double(c[2 * pr + 1]) / two32;
      const double rad = sqrt(-2.0 * log(u1)), th = 2.0 * M_PI * u2;
      const size_t k = blk * 4 + 2 * pr;
      if (k < count) out[k] = rad * cos(th);
      if (k + 1 < count) out[k + 1] = rad * sin(th);
    }
  }
}

// Haar orthogonal matrix: Householder QR of the normal matrix M (row-major, M[i][j] = normal
// i*g + j), Q accumulated explicitly, columns multiplied by sign(R_jj) (Mezzadri 2007).
void haar(int g, uint64_t seed, uint64_t index, double* Q) {
  std::vector<double> A(size_t(g) * g), V(size_t(g) * g, 0.0), diag(g);
  normals(seed, index, A.size(), A.data());
  for (int k = 0; k < g; ++k) {
    double nrm = 0.0;
    for (int i = k; i < g; ++i) nrm += A[i * g + k] * A[i * g + k];
    nrm = sqrt(nrm);
    const double alpha = A[k * g + k] > 0 ? -nrm : nrm;  // R_kk
    double* v = &V[size_t(k) * g];
    for (int i = 0; i < g; ++i) v[i] = i < k ? 0.0 : A[i * g + k];
    v[k] -= alpha;
    double vv = 0.0;
    for (int i = k; i < g; ++i) vv += v[i] * v[i];
    diag[k] = alpha;
    if (vv == 0.0) continue;
    for (int j = k; j < g; ++j) {  // A <- (I - 2 v v^T / v^T v) A
      double dot = 0.0;
      for (int i = k; i < g; ++i) dot += v[i] * A[i * g + j];
      const double f = 2.0 * dot / vv;
      for (int i = k; i < g; ++i) A[i * g + j] -= f * v[i];
    }
  }
  // Q = H_0 H_1 ... H_{g-1} applied to the identity, right to left
  for (int i = 0; i < g; ++i)
    for (int j = 0; j < g; ++j) Q[i * g + j] = i == j ? 1.0 : 0.0;
  for (int k = g - 1; k >= 0; --k) {
    const double* v = &V[size_t(k) * g];
    double vv = 0.0;
    for (int i = k; i < g; ++i) vv += v[i] * v[i];
    if (vv == 0.0) continue;
    for (int j = 0; j < g; ++j) {
      double dot = 0.0;
      for (int i = k; i < g; ++i) dot += v[i] * Q[i * g + j];
      const double f = 2.0 * dot / vv;
      for (int i = k; i < g; ++i) Q[i * g + j] -= f * v[i];
    }
  }
  for (int j = 0; j < g; ++j)
    if (diag[j] < 0)
      for (int i = 0; i < g; ++i) Q[i * g + j] = -Q[i * g + j];
}

void dct2(int g, double* Q) {
  for (int k = 0; k < g; ++k) {
    const double a = k == 0 ? sqrt(1.0 / g) : sqrt(2.0 / g);
    for (int n = 0; n < g; ++n) Q[k * g + n] = a * cos(M_PI * (n + 0.5) * k / g);
  }
}

// Sylvester construction: H_1 = [1], H_2m = [[H_m, H_m], [H_m, -H_m]], normalised by sqrt(g).
void hadamard(int g, double* Q) {
  Q[0] = 1.0;
  for (int m = 1; m < g; m *= 2)
    for (int i = 0; i < m; ++i)
      for (int j = 0; j < m; ++j) {
        const double v = Q[i * g + j];
        Q[i * g + j + m] = v;
        Q[(i + m) * g + j] = v;
        Q[(i + m) * g + j + m] = -v;
      }
  const double s = 1.0 / sqrt(double(g));
  for (size_t k = 0; k < size_t(g) * g; ++k) Q[k] *= s;
}

// C = A B (row-major g x g); each C[i][j] sums its products in increasing k, the loops run
// along rows of B and C
void matmul(int g, const double* A, const double* B, double* C) {
  for (int i = 0; i < g; ++i) {
    double* c = C + size_t(i) * g;
    for (int j = 0; j < g; ++j) c[j] = 0.0;
    for (int k = 0; k < g; ++k) {
      const double a = A[size_t(i) * g + k];
      const double* b = B + size_t(k) * g;
      for (int j = 0; j < g; ++j) c[j] += a * b[j];
    }
  }
}

// exp(A - A^T) by scaling and squaring with the diagonal Pade(8,8) approximant; the
// denominator system is solved by Gaussian elimination with partial pivoting.
void expm_skew(int g, const float* A, double* Q) {
  const size_t gg = size_t(g) * g;
  std::vector<double> S(gg), P(gg), N(gg), D(gg), T(gg), T2(gg);
  double nrm = 0.0;
  for (int i = 0; i < g; ++i) {
    double row = 0.0;
    for (int j = 0; j < g; ++j) {
      S[i * g + j] = double(A[i * g + j]) - double(A[j * g + i]);
      row += fabs(S[i * g + j]);
    }
    nrm = row > nrm ? row : nrm;
  }
  int sq = 0;
  while (nrm > 0.25) {
    nrm *= 0.5;
    ++sq;
  }
  for (auto& v : S) v = ldexp(v, -sq);
  // Pade(8,8) coefficients c_k = (16-k)! 8! / (16! k! (8-k)!)
  double c[9];
  c[0] = 1.0;
  for (int k = 1; k <= 8; ++k) c[k] = c[k - 1] * double(8 - k + 1) / double(k * (16 - k + 1));
  for (size_t i = 0; i < gg; ++i) {
    N[i] = 0.0;
    D[i] = 0.0;
    P[i] = (i / g == i % g) ? 1.0 : 0.0;  // S^0
  }
  for (int k = 0; k <= 8; ++k) {
    const double sgn = (k & 1) ? -1.0 : 1.0;
    for (size_t i = 0; i < gg; ++i) {
      N[i] += c[k] * P[i];
      D[i] += sgn * c[k] * P[i];
    }
    matmul(g, P.data(), S.data(), T.data());
    P.swap(T);
  }
  // solve D Q = N
  std::vector<double> Mx(D), R(N);
  for (int col = 0; col < g; ++col) {
    int piv = col;
    for (int i = col + 1; i < g; ++i)
      if (fabs(Mx[i * g + col]) > fabs(Mx[piv * g + col])) piv = i;
    if (piv != col)
      for (int j = 0; j < g; ++j) {
        std::swap(Mx[col * g + j], Mx[piv * g + j]);
        std::swap(R[col * g + j], R[piv * g + j]);
      }
    for (int i = col + 1; i < g; ++i) {
      const double f = Mx[i * g + col] / Mx[col * g + col];
      if (f == 0.0) continue;
      for (int j = col; j < g; ++j) Mx[i * g + j] -= f * Mx[col * g + j];
      for (int j = 0; j < g; ++j) R[i * g + j] -= f * R[col * g + j];
    }
  }
  for (int i = g - 1; i >= 0; --i)
    for (int j = 0; j < g; ++j) {
      double acc = R[i * g + j];
      for (int k = i + 1; k < g; ++k) acc -= Mx[i * g + k] * Q[k * g + j];
      Q[i * g + j] = acc / Mx[i * g + i];
    }
  for (int s = 0; s < sq; ++s) {
    matmul(g, Q, Q, T2.data());
    memcpy(Q, T2.data(), gg * sizeof(double));
  }
}

double orth_error(int g, const float* G) {
  double worst = 0.0;
  for (int i = 0; i < g; ++i)
    for (int j = 0; j < g; ++j) {
      double acc = 0.0;
      for (int k = 0; k < g; ++k) acc += double(G[i * g + k]) * double(G[j * g + k]);
      const double e = fabs(acc - (i == j ? 1.0 : 0.0));
      worst = e > worst ? e : worst;
    }
  return worst;
}

uint16_t bf16_rne(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  u += 0x7fffu + ((u >> 16) & 1u);
  return uint16_t(u >> 16);
}
float bf16_val(uint16_t h) {
  const uint32_t u = uint32_t(h) << 16;
  float f;
  memcpy(&f, &u, 4);
  return f;
}

// ------------------------------------------------------------------------------------------
// validation helpers
// ------------------------------------------------------------------------------------------

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

bool bits_ok(int b) { return b == 2 || b == 3 || b == 4 || b == 6 || b == 8; }

int32_t check_shape(const cg_gauge_shape& s) {
  if (s.L <= 0 || s.H <= 0 || s.d <= 0 || s.g <= 0) return CG_ERR_ARG;
  if (s.d % s.g || s.d > 256 || s.d % 8) return CG_ERR_UNSUPPORTED;
  return CG_OK;
}

int32_t check_codec(const cg_codec* c, int d) {
  if (!c) return CG_ERR_ARG;
  switch (c->backend) {
    case CG_BACKEND_PASSTHROUGH:
      return CG_OK;
    case CG_BACKEND_BLOCK_UNIFORM:
      if (!bits_ok(c->bits) || c->block_c <= 0) return CG_ERR_UNSUPPORTED;
      if (d % c->block_c || (c->block_c * c->bits) % 32 || c->block_c > 256) return CG_ERR_UNSUPPORTED;
      if (c->block_t < 1 || c->block_t > 32 || (c->block_t & (c->block_t - 1))) return CG_ERR_UNSUPPORTED;
      return CG_OK;
    case CG_BACKEND_ZFP:
      return bits_ok(c->bits) && d % 4 == 0 ? CG_OK : CG_ERR_UNSUPPORTED;
    case CG_BACKEND_KIVI:
      if (!bits_ok(c->bits)) return CG_ERR_UNSUPPORTED;
      if (c->key_tokens != 16 && c->key_tokens != 32 && c->key_tokens != 64) return CG_ERR_UNSUPPORTED;
      if ((c->key_tokens * c->bits) % 32) return CG_ERR_UNSUPPORTED;
      if (c->val_channels <= 0 || d % c->val_channels || (c->val_channels * c->bits) % 32) return CG_ERR_UNSUPPORTED;
      if (c->residual < 0) return CG_ERR_ARG;
      return CG_OK;
    default:
      return CG_ERR_ARG;
  }
}

int32_t check_view(const cg_kv_view* v, const cg_gauge_shape& s, int L) {
  if (!v || (!v->ptr && v->T != 0)) return CG_ERR_ARG;  // an empty view touches no memory
  if (v->dtype != CG_DTYPE_BF16 && v->dtype != CG_DTYPE_F32) return CG_ERR_ARG;
  if (v->L != L || v->H != s.H || v->d != s.d || v->B <= 0 || v->T < 0) return CG_ERR_SHAPE;
  if (!aligned16(v->ptr)) return CG_ERR_ALIGN;
  const int64_t unit = v->dtype == CG_DTYPE_BF16 ? 8 : 4;  // elements per 16 bytes
  if (v->stride_l % unit || v->stride_b % unit || v->stride_h % unit || v->stride_t % unit) return CG_ERR_ALIGN;
  if (v->stride_l < 0 || v->stride_b < 0 || v->stride_h < 0 || v->stride_t < 0) return CG_ERR_ARG;
  return CG_OK;
}

int32_t check_cache(const cg_cache* k, const cg_codec* c, const cg_gauge_shape& s, int B) {
  if (!k || !k->codes) return CG_ERR_ARG;
  if (k->L != s.L || k->H != s.H || k->d != s.d || k->B != B || k->T_cap <= 0) return CG_ERR_SHAPE;
  if (!aligned16(k->codes)) return CG_ERR_ALIGN;
  if (c->backend != CG_BACKEND_PASSTHROUGH && c->backend != CG_BACKEND_ZFP && (!k->side || !aligned16(k->side)))
    return CG_ERR_ARG;
  if (c->backend == CG_BACKEND_ZFP && k->T_cap % 4) return CG_ERR_SHAPE;
  if (c->backend == CG_BACKEND_KIVI) {
    if (!k->residual || !aligned16(k->residual)) return CG_ERR_ARG;
    if (k->T_cap % c->key_tokens) return CG_ERR_SHAPE;
  }
  if (c->backend == CG_BACKEND_BLOCK_UNIFORM && c->block_t > 1) {
    if (!k->residual || !aligned16(k->residual)) return CG_ERR_ARG;
    if (k->T_cap % c->block_t) return CG_ERR_SHAPE;
  }
  return CG_OK;
}

GaugeDev gauge_dev(const void* G_dev, const cg_gauge_shape& s) {
  const GaugeLayout gl = gauge_layout(s);
  const char* base = static_cast<const char*>(G_dev);
  GaugeDev G;
  G.f32 = reinterpret_cast<const float*>(base + gl.off_f32);
  for (int p = 0; p < 3; ++p) {
    G.hi[p] = reinterpret_cast<const uint16_t*>(base + gl.off_hi[p]);
    G.tr[p] = reinterpret_cast<const uint16_t*>(base + gl.off_tr[p]);
  }
  G.cs8 = reinterpret_cast<const float*>(base + gl.off_cs8);
  G.g = s.g;
  G.R = s.d / s.g;
  G.H = s.H;
  return G;
}

CodecDev codec_dev(const cg_codec* c) {
  CodecDev d;
  d.backend = c->backend;
  d.bits = c->bits;
  d.n = c->block_c;
  d.kg = c->key_tokens;
  d.kvc = c->val_channels;
  d.win = c->residual;
  d.bt = c->backend == CG_BACKEND_BLOCK_UNIFORM ? c->block_t : 1;
  return d;
}

ViewDev view_dev(const cg_kv_view* v) {
  ViewDev d;
  d.ptr = v->ptr;
  d.sl = v->stride_l;
  d.sb = v->stride_b;
  d.sh = v->stride_h;
  d.st = v->stride_t;
  d.L = v->L;
  d.B = v->B;
  d.H = v->H;
  d.T = v->T;
  d.d = v->d;
  d.bf16 = v->dtype == CG_DTYPE_BF16;
  return d;
}

CacheDev cache_dev(const cg_cache* k) {
  CacheDev d;
  d.codes = static_cast<uint8_t*>(k->codes);
  d.side = static_cast<uint32_t*>(k->side);
  d.ring = static_cast<uint16_t*>(k->residual);
  d.L = k->L;
  d.B = k->B;
  d.H = k->H;
  d.T_cap = k->T_cap;
  d.d = k->d;
  return d;
}

// A query or output view of kv_attend: [nl][B][Hq][1][d], Hq a multiple of the KV heads.
int32_t check_qview(const cg_kv_view* v, const cg_gauge_shape& s, int L) {
  if (!v || !v->ptr) return CG_ERR_ARG;
  if (v->dtype != CG_DTYPE_BF16 && v->dtype != CG_DTYPE_F32) return CG_ERR_ARG;
  if (v->L != L || v->d != s.d || v->B <= 0 || v->T != 1 || v->H < s.H || v->H % s.H) return CG_ERR_SHAPE;
  if (!aligned16(v->ptr)) return CG_ERR_ALIGN;
  const int64_t unit = v->dtype == CG_DTYPE_BF16 ? 8 : 4;
  if (v->stride_l % unit || v->stride_b % unit || v->stride_h % unit || v->stride_t % unit) return CG_ERR_ALIGN;
  if (v->stride_l < 0 || v->stride_b < 0 || v->stride_h < 0 || v->stride_t < 0) return CG_ERR_ARG;
  return CG_OK;
}

int kivi_tq(int T, const cg_codec* c) {
  return T < c->residual ? 0 : ((T - c->residual) / c->key_tokens) * c->key_tokens;
}

}  // namespace

namespace cg {

// Matrix-core kernels take bf16 block-uniform (and passthrough) caches of head dimension 128;
// everything else runs on the general kernels.  The environment variable CG_KERNELS=generic,
// read at every launch, forces the general kernels (the tests run both paths on one input).
static bool force_generic() {
  const char* e = getenv("CG_KERNELS");
  return e && strcmp(e, "generic") == 0;
}

hipError_t launch_encode(int s, const ViewDev& X, int l0, const GaugeDev& G, const CodecDev& c, const CacheDev& k,
                         int t0, int tq, int* err, hipStream_t st) {
  if (!force_generic() && mfma_encode_supported(X, G, c)) return launch_encode_mfma(s, X, l0, G, c, k, t0, tq, err, st);
  return launch_encode_generic(s, X, l0, G, c, k, t0, tq, err, st);
}

hipError_t launch_decode(int s, const CacheDev& k, int l0, const GaugeDev& G, const CodecDev& c, int t0, int len,
                         const int* pos, int pos_add, const ViewDev& Y, int* err, hipStream_t st) {
  if (!force_generic() && mfma_decode_supported(s, Y, G, c))
    return launch_decode_mfma(s, k, l0, G, c, t0, len, pos, pos_add, Y, err, st);
  return launch_decode_generic(s, k, l0, G, c, t0, len, pos, pos_add, Y, err, st);
}

}  // namespace cg

// ------------------------------------------------------------------------------------------
// C ABI
// ------------------------------------------------------------------------------------------

extern "C" {

const char* cg_status_str(int32_t status) {
  switch (status) {
    case CG_OK: return "ok";
    case CG_ERR_ARG: return "invalid argument";
    case CG_ERR_SHAPE: return "shape mismatch";
    case CG_ERR_ALIGN: return "misaligned pointer or stride";
    case CG_ERR_UNSUPPORTED: return "unsupported configuration";
    case CG_ERR_NOT_ORTHOGONAL: return "gauge is not orthogonal";
    case CG_ERR_CAPACITY: return "token range exceeds cache capacity";
    case CG_ERR_DEVICE: return "HIP runtime error";
    default: return "unknown status";
  }
}

size_t gauge_device_bytes(cg_gauge_shape shp) {
  if (check_shape(shp) != CG_OK) return 0;
  return gauge_layout(shp).total;
}

int32_t gauge_make(int32_t kind, cg_gauge_shape shp, uint64_t seed, const float* params, float* G_host, void* G_dev,
                   void* stream) {
  int32_t rc = check_shape(shp);
  if (rc != CG_OK) return rc;
  if (!G_host && !G_dev) return CG_ERR_ARG;
  if (kind < CG_GAUGE_IDENTITY || kind > CG_GAUGE_USER) return CG_ERR_ARG;
  if ((kind == CG_GAUGE_EXPM || kind == CG_GAUGE_USER) && !params) return CG_ERR_ARG;
  const int g = shp.g, R = shp.d / shp.g;
  if (kind == CG_GAUGE_HADAMARD && (g & (g - 1))) return CG_ERR_UNSUPPORTED;
  if (G_dev && !aligned16(G_dev)) return CG_ERR_ALIGN;
  const GaugeLayout gl = gauge_layout(shp);
  const size_t gg = size_t(g) * g;
  std::vector<float> G32(gl.nblk * gg);
  std::atomic<bool> not_orth{false};
  // blocks [b0, b1): each block depends only on its own index and parameters
  auto blocks = [&](int64_t b0, int64_t b1) {
    std::vector<double> Q(gg);
    for (int64_t blk = b0; blk < b1; ++blk) {
      switch (kind) {
        case CG_GAUGE_IDENTITY:
          for (size_t i = 0; i < gg; ++i) Q[i] = (i / g == i % g) ? 1.0 : 0.0;
          break;
        case CG_GAUGE_HAAR: haar(g, seed, uint64_t(blk), Q.data()); break;
        case CG_GAUGE_DCT2: dct2(g, Q.data()); break;
        case CG_GAUGE_HADAMARD: hadamard(g, Q.data()); break;
        case CG_GAUGE_EXPM: expm_skew(g, params + blk * gg, Q.data()); break;
        case CG_GAUGE_USER:
          for (size_t i = 0; i < gg; ++i) Q[i] = params[blk * gg + i];
          break;
      }
      float* out = &G32[blk * gg];
      for (size_t i = 0; i < gg; ++i) out[i] = float(Q[i]);
      if (kind == CG_GAUGE_USER && orth_error(g, out) > 1e-5) not_orth = true;
    }
  };
  // the exponential of a wide block costs O(g^3) per block: spread the blocks over host threads
  // (at most 16; the serial loop when threads cannot be started)
  int nth = 1;
  if (kind == CG_GAUGE_EXPM && g >= 32)
    nth = int(std::min<int64_t>(gl.nblk, std::max(1u, std::min(16u, std::thread::hardware_concurrency()))));
  bool serial = nth <= 1;
  if (!serial) {
    try {
      std::vector<std::thread> pool;
      const int64_t per = (gl.nblk + nth - 1) / nth;
      for (int t = 0; t < nth; ++t) {
        const int64_t b0 = t * per, b1 = std::min<int64_t>(gl.nblk, b0 + per);
        if (b0 < b1) pool.emplace_back(blocks, b0, b1);
      }
      for (auto& th : pool) th.join();
    } catch (...) {
      serial = true;
    }
  }
  if (serial) blocks(0, gl.nblk);
  if (not_orth) return CG_ERR_NOT_ORTHOGONAL;
  (void)R;
  if (G_host) memcpy(G_host, G32.data(), G32.size() * sizeof(float));
  if (G_dev) {
    std::vector<unsigned char> buf(gl.total, 0);
    memcpy(buf.data() + gl.off_f32, G32.data(), G32.size() * sizeof(float));
    for (int64_t blk = 0; blk < gl.nblk; ++blk) {
      const float* src = &G32[blk * gg];
      for (int i = 0; i < g; ++i)
        for (int j = 0; j < g; ++j) {
          // split G[i][j] into three bf16 terms, and the transposed block likewise
          float rem = src[i * g + j];
          for (int p = 0; p < 3; ++p) {
            const uint16_t hb = bf16_rne(rem);
            reinterpret_cast<uint16_t*>(buf.data() + gl.off_hi[p])[blk * gg + size_t(i) * g + j] = hb;
            reinterpret_cast<uint16_t*>(buf.data() + gl.off_tr[p])[blk * gg + size_t(j) * g + i] = hb;
            rem = rem - bf16_val(hb);  // exact in binary32
          }
        }
    }
    // decoder column sums per 8-channel segment (double sums of the bf16 terms: exact)
    const int d = shp.d, R = d / g;
    float* cs8 = reinterpret_cast<float*>(buf.data() + gl.off_cs8);
    for (int64_t head = 0; head < gl.nhead; ++head)
      for (int c = 0; c < d / 8; ++c)
        for (int i = 0; i < d; ++i) {
          const int r = i / g;
          double acc = 0.0;
          if ((8 * c) / g == r) {
            const int64_t blk = head * R + r;
            for (int j = 8 * c; j < 8 * c + 8; ++j)
              for (int p = 0; p < kDecPlanes; ++p)
                acc += bf16_val(reinterpret_cast<const uint16_t*>(buf.data() + gl.off_tr[p])[blk * gg + size_t(i % g) * g + (j % g)]);
          }
          cs8[(size_t(head) * (d / 8) + c) * d + i] = float(acc);
        }
    hipStream_t st = static_cast<hipStream_t>(stream);
    if (hipMemcpyAsync(G_dev, buf.data(), buf.size(), hipMemcpyHostToDevice, st) != hipSuccess)
      return CG_ERR_DEVICE;
    if (hipStreamSynchronize(st) != hipSuccess) return CG_ERR_DEVICE;
  }
  return CG_OK;
}

int32_t cache_bytes(const cg_codec* codec, int32_t s, int32_t L, int32_t B, int32_t H, int32_t T_cap, int32_t d,
                    size_t* codes, size_t* side, size_t* residual) {
  if (!codec || s < 0 || s > 1 || L <= 0 || B <= 0 || H <= 0 || T_cap <= 0 || d <= 0 || d % 8) return CG_ERR_ARG;
  int32_t rc = check_codec(codec, d);
  if (rc != CG_OK) return rc;
  const size_t slices = size_t(L) * B * H;
  size_t c = 0, sd = 0, r = 0;
  const int b = codec->bits;
  switch (codec->backend) {
    case CG_BACKEND_PASSTHROUGH: c = slices * T_cap * d * 4; break;
    case CG_BACKEND_ZFP:
      if (T_cap % 4) return CG_ERR_SHAPE;
      c = slices * (T_cap / 4) * (d / 4) * size_t(2 * b);
      break;
    case CG_BACKEND_BLOCK_UNIFORM: {
      const int bt = codec->block_t;
      if (T_cap % bt) return CG_ERR_SHAPE;
      c = slices * T_cap * (size_t(d) * b / 8);
      sd = slices * (T_cap / bt) * (d / codec->block_c) * 4;
      r = bt > 1 ? slices * size_t(bt) * d * 2 : 0;
      break;
    }
    case CG_BACKEND_KIVI: {
      if (T_cap % codec->key_tokens) return CG_ERR_SHAPE;
      const int kg = codec->key_tokens;
      if (s == 0) {
        c = slices * (T_cap / kg) * d * (size_t(kg) * b / 8);
        sd = slices * (T_cap / kg) * d * 4;
      } else {
        c = slices * T_cap * (size_t(d) * b / 8);
        sd = slices * T_cap * (d / codec->val_channels) * 4;
      }
      r = slices * size_t(codec->residual + kg) * d * 2;
      break;
    }
  }
  if (codes) *codes = c;
  if (side) *side = sd;
  if (residual) *residual = r;
  return CG_OK;
}

int32_t kv_encode(int32_t s, const cg_kv_view* X, const void* G_dev, cg_gauge_shape shp, const cg_codec* codec,
                  const cg_cache* out, int32_t t0, int32_t* err_flag, void* stream) {
  int32_t rc = check_shape(shp);
  if (rc != CG_OK) return rc;
  if (s < 0 || s > 1 || !G_dev) return CG_ERR_ARG;
  if (!aligned16(G_dev)) return CG_ERR_ALIGN;
  if ((rc = check_codec(codec, shp.d)) != CG_OK) return rc;
  if ((rc = check_view(X, shp, shp.L)) != CG_OK) return rc;
  if ((rc = check_cache(out, codec, shp, X->B)) != CG_OK) return rc;
  if (t0 < 0) return CG_ERR_ARG;
  if (int64_t(t0) + X->T > out->T_cap) return CG_ERR_CAPACITY;
  int tq = 0;
  if (codec->backend == CG_BACKEND_KIVI) {
    if (t0 != 0 || X->dtype != CG_DTYPE_BF16) return CG_ERR_UNSUPPORTED;
    tq = kivi_tq(X->T, codec);
  } else if (codec->backend == CG_BACKEND_BLOCK_UNIFORM && codec->block_t > 1) {
    if (t0 % codec->block_t || X->dtype != CG_DTYPE_BF16) return CG_ERR_UNSUPPORTED;
    tq = (X->T / codec->block_t) * codec->block_t;
  } else if (codec->backend == CG_BACKEND_ZFP) {
    if (t0 % 4 || X->T % 4) return CG_ERR_UNSUPPORTED;  // whole 4-token block rows
  }
  if (err_flag && (reinterpret_cast<uintptr_t>(err_flag) & 3u)) return CG_ERR_ALIGN;
  hipError_t e = launch_encode(s, view_dev(X), 0, gauge_dev(G_dev, shp), codec_dev(codec), cache_dev(out), t0, tq,
                               err_flag, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? CG_OK : CG_ERR_DEVICE;
}

int32_t kv_decode(int32_t s, const cg_cache* in, const void* G_dev, cg_gauge_shape shp, const cg_codec* codec,
                  const int32_t* lens, int32_t t0, const cg_kv_view* Xhat, int32_t* err_flag, void* stream) {
  int32_t rc = check_shape(shp);
  if (rc != CG_OK) return rc;
  if (s < 0 || s > 1 || !G_dev) return CG_ERR_ARG;
  if (!aligned16(G_dev)) return CG_ERR_ALIGN;
  if ((rc = check_codec(codec, shp.d)) != CG_OK) return rc;
  if ((rc = check_view(Xhat, shp, shp.L)) != CG_OK) return rc;
  if ((rc = check_cache(in, codec, shp, Xhat->B)) != CG_OK) return rc;
  if (t0 < 0) return CG_ERR_ARG;
  if (int64_t(t0) + Xhat->T > in->T_cap) return CG_ERR_CAPACITY;
  if (lens && (reinterpret_cast<uintptr_t>(lens) & 3u)) return CG_ERR_ALIGN;
  const bool held = codec->backend == CG_BACKEND_KIVI || (codec->backend == CG_BACKEND_BLOCK_UNIFORM && codec->block_t > 1);
  // with device row lengths the rows bound themselves on the device; else the host length does
  if (!lens && held && (in->len < 0 || in->len > in->T_cap || int64_t(t0) + Xhat->T > in->len)) return CG_ERR_CAPACITY;
  if (codec->backend == CG_BACKEND_ZFP && (lens || t0 % 4 || Xhat->T % 4)) return CG_ERR_UNSUPPORTED;
  if (err_flag && (reinterpret_cast<uintptr_t>(err_flag) & 3u)) return CG_ERR_ALIGN;
  hipError_t e = launch_decode(s, cache_dev(in), 0, gauge_dev(G_dev, shp), codec_dev(codec), t0, in->len, lens, 0,
                               view_dev(Xhat), err_flag, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? CG_OK : CG_ERR_DEVICE;
}

int32_t kv_append_step(int32_t l0, int32_t l1, const cg_kv_view* k_new, const cg_kv_view* v_new, const int32_t* pos,
                       const void* G_dev, cg_gauge_shape shp, const cg_codec* codec, const cg_cache* kc,
                       const cg_cache* vc, const cg_kv_view* k_hist, const cg_kv_view* v_hist, int32_t* err_flag,
                       void* stream) {
  int32_t rc = check_shape(shp);
  if (rc != CG_OK) return rc;
  if (!G_dev || !pos || l0 < 0 || l1 <= l0 || l1 > shp.L) return CG_ERR_ARG;
  if (!aligned16(G_dev)) return CG_ERR_ALIGN;
  if ((reinterpret_cast<uintptr_t>(pos) & 3u)) return CG_ERR_ALIGN;
  if ((rc = check_codec(codec, shp.d)) != CG_OK) return rc;
  if (codec->backend == CG_BACKEND_ZFP) return CG_ERR_UNSUPPORTED;  // blocks span 4 tokens
  const int nl = l1 - l0;
  if ((rc = check_view(k_new, shp, nl)) != CG_OK) return rc;
  if ((rc = check_view(v_new, shp, nl)) != CG_OK) return rc;
  if (k_new->T != 1 || v_new->T != 1 || v_new->B != k_new->B) return CG_ERR_SHAPE;
  const bool staged = codec->backend == CG_BACKEND_KIVI || (codec->backend == CG_BACKEND_BLOCK_UNIFORM && codec->block_t > 1);
  if (staged && (k_new->dtype != CG_DTYPE_BF16 || v_new->dtype != CG_DTYPE_BF16)) return CG_ERR_UNSUPPORTED;
  const int B = k_new->B;
  if ((rc = check_cache(kc, codec, shp, B)) != CG_OK) return rc;
  if ((rc = check_cache(vc, codec, shp, B)) != CG_OK) return rc;
  if (k_hist && (rc = check_view(k_hist, shp, nl)) != CG_OK) return rc;
  if (v_hist && (rc = check_view(v_hist, shp, nl)) != CG_OK) return rc;
  if ((k_hist && k_hist->B != B) || (v_hist && v_hist->B != B)) return CG_ERR_SHAPE;
  if ((k_hist && k_hist->T > kc->T_cap) || (v_hist && v_hist->T > vc->T_cap)) return CG_ERR_CAPACITY;
  if (err_flag && (reinterpret_cast<uintptr_t>(err_flag) & 3u)) return CG_ERR_ALIGN;
  hipStream_t st = static_cast<hipStream_t>(stream);
  const GaugeDev G = gauge_dev(G_dev, shp);
  const CodecDev c = codec_dev(codec);
  hipError_t e = launch_append(0, view_dev(k_new), l0, pos, G, c, cache_dev(kc), err_flag, st);
  if (e == hipSuccess) e = launch_append(1, view_dev(v_new), l0, pos, G, c, cache_dev(vc), err_flag, st);
  if (e == hipSuccess && k_hist)
    e = launch_decode(0, cache_dev(kc), l0, G, c, 0, 0, pos, 1, view_dev(k_hist), err_flag, st);
  if (e == hipSuccess && v_hist)
    e = launch_decode(1, cache_dev(vc), l0, G, c, 0, 0, pos, 1, view_dev(v_hist), err_flag, st);
  return e == hipSuccess ? CG_OK : CG_ERR_DEVICE;
}

size_t spectral_workspace_bytes(cg_gauge_shape shp, int32_t block_t) {
  if (check_shape(shp) != CG_OK || block_t < 2 || block_t > 32 || (block_t & (block_t - 1))) return 0;
  return spec_layout(shp, block_t).total;
}

int32_t kv_spectral_stats(int32_t s, const cg_kv_view* X, const void* G_dev, cg_gauge_shape shp, int32_t block_t,
                          float tau, void* workspace, double* stats, double* energy, void* stream) {
  int32_t rc = check_shape(shp);
  if (rc != CG_OK) return rc;
  if (s < 0 || s > 1 || !G_dev || !workspace || !stats) return CG_ERR_ARG;
  if (block_t < 2 || block_t > 32 || (block_t & (block_t - 1))) return CG_ERR_UNSUPPORTED;
  if (!(tau > 0.0f) || !isfinite(tau)) return CG_ERR_ARG;
  if (!aligned16(G_dev) || !aligned16(workspace) || (reinterpret_cast<uintptr_t>(stats) & 7u) ||
      (reinterpret_cast<uintptr_t>(energy) & 7u))
    return CG_ERR_ALIGN;
  if ((rc = check_view(X, shp, shp.L)) != CG_OK) return rc;
  if (X->T > 0 && !X->ptr) return CG_ERR_ARG;
  hipError_t e = launch_spectral(s, view_dev(X), gauge_dev(G_dev, shp), block_t, tau, workspace, stats, energy,
                                 force_generic(), static_cast<hipStream_t>(stream));
  return e == hipSuccess ? CG_OK : CG_ERR_DEVICE;
}

size_t gauge_grad_workspace_bytes(cg_gauge_shape shp, int32_t B, int32_t T, int32_t block_t) {
  if (check_shape(shp) != CG_OK || block_t < 2 || block_t > 32 || (block_t & (block_t - 1)) || B <= 0 || T < 0 ||
      shp.d % 16 || shp.d > 128)
    return 0;
  return grad_layout(shp, B, T, block_t).total;
}

int32_t kv_gauge_grad(int32_t s, const cg_kv_view* X, const float* A, const void* G_dev, cg_gauge_shape shp,
                      int32_t block_t, float tau, float lambda_f, float lambda_r, void* workspace, double* stats,
                      double* grad, void* stream) {
  int32_t rc = check_shape(shp);
  if (rc != CG_OK) return rc;
  if (s < 0 || s > 1 || !A || !G_dev || !workspace || !stats || !grad) return CG_ERR_ARG;
  if (block_t < 2 || block_t > 32 || (block_t & (block_t - 1)) || shp.d % 16 || shp.d > 128) return CG_ERR_UNSUPPORTED;
  if (!(tau > 0.0f) || !isfinite(tau) || !isfinite(lambda_f) || !isfinite(lambda_r)) return CG_ERR_ARG;
  if (!aligned16(G_dev) || !aligned16(workspace) || (reinterpret_cast<uintptr_t>(A) & 3u) ||
      (reinterpret_cast<uintptr_t>(stats) & 7u) || (reinterpret_cast<uintptr_t>(grad) & 7u))
    return CG_ERR_ALIGN;
  if ((rc = check_view(X, shp, shp.L)) != CG_OK) return rc;
  if (X->T > 0 && !X->ptr) return CG_ERR_ARG;
  hipError_t e = launch_gauge_grad(s, view_dev(X), gauge_dev(G_dev, shp), A, block_t, tau, lambda_f, lambda_r, workspace,
                                   stats, grad, force_generic(), static_cast<hipStream_t>(stream));
  return e == hipSuccess ? CG_OK : CG_ERR_DEVICE;
}

size_t attend_workspace_bytes(cg_gauge_shape shp, int32_t nl, int32_t B, int32_t Hq, int32_t T_cap) {
  if (check_shape(shp) != CG_OK || nl <= 0 || B <= 0 || T_cap <= 0 || Hq < shp.H || Hq % shp.H) return 0;
  return attend_plan(nl, B, shp.H, Hq, shp.d, T_cap).ws_bytes;
}

// kv_attend and kv_attend_noalloc: the same validation and split plan; the partial results of
// split rows go to the caller's workspace, or (noalloc) to the library's device scratch.
static int32_t attend_entry(int32_t l0, int32_t l1, const cg_kv_view* q, const cg_cache* kc, const cg_cache* vc,
                            const void* G_dev, cg_gauge_shape shp, const cg_codec* codec, const int32_t* lens,
                            float scale, const cg_kv_view* out, void* workspace, bool noalloc, int32_t* err_flag,
                            void* stream) {
  int32_t rc = check_shape(shp);
  if (rc != CG_OK) return rc;
  if (!G_dev || l0 < 0 || l1 <= l0 || l1 > shp.L || !isfinite(scale)) return CG_ERR_ARG;
  if (!aligned16(G_dev)) return CG_ERR_ALIGN;
  if (lens && (reinterpret_cast<uintptr_t>(lens) & 3u)) return CG_ERR_ALIGN;
  if ((rc = check_codec(codec, shp.d)) != CG_OK) return rc;
  if (codec->backend == CG_BACKEND_ZFP) return CG_ERR_UNSUPPORTED;
  const int nl = l1 - l0;
  if ((rc = check_qview(q, shp, nl)) != CG_OK) return rc;
  if ((rc = check_qview(out, shp, nl)) != CG_OK) return rc;
  if (out->B != q->B || out->H != q->H) return CG_ERR_SHAPE;
  const int B = q->B;
  if ((rc = check_cache(kc, codec, shp, B)) != CG_OK) return rc;
  if ((rc = check_cache(vc, codec, shp, B)) != CG_OK) return rc;
  if (kc->T_cap != vc->T_cap) return CG_ERR_SHAPE;
  if (!lens && (kc->len < 0 || kc->len > kc->T_cap || vc->len != kc->len)) return CG_ERR_CAPACITY;
  const AttendPlan cap = attend_plan(nl, B, shp.H, q->H, shp.d, kc->T_cap);
  if (!noalloc && cap.ws_bytes && (!workspace || !aligned16(workspace))) return workspace ? CG_ERR_ALIGN : CG_ERR_ARG;
  if (err_flag && (reinterpret_cast<uintptr_t>(err_flag) & 3u)) return CG_ERR_ALIGN;
  // rows of known length split over that length; device lengths over the capacity
  const AttendPlan p = lens ? cap : attend_plan(nl, B, shp.H, q->H, shp.d, std::max(1, kc->len));
  if (noalloc) {
    if (p.ws_bytes > attend_scratch_bytes()) return CG_ERR_CAPACITY;
    workspace = nullptr;
    if (p.ws_bytes && attend_scratch(&workspace) != hipSuccess) return CG_ERR_DEVICE;
  }
  AttendDev a;
  a.q = view_dev(q);
  a.o = view_dev(out);
  a.kc = cache_dev(kc);
  a.vc = cache_dev(vc);
  a.l0 = l0;
  a.Hq = q->H;
  a.grp = q->H / shp.H;
  a.lens = lens;
  a.len = kc->len;
  a.scale = scale;
  a.nsplit = p.nsplit;
  a.chunk = p.chunk;
  a.nqc = p.nqc;
  a.part = static_cast<float*>(workspace);
  a.err = err_flag;
  a.cap = kc->T_cap;
  a.win = 0;
  hipError_t e = launch_attend(a, gauge_dev(G_dev, shp), codec_dev(codec), force_generic(),
                               static_cast<hipStream_t>(stream));
  return e == hipSuccess ? CG_OK : CG_ERR_DEVICE;
}

int32_t kv_attend(int32_t l0, int32_t l1, const cg_kv_view* q, const cg_cache* kc, const cg_cache* vc,
                  const void* G_dev, cg_gauge_shape shp, const cg_codec* codec, const int32_t* lens, float scale,
                  const cg_kv_view* out, void* workspace, int32_t* err_flag, void* stream) {
  return attend_entry(l0, l1, q, kc, vc, G_dev, shp, codec, lens, scale, out, workspace, false, err_flag, stream);
}

int32_t kv_attend_noalloc(int32_t l0, int32_t l1, const cg_kv_view* q, const cg_cache* kc, const cg_cache* vc,
                          const void* G_dev, cg_gauge_shape shp, const cg_codec* codec, const int32_t* lens,
                          float scale, const cg_kv_view* out, int32_t* err_flag, void* stream) {
  return attend_entry(l0, l1, q, kc, vc, G_dev, shp, codec, lens, scale, out, nullptr, true, err_flag, stream);
}

// page tables: block-uniform per-token blocks or passthrough, pages of a multiple of 64 positions
static int32_t check_pages(const cg_page_table* pt, const cg_codec* codec, const cg_cache* kc) {
  if (!pt || !pt->pages || pt->max_pages <= 0) return CG_ERR_ARG;
  if (reinterpret_cast<uintptr_t>(pt->pages) & 3u) return CG_ERR_ALIGN;
  const bool ok = codec->backend == CG_BACKEND_PASSTHROUGH ||
                  (codec->backend == CG_BACKEND_BLOCK_UNIFORM && codec->block_t == 1);
  if (!ok) return CG_ERR_UNSUPPORTED;
  if (pt->page_size <= 0 || pt->page_size % 64 || pt->page_size != kc->T_cap) return CG_ERR_SHAPE;
  return CG_OK;
}

size_t attend_paged_workspace_bytes(cg_gauge_shape shp, int32_t nl, int32_t B, int32_t Hq, int32_t max_pages,
                                    int32_t page_size) {
  if (max_pages <= 0 || page_size <= 0 || int64_t(max_pages) * page_size > INT32_MAX) return 0;
  return attend_workspace_bytes(shp, nl, B, Hq, max_pages * page_size);
}

int32_t kv_attend_paged(int32_t l0, int32_t l1, const cg_kv_view* q, const cg_cache* kc, const cg_cache* vc,
                        const cg_page_table* pages, const void* G_dev, cg_gauge_shape shp, const cg_codec* codec,
                        const int32_t* lens, float scale, const cg_kv_view* out, void* workspace, int32_t* err_flag,
                        void* stream) {
  int32_t rc = check_shape(shp);
  if (rc != CG_OK) return rc;
  if (!G_dev || !lens || l0 < 0 || l1 <= l0 || l1 > shp.L || !isfinite(scale)) return CG_ERR_ARG;
  if (!aligned16(G_dev)) return CG_ERR_ALIGN;
  if (reinterpret_cast<uintptr_t>(lens) & 3u) return CG_ERR_ALIGN;
  if ((rc = check_codec(codec, shp.d)) != CG_OK) return rc;
  const int nl = l1 - l0;
  if ((rc = check_qview(q, shp, nl)) != CG_OK) return rc;
  if ((rc = check_qview(out, shp, nl)) != CG_OK) return rc;
  if (out->B != q->B || out->H != q->H) return CG_ERR_SHAPE;
  // the caches are page pools: their batch dimension counts pages
  if (!kc || !vc) return CG_ERR_ARG;
  if ((rc = check_cache(kc, codec, shp, kc->B)) != CG_OK) return rc;
  if ((rc = check_cache(vc, codec, shp, kc->B)) != CG_OK) return rc;
  if (kc->T_cap != vc->T_cap) return CG_ERR_SHAPE;
  if ((rc = check_pages(pages, codec, kc)) != CG_OK) return rc;
  if (int64_t(pages->max_pages) * pages->page_size > INT32_MAX) return CG_ERR_CAPACITY;
  const int cap = pages->max_pages * pages->page_size;
  const AttendPlan p = attend_plan(nl, q->B, shp.H, q->H, shp.d, cap);
  if (p.ws_bytes && (!workspace || !aligned16(workspace))) return workspace ? CG_ERR_ALIGN : CG_ERR_ARG;
  if (err_flag && (reinterpret_cast<uintptr_t>(err_flag) & 3u)) return CG_ERR_ALIGN;
  AttendDev a;
  a.q = view_dev(q);
  a.o = view_dev(out);
  a.kc = cache_dev(kc);
  a.vc = cache_dev(vc);
  a.l0 = l0;
  a.Hq = q->H;
  a.grp = q->H / shp.H;
  a.lens = lens;
  a.len = 0;
  a.scale = scale;
  a.nsplit = p.nsplit;
  a.chunk = p.chunk;
  a.nqc = p.nqc;
  a.part = static_cast<float*>(workspace);
  a.err = err_flag;
  a.pt.pages = pages->pages;
  a.pt.max_pages = pages->max_pages;
  a.pt.page_size = pages->page_size;
  a.cap = cap;
  a.win = 0;
  hipError_t e = launch_attend(a, gauge_dev(G_dev, shp), codec_dev(codec), force_generic(),
                               static_cast<hipStream_t>(stream));
  return e == hipSuccess ? CG_OK : CG_ERR_DEVICE;
}

int32_t kv_encode_paged(int32_t s, const cg_kv_view* X, const cg_page_table* pages, const void* G_dev,
                        cg_gauge_shape shp, const cg_codec* codec, const cg_cache* out, int32_t t0, int32_t* err_flag,
                        void* stream) {
  int32_t rc = check_shape(shp);
  if (rc != CG_OK) return rc;
  if (s < 0 || s > 1 || !G_dev) return CG_ERR_ARG;
  if (!aligned16(G_dev)) return CG_ERR_ALIGN;
  if ((rc = check_codec(codec, shp.d)) != CG_OK) return rc;
  if ((rc = check_view(X, shp, shp.L)) != CG_OK) return rc;
  if (!out) return CG_ERR_ARG;
  if ((rc = check_cache(out, codec, shp, out->B)) != CG_OK) return rc;
  if ((rc = check_pages(pages, codec, out)) != CG_OK) return rc;
  if (t0 < 0) return CG_ERR_ARG;
  if (t0 % 32) return CG_ERR_UNSUPPORTED;  // 32-position tiles stay inside one page
  if (int64_t(t0) + X->T > int64_t(pages->max_pages) * pages->page_size) return CG_ERR_CAPACITY;
  if (err_flag && (reinterpret_cast<uintptr_t>(err_flag) & 3u)) return CG_ERR_ALIGN;
  PageDev pt;
  pt.pages = pages->pages;
  pt.max_pages = pages->max_pages;
  pt.page_size = pages->page_size;
  hipError_t e = launch_encode_generic(s, view_dev(X), 0, gauge_dev(G_dev, shp), codec_dev(codec), cache_dev(out), t0,
                                       X->T, err_flag, static_cast<hipStream_t>(stream), pt);
  return e == hipSuccess ? CG_OK : CG_ERR_DEVICE;
}

int32_t kv_append_paged(int32_t l0, int32_t l1, const cg_kv_view* k_new, const cg_kv_view* v_new, const int32_t* pos,
                        const cg_page_table* pages, const void* G_dev, cg_gauge_shape shp, const cg_codec* codec,
                        const cg_cache* kc, const cg_cache* vc, int32_t* err_flag, void* stream) {
  int32_t rc = check_shape(shp);
  if (rc != CG_OK) return rc;
  if (!G_dev || !pos || l0 < 0 || l1 <= l0 || l1 > shp.L) return CG_ERR_ARG;
  if (!aligned16(G_dev)) return CG_ERR_ALIGN;
  if ((reinterpret_cast<uintptr_t>(pos) & 3u)) return CG_ERR_ALIGN;
  if ((rc = check_codec(codec, shp.d)) != CG_OK) return rc;
  const int nl = l1 - l0;
  if ((rc = check_view(k_new, shp, nl)) != CG_OK) return rc;
  if ((rc = check_view(v_new, shp, nl)) != CG_OK) return rc;
  if (k_new->T != 1 || v_new->T != 1 || v_new->B != k_new->B) return CG_ERR_SHAPE;
  if (!kc || !vc) return CG_ERR_ARG;
  if ((rc = check_cache(kc, codec, shp, kc->B)) != CG_OK) return rc;
  if ((rc = check_cache(vc, codec, shp, kc->B)) != CG_OK) return rc;
  if (kc->T_cap != vc->T_cap) return CG_ERR_SHAPE;
  if ((rc = check_pages(pages, codec, kc)) != CG_OK) return rc;
  if (err_flag && (reinterpret_cast<uintptr_t>(err_flag) & 3u)) return CG_ERR_ALIGN;
  hipStream_t st = static_cast<hipStream_t>(stream);
  const GaugeDev G = gauge_dev(G_dev, shp);
  const CodecDev c = codec_dev(codec);
  PageDev pt;
  pt.pages = pages->pages;
  pt.max_pages = pages->max_pages;
  pt.page_size = pages->page_size;
  hipError_t e = launch_append(0, view_dev(k_new), l0, pos, G, c, cache_dev(kc), err_flag, st, pt);
  if (e == hipSuccess) e = launch_append(1, view_dev(v_new), l0, pos, G, c, cache_dev(vc), err_flag, st, pt);
  return e == hipSuccess ? CG_OK : CG_ERR_DEVICE;
}

int32_t cg_selftest(int32_t which, uint64_t* mismatches_dev, void* stream) {
  if (which < 0 || which > 2 || !mismatches_dev) return CG_ERR_ARG;
  if (reinterpret_cast<uintptr_t>(mismatches_dev) & 7u) return CG_ERR_ALIGN;
  hipError_t e = launch_selftest(which, reinterpret_cast<unsigned long long*>(mismatches_dev),
                                 static_cast<hipStream_t>(stream));
  return e == hipSuccess ? CG_OK : CG_ERR_DEVICE;
}

int32_t cg_stream_probe(const void* src, int64_t read_bytes, void* dst, int64_t write_bytes, void* stream) {
  if (!src || read_bytes <= 0 || read_bytes % 8192 || write_bytes < 0 || write_bytes % 16 || (write_bytes && !dst))
    return CG_ERR_ARG;
  if ((reinterpret_cast<uintptr_t>(src) | reinterpret_cast<uintptr_t>(dst)) & 15u) return CG_ERR_ALIGN;
  hipError_t e = launch_stream_probe(src, read_bytes, dst, write_bytes, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? CG_OK : CG_ERR_DEVICE;
}

}  // extern "C"
