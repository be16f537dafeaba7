/*
 * CPU oracle for the gauge-coded KV-cache codec of Codec-Gauge
 * ("Learning Compression-Friendly Gauges for Transformer KV Caches").
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library links, loads or calls
 * this file; only the test-suite, the smoke check and the CPU-baseline leg of the
 * benchmark do.  It shares no code, header, table or helper with the HIP path.
 *
 * What it computes (paper section 3, the codec-wrapper equations):
 *     Z = G X,   B_c = C(Z),   Zhat = D(B_c),   Xhat = G^{-1} Zhat = G^T Zhat
 * with one orthogonal g x g gauge per (layer, K/V, head, channel group) (section 3,
 * Table 1; section 4.1 eq. G = exp(A - A^T)), acting on contiguous channel groups
 * of each cached vector and never mixing tokens, heads or layers.
 *
 * Backends (section 4.3, Compression Conditions):
 *   - error-free passthrough (the no-compression sanity rows of section 4.4),
 *   - block-uniform b-bit quantisation with one (min, scale) range per block: a block is
 *     n channels of one token vector, or, in the token-channel tiles the paper names, the
 *     same n channels over T_b consecutive tokens (an unfinished tile waits in a bf16
 *     staging window),
 *   - KIVI-style quantisation: per-channel key ranges over token groups and
 *     per-token value ranges over channel groups, with a full-precision window
 *     of recent tokens,
 *   - a zfp-style fixed-rate transform codec (the paper's primary backend is zfp at fixed
 *     rates, section 4.3), written from the published description of zfp's algorithm
 *     (block-floating-point alignment, decorrelating transform, sequency ordering,
 *     negabinary, embedded bit-plane coding with group tests) over the 2-D field whose
 *     x axis is the channel and whose y axis runs over the tokens.
 *
 * Precision: the gauge is "exact result, then round once to fp32": products of
 * fp32 by bf16/fp32 are exact in binary64 and the sums are carried in binary64.
 * The quantiser is written out step by step in binary32 with IEEE round-to-
 * nearest-even and no fused multiply-add (build with -ffp-contract=off):
 *   mn_h = fp16 round toward -inf (min z), canonical +0
 *   sc_h = fp16 round toward +inf (fl32(fl32(max - mn_h) / (2^b - 1)))
 *   inv  = fl32(1 / sc_h)  (0 when sc_h == 0)
 *   q    = clamp(rint_even(fl32(fl32(z - mn_h) * inv)), 0, 2^b - 1)
 *   zhat = fl32(mn_h + q * sc_h)          (q * sc_h is exact in binary32)
 * The paper leaves range form, side-info precision, rounding directions, tie
 * rule, division form, bit order and buffer layout unstated; the readings taken
 * here are listed with the design notes of the repository.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORC_FLAG_NONFINITE 1
#define ORC_FLAG_SIDE_OVERFLOW 2
#define ORC_EARG (-1)
#define ORC_ENOTORTH (-2)

enum { ORC_BACKEND_PASSTHROUGH = 0, ORC_BACKEND_BLOCK_UNIFORM = 1, ORC_BACKEND_KIVI = 2, ORC_BACKEND_ZFP = 3 };
enum { ORC_GAUGE_IDENTITY = 0, ORC_GAUGE_HAAR = 1, ORC_GAUGE_DCT2 = 2, ORC_GAUGE_HADAMARD = 3,
       ORC_GAUGE_EXPM = 4, ORC_GAUGE_USER = 5 };

/* ------------------------------------------------------------------------------------------ */
/* IEEE binary16 / bfloat16 helpers, written from the format definitions.                      */
/* ------------------------------------------------------------------------------------------ */

static float f32_from_bits(uint32_t u) { float f; memcpy(&f, &u, 4); return f; }
static uint32_t bits_from_f32(float f) { uint32_t u; memcpy(&u, &f, 4); return u; }

/* bfloat16 is the upper half of a binary32 word. */
float orc_bf16_to_f32(uint16_t h) { return f32_from_bits((uint32_t)h << 16); }

/* binary32 -> bfloat16, round to nearest, ties to even. */
uint16_t orc_f32_to_bf16(float f) {
  uint32_t u = bits_from_f32(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x0040u); /* quiet NaN */
  uint32_t upper = u >> 16, lower = u & 0xffffu;
  if (lower > 0x8000u || (lower == 0x8000u && (upper & 1u))) upper += 1u;
  return (uint16_t)upper;
}

/* Round a real value onto the binary16 grid in a given direction (dir < 0: toward -inf,
 * dir > 0: toward +inf).  The binary16 numbers in the binade [2^e, 2^(e+1)) are spaced
 * 2^(e-10) apart, e in [-14, 15]; below 2^-14 the spacing stays 2^-24 (subnormals).
 * Overflow follows IEEE directed rounding: toward -inf maps +huge to +65504 and -huge
 * to -inf; toward +inf maps +huge to +inf and -huge to -65504.  Zero results are +0. */
double orc_f16_round_dir(double v, int dir) {
  if (v == 0.0) return 0.0;
  if (isnan(v)) return v;
  if (isinf(v)) {
    if (v > 0) return dir < 0 ? 65504.0 : INFINITY;
    return dir < 0 ? -INFINITY : -65504.0;
  }
  double a = fabs(v);
  int e2;
  frexp(a, &e2);        /* a = m * 2^e2, m in [0.5, 1) */
  int e = e2 - 1;       /* a in [2^e, 2^(e+1)) */
  if (e < -14) e = -14;
  if (e > 15) e = 15;
  double spacing = ldexp(1.0, e - 10);
  double k = v / spacing; /* exact: power-of-two scaling */
  double r = (dir < 0 ? floor(k) : ceil(k)) * spacing;
  if (r > 65504.0) r = (dir < 0) ? 65504.0 : INFINITY;
  if (r < -65504.0) r = (dir < 0) ? -INFINITY : -65504.0;
  if (r == 0.0) r = 0.0; /* canonical +0 */
  return r;
}

/* Encode a value that lies exactly on the binary16 grid (or is +-inf / NaN) as its bits. */
uint16_t orc_f16_bits(double v) {
  uint16_t sign = (v < 0.0 || (v == 0.0 && signbit(v))) ? 0x8000u : 0u;
  if (isnan(v)) return 0x7e00u;
  double a = fabs(v);
  if (isinf(a)) return (uint16_t)(sign | 0x7c00u);
  if (a == 0.0) return sign;
  if (a < ldexp(1.0, -14)) return (uint16_t)(sign | (uint16_t)(a / ldexp(1.0, -24)));
  int e2;
  double m = frexp(a, &e2); /* a = m 2^e2, m in [0.5,1) -> a = (2m) 2^(e2-1) */
  int e = e2 - 1;
  uint16_t mant = (uint16_t)((2.0 * m - 1.0) * 1024.0);
  return (uint16_t)(sign | (uint16_t)((e + 15) << 10) | mant);
}

double orc_f16_value(uint16_t h) {
  int sign = (h >> 15) & 1, ex = (h >> 10) & 0x1f, mant = h & 0x3ff;
  double v;
  if (ex == 0x1f) v = mant ? NAN : INFINITY;
  else if (ex == 0) v = ldexp((double)mant, -24);
  else v = ldexp(1.0 + mant / 1024.0, ex - 15);
  return sign ? -v : v;
}

/* ------------------------------------------------------------------------------------------ */
/* Philox4x32-10 (Salmon, Moraes, Dror, Shaw, "Parallel random numbers: as easy as 1, 2, 3",  */
/* SC 2011): ten rounds of two 32x32->64 multiplies with a Weyl-sequence key schedule.        */
/* ------------------------------------------------------------------------------------------ */

void orc_philox4x32_10(const uint32_t ctr_in[4], const uint32_t key_in[2], uint32_t out[4]) {
  uint32_t c0 = ctr_in[0], c1 = ctr_in[1], c2 = ctr_in[2], c3 = ctr_in[3];
  uint32_t k0 = key_in[0], k1 = key_in[1];
  for (int round = 0; round < 10; ++round) {
    if (round > 0) { k0 += 0x9E3779B9u; k1 += 0xBB67AE85u; }
    uint64_t p0 = (uint64_t)0xD2511F53u * c0;
    uint64_t p1 = (uint64_t)0xCD9E8D57u * c2;
    uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
    uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
    uint32_t n0 = hi1 ^ c1 ^ k0, n1 = lo1, n2 = hi0 ^ c3 ^ k1, n3 = lo0;
    c0 = n0; c1 = n1; c2 = n2; c3 = n3;
  }
  out[0] = c0; out[1] = c1; out[2] = c2; out[3] = c3;
}

/* Standard normal number k of stream `index` under `seed`: Philox block c = k/4 with counter
 * (c, 0, index_lo, index_hi) and key (seed_lo, seed_hi) gives four words; each pair
 * (u1, u2) feeds one Box-Muller transform with u1 = (w1 + 1) 2^-32 in (0, 1] and
 * u2 = w2 2^-32 in [0, 1): the pair yields r cos(2 pi u2) then r sin(2 pi u2). */
double orc_gaussian(uint64_t seed, uint64_t index, uint64_t k) {
  uint32_t ctr[4] = {(uint32_t)(k / 4), 0u, (uint32_t)index, (uint32_t)(index >> 32)};
  uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
  uint32_t w[4];
  orc_philox4x32_10(ctr, key, w);
  int pair = (int)((k % 4) / 2), which = (int)(k % 2);
  double u1 = ((double)w[2 * pair] + 1.0) * ldexp(1.0, -32);
  double u2 = (double)w[2 * pair + 1] * ldexp(1.0, -32);
  double r = sqrt(-2.0 * log(u1));
  double ang = 2.0 * M_PI * u2;
  return which == 0 ? r * cos(ang) : r * sin(ang);
}

/* ------------------------------------------------------------------------------------------ */
/* Gauges (section 3 / Table 1: one g x g orthogonal matrix per (l, s, h, r); section 4.1:    */
/* G = exp(A - A^T); section 4.3: identity, sampled random orthogonal, Hadamard and DCT        */
/* controls).  All are built in binary64, then rounded once to binary32.  Convention:        */
/* z = G x, i.e. G[i][j] multiplies input channel j into output channel i.                    */
/* ------------------------------------------------------------------------------------------ */

static void gauge_identity(int g, double* Q) {
  for (int i = 0; i < g; ++i)
    for (int j = 0; j < g; ++j) Q[i * g + j] = (i == j) ? 1.0 : 0.0;
}

/* Orthonormal DCT-II: row k is frequency k, C[k][n] = sqrt(c_k / g) cos(pi (2n+1) k / (2g)),
 * c_0 = 1, c_k = 2 otherwise. */
static void gauge_dct2(int g, double* Q) {
  for (int k = 0; k < g; ++k)
    for (int n = 0; n < g; ++n)
      Q[k * g + n] = sqrt((k == 0 ? 1.0 : 2.0) / g) * cos(M_PI * (2.0 * n + 1.0) * k / (2.0 * g));
}

/* Sylvester-ordered Hadamard matrix, normalised: H[i][j] = (-1)^{popcount(i & j)} / sqrt(g). */
static int gauge_hadamard(int g, double* Q) {
  if (g <= 0 || (g & (g - 1))) return ORC_EARG;
  double s = 1.0 / sqrt((double)g);
  for (int i = 0; i < g; ++i)
    for (int j = 0; j < g; ++j) Q[i * g + j] = (__builtin_popcount((unsigned)(i & j)) & 1) ? -s : s;
  return 0;
}

/* Haar-distributed orthogonal matrix: Q of the QR factorisation of a g x g standard-normal
 * matrix M with R's diagonal taken positive (Mezzadri, "How to generate random matrices from
 * the classical compact groups", 2007).  Gram-Schmidt on the columns of M (applied twice for
 * orthogonality in binary64) yields exactly that factor, since each R_jj is a positive norm.
 * M[i][j] is normal number i*g + j of stream `index`. */
static void gauge_haar(int g, uint64_t seed, uint64_t index, double* Q) {
  double* M = (double*)malloc(sizeof(double) * g * g);
  for (int i = 0; i < g; ++i)
    for (int j = 0; j < g; ++j) M[i * g + j] = orc_gaussian(seed, index, (uint64_t)i * g + j);
  for (int j = 0; j < g; ++j) {
    /* column j of M into column j of Q, minus its projections on earlier columns (twice) */
    for (int i = 0; i < g; ++i) Q[i * g + j] = M[i * g + j];
    for (int pass = 0; pass < 2; ++pass) {
      for (int p = 0; p < j; ++p) {
        double dot = 0.0;
        for (int i = 0; i < g; ++i) dot += Q[i * g + p] * Q[i * g + j];
        for (int i = 0; i < g; ++i) Q[i * g + j] -= dot * Q[i * g + p];
      }
    }
    double nrm = 0.0;
    for (int i = 0; i < g; ++i) nrm += Q[i * g + j] * Q[i * g + j];
    nrm = sqrt(nrm);
    for (int i = 0; i < g; ++i) Q[i * g + j] /= nrm;
  }
  free(M);
}

/* exp(S) for the skew-symmetric S = A - A^T (section 4.1 eq.): scaling and squaring with a
 * Taylor series.  S is scaled by 2^-s until its max-row-sum norm is below 1/2; the series is
 * summed until its terms stop changing the sum; the result is squared s times. */
static void gauge_expm(int g, const float* A, double* Q) {
  size_t gg = (size_t)g * g;
  double* S = (double*)malloc(sizeof(double) * gg);
  double* term = (double*)malloc(sizeof(double) * gg);
  double* tmp = (double*)malloc(sizeof(double) * gg);
  double norm = 0.0;
  for (int i = 0; i < g; ++i) {
    double row = 0.0;
    for (int j = 0; j < g; ++j) {
      S[i * g + j] = (double)A[i * g + j] - (double)A[j * g + i];
      row += fabs(S[i * g + j]);
    }
    if (row > norm) norm = row;
  }
  int sq = 0;
  while (norm > 0.5) { norm *= 0.5; ++sq; }
  double scale = ldexp(1.0, -sq);
  for (size_t k = 0; k < gg; ++k) S[k] *= scale;
  gauge_identity(g, Q);
  gauge_identity(g, term);
  for (int n = 1; n < 60; ++n) {
    /* term <- term * S / n */
    double tmax = 0.0;
    for (int i = 0; i < g; ++i)
      for (int j = 0; j < g; ++j) {
        double acc = 0.0;
        for (int k = 0; k < g; ++k) acc += term[i * g + k] * S[k * g + j];
        tmp[i * g + j] = acc / n;
      }
    for (size_t k = 0; k < gg; ++k) {
      term[k] = tmp[k];
      Q[k] += term[k];
      if (fabs(term[k]) > tmax) tmax = fabs(term[k]);
    }
    if (tmax < 1e-18) break;
  }
  for (int s = 0; s < sq; ++s) {
    for (int i = 0; i < g; ++i)
      for (int j = 0; j < g; ++j) {
        double acc = 0.0;
        for (int k = 0; k < g; ++k) acc += Q[i * g + k] * Q[k * g + j];
        tmp[i * g + j] = acc;
      }
    memcpy(Q, tmp, sizeof(double) * gg);
  }
  free(S); free(term); free(tmp);
}

/* max |G G^T - I| in binary64 over one g x g binary32 gauge. */
double orc_orthogonality_error(int g, const float* G) {
  double worst = 0.0;
  for (int i = 0; i < g; ++i)
    for (int j = 0; j < g; ++j) {
      double acc = 0.0;
      for (int k = 0; k < g; ++k) acc += (double)G[i * g + k] * (double)G[j * g + k];
      double e = fabs(acc - (i == j ? 1.0 : 0.0));
      if (e > worst) worst = e;
    }
  return worst;
}

/* Build every gauge of a cache: G[L][2][H][R][g][g] (binary32, row-major), R = d / g.
 * Random gauges are independent per block, with stream index ((l*2 + s)*H + h)*R + r.
 * EXPM reads the generators A with the same shape from `params`; USER copies `params`
 * and rejects any block whose max |G G^T - I| exceeds 1e-5. */
int orc_gauge_make(int kind, int L, int H, int d, int g, uint64_t seed, const float* params, float* G) {
  if (L <= 0 || H <= 0 || d <= 0 || g <= 0 || d % g) return ORC_EARG;
  int R = d / g;
  size_t gg = (size_t)g * g;
  double* Q = (double*)malloc(sizeof(double) * gg);
  int rc = 0;
  for (int l = 0; l < L && rc == 0; ++l)
    for (int s = 0; s < 2 && rc == 0; ++s)
      for (int h = 0; h < H && rc == 0; ++h)
        for (int r = 0; r < R && rc == 0; ++r) {
          uint64_t idx = (((uint64_t)l * 2 + s) * H + h) * R + r;
          float* out = G + idx * gg;
          switch (kind) {
            case ORC_GAUGE_IDENTITY: gauge_identity(g, Q); break;
            case ORC_GAUGE_DCT2: gauge_dct2(g, Q); break;
            case ORC_GAUGE_HADAMARD: rc = gauge_hadamard(g, Q); break;
            case ORC_GAUGE_HAAR: gauge_haar(g, seed, idx, Q); break;
            case ORC_GAUGE_EXPM:
              if (!params) { rc = ORC_EARG; break; }
              gauge_expm(g, params + idx * gg, Q);
              break;
            case ORC_GAUGE_USER:
              if (!params) { rc = ORC_EARG; break; }
              for (size_t k = 0; k < gg; ++k) Q[k] = params[idx * gg + k];
              break;
            default: rc = ORC_EARG;
          }
          if (rc) break;
          for (size_t k = 0; k < gg; ++k) out[k] = (float)Q[k];
          if (kind == ORC_GAUGE_USER && orc_orthogonality_error(g, out) > 1e-5) rc = ORC_ENOTORTH;
        }
  free(Q);
  return rc;
}

/* ------------------------------------------------------------------------------------------ */
/* Gauge application (section 3: Z[b,h,t,r] = G_{l,s,h,r} X[b,h,t,r]; Xhat = G^T Zhat).       */
/* Gs points at the R gauges of one (l, s, h).                                                 */
/* ------------------------------------------------------------------------------------------ */

void orc_gauge_apply(int d, int g, const float* Gs, const float* x, float* z) {
  int R = d / g;
  for (int r = 0; r < R; ++r) {
    const float* Gr = Gs + (size_t)r * g * g;
    for (int i = 0; i < g; ++i) {
      double acc = 0.0;
      for (int j = 0; j < g; ++j) acc += (double)Gr[i * g + j] * (double)x[r * g + j];
      z[r * g + i] = (float)acc;
    }
  }
}

void orc_gauge_inverse(int d, int g, const float* Gs, const float* z, float* x) {
  int R = d / g;
  for (int r = 0; r < R; ++r) {
    const float* Gr = Gs + (size_t)r * g * g;
    for (int i = 0; i < g; ++i) {
      double acc = 0.0;
      for (int j = 0; j < g; ++j) acc += (double)Gr[j * g + i] * (double)z[r * g + j];
      x[r * g + i] = (float)acc;
    }
  }
}

/* ------------------------------------------------------------------------------------------ */
/* Scalar quantiser for one block (section 4.3: one range per block), step by step.           */
/* ------------------------------------------------------------------------------------------ */

int orc_quantize_block(const float* z, int n, int bits, uint8_t* q, uint16_t* mn_bits, uint16_t* sc_bits) {
  int flags = 0;
  float mn = z[0], mx = z[0];
  for (int i = 0; i < n; ++i) {
    if (!isfinite(z[i])) flags |= ORC_FLAG_NONFINITE;
    if (z[i] < mn) mn = z[i];
    if (z[i] > mx) mx = z[i];
  }
  int qmax = (1 << bits) - 1;
  double mn_h = orc_f16_round_dir((double)mn, -1);
  float mnf = (float)mn_h;
  float diff = mx - mnf;
  float s32 = diff / (float)qmax;
  double sc_h = orc_f16_round_dir((double)s32, +1);
  if (isinf(mn_h) || isinf(sc_h) || isnan(mn_h) || isnan(sc_h)) flags |= ORC_FLAG_SIDE_OVERFLOW;
  float scf = (float)sc_h;
  float inv = (scf == 0.0f) ? 0.0f : 1.0f / scf;
  for (int i = 0; i < n; ++i) {
    float dz = z[i] - mnf;
    float t = dz * inv;
    float r = nearbyintf(t);
    if (!(r >= 0.0f)) r = 0.0f;
    if (r > (float)qmax) r = (float)qmax;
    q[i] = (uint8_t)r;
  }
  *mn_bits = orc_f16_bits(mn_h);
  *sc_bits = orc_f16_bits(sc_h);
  return flags;
}

void orc_dequantize_block(const uint8_t* q, int n, uint16_t mn_bits, uint16_t sc_bits, float* zhat) {
  float mnf = (float)orc_f16_value(mn_bits);
  float scf = (float)orc_f16_value(sc_bits);
  for (int i = 0; i < n; ++i) {
    float p = (float)q[i] * scf;
    zhat[i] = mnf + p;
  }
}

/* LSB-first bit stream: bit k of the stream is bit (k mod b) of code floor(k / b);
 * stream bit k lives in byte k/8 at bit position k%8. */
void orc_pack_codes(const uint8_t* q, int n, int bits, uint8_t* out) {
  int nbytes = (n * bits + 7) / 8;
  memset(out, 0, (size_t)nbytes);
  for (int i = 0; i < n; ++i)
    for (int k = 0; k < bits; ++k) {
      int pos = i * bits + k;
      if ((q[i] >> k) & 1) out[pos / 8] |= (uint8_t)(1u << (pos % 8));
    }
}

void orc_unpack_codes(const uint8_t* in, int n, int bits, uint8_t* q) {
  for (int i = 0; i < n; ++i) {
    int v = 0;
    for (int k = 0; k < bits; ++k) {
      int pos = i * bits + k;
      v |= ((in[pos / 8] >> (pos % 8)) & 1) << k;
    }
    q[i] = (uint8_t)v;
  }
}

/* ------------------------------------------------------------------------------------------ */
/* zfp-style fixed-rate codec of 4 x 4 blocks (4 consecutive channels x 4 consecutive tokens), */
/* following the published description of zfp (Lindstrom 2014):                                */
/*   1. block exponent e: the smallest e with |v| < 2^e for every value (frexp exponent of the */
/*      largest magnitude), at least -126; an all-zero block is one 0 bit;                     */
/*   2. fixed point: i = trunc(v 2^(30 - e)), |i| < 2^30;                                      */
/*   3. decorrelating transform along the channels, then along the tokens, each the 4-point   */
/*      map A = 1/16 [[4 4 4 4] [5 1 -1 -5] [-4 4 4 -4] [-2 6 -6 2]] computed by integer      */
/*      lifting (additions and halvings), inverse by the lifting steps undone in reverse;     */
/*   4. coefficients ordered by sequency (i + j, then i^2 + j^2, then the token index j);     */
/*   5. negabinary u = (i + 0xAAAAAAAA) ^ 0xAAAAAAAA;                                          */
/*   6. bit planes 31 .. 0: the plane's bits of the coefficients already significant, then   */
/*      group tests over the rest (a 1 bit says some remaining coefficient has a 1 in the     */
/*      plane; then their bits one by one up to that 1, which becomes significant with the   */
/*      ones before it; the last remaining coefficient's 1 is implied), until the budget of  */
/*      16 rate bits per block (header included: 1 + 8 exponent bits) is spent.              */
/* The bit stream of a block is LSB-first; blocks are 2 rate bytes each, so the rate is      */
/* exact: rate bits per value.  Non-finite inputs flag NONFINITE and code a zero block.       */
/* ------------------------------------------------------------------------------------------ */

static int zfp_order[16];  /* sequency position -> block index 4 j + i */
static int zfp_order_ready = 0;

static void zfp_make_order(void) {
  if (zfp_order_ready) return;
  int idx[16];
  for (int k = 0; k < 16; ++k) idx[k] = k;
  /* insertion sort by (i + j, i^2 + j^2, j) */
  for (int a = 1; a < 16; ++a) {
    int v = idx[a], b = a - 1;
    for (; b >= 0; --b) {
      int p = idx[b];
      int pi = p % 4, pj = p / 4, vi = v % 4, vj = v / 4;
      int kp = (pi + pj) * 1000 + (pi * pi + pj * pj) * 10 + pj;
      int kv = (vi + vj) * 1000 + (vi * vi + vj * vj) * 10 + vj;
      if (kp <= kv) break;
      idx[b + 1] = p;
    }
    idx[b + 1] = v;
  }
  memcpy(zfp_order, idx, sizeof idx);
  zfp_order_ready = 1;
}

void orc_zfp_order(int* out) {
  zfp_make_order();
  memcpy(out, zfp_order, sizeof zfp_order);
}

/* two's-complement wrapping add / subtract / double and arithmetic halving on 32 bits */
static int32_t wadd(int32_t a, int32_t b) { return (int32_t)((uint32_t)a + (uint32_t)b); }
static int32_t wsub(int32_t a, int32_t b) { return (int32_t)((uint32_t)a - (uint32_t)b); }
static int32_t wdbl(int32_t a) { return (int32_t)((uint32_t)a << 1); }
static int32_t half(int32_t a) { return a >= 0 ? a / 2 : -((-(int64_t)a + 1) / 2); }  /* floor(a / 2) */

/* forward 4-point transform of p[0], p[s], p[2s], p[3s] by lifting */
void orc_zfp_fwd4(int32_t* p, int s) {
  int32_t x = p[0], y = p[s], z = p[2 * s], w = p[3 * s];
  /* averages and half-differences of the outer pair (x, w) and the inner pair (y, z) */
  x = half(wadd(x, w)); w = wsub(w, x);
  z = half(wadd(z, y)); y = wsub(y, z);
  /* mean of the four; the even combination; the two odd ones */
  x = half(wadd(x, z)); z = wsub(z, x);
  w = half(wadd(w, y)); y = wsub(y, w);
  /* final rotation of the two odd coefficients */
  w = wadd(w, half(y)); y = wsub(y, half(w));
  p[0] = x; p[s] = y; p[2 * s] = z; p[3 * s] = w;
}

/* the lifting steps above undone in reverse order */
void orc_zfp_inv4(int32_t* p, int s) {
  int32_t x = p[0], y = p[s], z = p[2 * s], w = p[3 * s];
  y = wadd(y, half(w)); w = wsub(w, half(y));
  y = wadd(y, w); w = wsub(wdbl(w), y);
  z = wadd(z, x); x = wsub(wdbl(x), z);
  y = wadd(y, z); z = wsub(wdbl(z), y);
  w = wadd(w, x); x = wsub(wdbl(x), w);
  p[0] = x; p[s] = y; p[2 * s] = z; p[3 * s] = w;
}

uint32_t orc_negabinary(int32_t i) { return ((uint32_t)i + 0xAAAAAAAAu) ^ 0xAAAAAAAAu; }
int32_t orc_from_negabinary(uint32_t u) { return (int32_t)((u ^ 0xAAAAAAAAu) - 0xAAAAAAAAu); }

typedef struct {
  uint8_t* buf;
  int pos, cap;
} orc_bits;

static int bits_put(orc_bits* w, int bit) {
  if (w->pos >= w->cap) return 0;
  if (bit) w->buf[w->pos >> 3] |= (uint8_t)(1u << (w->pos & 7));
  w->pos++;
  return 1;
}
static int bits_get(orc_bits* r, int* bit) {
  if (r->pos >= r->cap) return 0;
  *bit = (r->buf[r->pos >> 3] >> (r->pos & 7)) & 1;
  r->pos++;
  return 1;
}

/* v[4 j + i]: channel i, token j of the block.  out: 2 rate bytes (cleared here). */
int orc_zfp_encode_block(const float* v, int rate, uint8_t* out) {
  zfp_make_order();
  const int maxbits = 16 * rate;
  memset(out, 0, (size_t)(maxbits / 8));
  orc_bits w = {out, 0, maxbits};
  int flags = 0;
  float amax = 0.0f;
  for (int k = 0; k < 16; ++k) {
    if (!isfinite(v[k])) flags |= ORC_FLAG_NONFINITE;
    else if (fabsf(v[k]) > amax) amax = fabsf(v[k]);
  }
  if (flags || amax == 0.0f) {
    bits_put(&w, 0);
    return flags;
  }
  int e;
  frexpf(amax, &e);
  if (e < -126) e = -126;
  bits_put(&w, 1);
  for (int k = 0; k < 8; ++k) bits_put(&w, ((e + 127) >> k) & 1);
  int32_t q[16];
  for (int k = 0; k < 16; ++k) q[k] = (int32_t)ldexpf(v[k], 30 - e);  /* exact scaling, truncation */
  for (int j = 0; j < 4; ++j) orc_zfp_fwd4(q + 4 * j, 1);  /* along the channels */
  for (int i = 0; i < 4; ++i) orc_zfp_fwd4(q + i, 4);      /* along the tokens */
  uint32_t u[16];
  for (int k = 0; k < 16; ++k) u[k] = orc_negabinary(q[zfp_order[k]]);
  int n = 0;
  for (int plane = 31; plane >= 0; --plane) {
    for (int c = 0; c < n; ++c)
      if (!bits_put(&w, (u[c] >> plane) & 1)) return flags;
    while (n < 16) {
      int any = 0;
      for (int c = n; c < 16; ++c) any |= (u[c] >> plane) & 1;
      if (!bits_put(&w, any)) return flags;
      if (!any) break;
      for (;;) {
        if (n == 15) {  /* the only candidate left holds the 1 */
          n = 16;
          break;
        }
        int bit = (u[n] >> plane) & 1;
        if (!bits_put(&w, bit)) return flags;
        n++;
        if (bit) break;
      }
    }
  }
  return flags;
}

void orc_zfp_decode_block(const uint8_t* in, int rate, float* v) {
  zfp_make_order();
  orc_bits r = {(uint8_t*)in, 0, 16 * rate};
  int bit;
  for (int k = 0; k < 16; ++k) v[k] = 0.0f;
  if (!bits_get(&r, &bit) || !bit) return;
  int eb = 0;
  for (int k = 0; k < 8; ++k) {
    if (!bits_get(&r, &bit)) return;
    eb |= bit << k;
  }
  const int e = eb - 127;
  uint32_t u[16] = {0};
  int n = 0, done = 0;
  for (int plane = 31; plane >= 0 && !done; --plane) {
    for (int c = 0; c < n && !done; ++c) {
      if (!bits_get(&r, &bit)) done = 1;
      else u[c] |= (uint32_t)bit << plane;
    }
    while (n < 16 && !done) {
      int any;
      if (!bits_get(&r, &any)) { done = 1; break; }
      if (!any) break;
      for (;;) {
        if (n == 15) {
          u[15] |= 1u << plane;
          n = 16;
          break;
        }
        if (!bits_get(&r, &bit)) { done = 1; break; }
        if (bit) u[n] |= 1u << plane;
        n++;
        if (bit) break;
      }
    }
  }
  int32_t q[16];
  for (int k = 0; k < 16; ++k) q[zfp_order[k]] = orc_from_negabinary(u[k]);
  for (int i = 0; i < 4; ++i) orc_zfp_inv4(q + i, 4);
  for (int j = 0; j < 4; ++j) orc_zfp_inv4(q + 4 * j, 1);
  for (int k = 0; k < 16; ++k) v[k] = ldexpf((float)q[k], e - 30);
}

/* ------------------------------------------------------------------------------------------ */
/* Whole-cache encode / decode / rolling append, over the byte layouts of the codec library:  */
/*   X, Xhat     [L][B][H][T][d] contiguous, bf16 bits or binary32                            */
/*   BU codes    [L][B][H][T_cap][d*b/8]  (blocks of n channels, LSB-first streams)           */
/*   BU side     [L][B][H][T_cap/Tb][d/n][2] binary16 (min, scale); Tb = 1: per token         */
/*   BU staging  (Tb > 1) [L][B][H][Tb][d] raw bf16, slot = t mod Tb; a cache holding T       */
/*               tokens quantises the first floor(T / Tb) Tb of them                          */
/*   passthrough [L][B][H][T_cap][d] binary32 z                                               */
/*   KIVI keys   codes [L][B][H][T_cap/G][d][G*b/8], side [L][B][H][T_cap/G][d][2]            */
/*   KIVI values as BU with n = value channel group                                           */
/*   KIVI ring   [L][B][H][W + G][d] raw bf16, slot = t mod (W + G)                           */
/*   zfp-style   codes [L][B][H][T_cap/4][d/4][2 rate] (one 4 x 4 block per 4 tokens x 4        */
/*               channels), no side information                                               */
/* where G is the key token group and W the full-precision window.  For a cache holding T     */
/* tokens, KIVI quantises the first T_q = floor((T - W) / G) G tokens (0 when T < W).         */
/* ------------------------------------------------------------------------------------------ */

typedef struct {
  int backend, bits, n, kg, kvc, win;   /* n: BU block; kg: key token group; kvc: value channel group */
  int bt;                               /* BU tile tokens Tb (1: one token per block) */
  int L, B, H, d, g, T_cap;
} orc_layout;

static int kivi_tq(int T, int win, int kg) { return T < win ? 0 : ((T - win) / kg) * kg; }

static float load_x(const void* X, int x_bf16, size_t idx) {
  return x_bf16 ? orc_bf16_to_f32(((const uint16_t*)X)[idx]) : ((const float*)X)[idx];
}

static int check_layout(const orc_layout* o) {
  if (o->L <= 0 || o->B <= 0 || o->H <= 0 || o->d <= 0 || o->g <= 0 || o->d % o->g) return ORC_EARG;
  if (o->backend == ORC_BACKEND_PASSTHROUGH) return 0;
  if (o->bits < 1 || o->bits > 8) return ORC_EARG;
  if (o->backend == ORC_BACKEND_ZFP) return (o->d % 4 || o->T_cap % 4) ? ORC_EARG : 0;
  if (o->backend == ORC_BACKEND_BLOCK_UNIFORM) {
    if (o->n <= 0 || o->n > 256 || o->d % o->n || (o->n * o->bits) % 8) return ORC_EARG;
    if (o->bt < 1 || o->bt > 256 || o->T_cap % o->bt) return ORC_EARG;
    return 0;
  }
  if (o->backend == ORC_BACKEND_KIVI) {
    if (o->kg <= 0 || o->kg > 256 || o->kvc <= 0 || o->kvc > 256 || o->d % o->kvc || (o->kvc * o->bits) % 8 || (o->kg * o->bits) % 8)
      return ORC_EARG;
    if (o->T_cap % o->kg || o->win < 0) return ORC_EARG;
    return 0;
  }
  return ORC_EARG;
}

/* Block-uniform (or KIVI value, n = channel group) encode of one token vector z[d] into its
 * code row and side row. */
static int encode_row(const float* z, int d, int n, int bits, uint8_t* code_row, uint16_t* side_row) {
  int flags = 0;
  uint8_t q[256];
  int row_block_bytes = n * bits / 8;
  for (int k = 0; k < d / n; ++k) {
    flags |= orc_quantize_block(z + k * n, n, bits, q, &side_row[2 * k], &side_row[2 * k + 1]);
    orc_pack_codes(q, n, bits, code_row + (size_t)k * row_block_bytes);
  }
  return flags;
}

/* Block-uniform token-channel tile: the bt gauge-space rows zt[bt][d] of consecutive tokens
 * share one range per block of n channels (the bt x n values quantised as one block, token
 * by token); each token keeps its own code row, blocks in channel order as for bt = 1. */
static int encode_tile(const float* zt, int bt, int d, int n, int bits, uint8_t* code_rows, uint16_t* side_tile) {
  int flags = 0, row_bytes = d * bits / 8, blk_bytes = n * bits / 8;
  float* vals = (float*)malloc(sizeof(float) * (size_t)bt * n);
  uint8_t* q = (uint8_t*)malloc((size_t)bt * n);
  for (int k = 0; k < d / n; ++k) {
    for (int u = 0; u < bt; ++u)
      for (int c = 0; c < n; ++c) vals[u * n + c] = zt[(size_t)u * d + k * n + c];
    flags |= orc_quantize_block(vals, bt * n, bits, q, &side_tile[2 * k], &side_tile[2 * k + 1]);
    for (int u = 0; u < bt; ++u)
      orc_pack_codes(q + u * n, n, bits, code_rows + (size_t)u * row_bytes + (size_t)k * blk_bytes);
  }
  free(vals); free(q);
  return flags;
}

static void decode_row(const uint8_t* code_row, const uint16_t* side_row, int d, int n, int bits, float* zhat) {
  uint8_t q[256];
  int row_block_bytes = n * bits / 8;
  for (int k = 0; k < d / n; ++k) {
    orc_unpack_codes(code_row + (size_t)k * row_block_bytes, n, bits, q);
    orc_dequantize_block(q, n, side_row[2 * k], side_row[2 * k + 1], zhat + k * n);
  }
}

/* KIVI key group: tokens [grp*G, grp*G + G) of one slice; zt[G][d] gauge-space rows. */
static int encode_key_group(const float* zt, int G, int d, int bits, uint8_t* codes_grp, uint16_t* side_grp) {
  int flags = 0;
  float col[256];
  uint8_t q[256];
  int cbytes = G * bits / 8;
  for (int c = 0; c < d; ++c) {
    for (int t = 0; t < G; ++t) col[t] = zt[(size_t)t * d + c];
    flags |= orc_quantize_block(col, G, bits, q, &side_grp[2 * c], &side_grp[2 * c + 1]);
    orc_pack_codes(q, G, bits, codes_grp + (size_t)c * cbytes);
  }
  return flags;
}

static void decode_key_token(const uint8_t* codes_grp, const uint16_t* side_grp, int G, int d, int bits, int tin,
                             float* zhat) {
  uint8_t q[256];
  float col[256];
  int cbytes = G * bits / 8;
  for (int c = 0; c < d; ++c) {
    orc_unpack_codes(codes_grp + (size_t)c * cbytes, G, bits, q);
    orc_dequantize_block(q, G, side_grp[2 * c], side_grp[2 * c + 1], col);
    zhat[c] = col[tin];
  }
}

static size_t slice_index(const orc_layout* o, int l, int b, int h) { return ((size_t)l * o->B + b) * o->H + h; }

/* Flush KIVI ring tokens [t_begin, t_begin + G) of one slice into the quantised store. */
static int kivi_flush(const orc_layout* o, int s, size_t sl, const float* Gs, int t_begin, uint8_t* codes,
                      uint16_t* side, const uint16_t* ring) {
  int d = o->d, G = o->kg, ringsz = o->win + o->kg;
  int flags = 0;
  float* x = (float*)malloc(sizeof(float) * d);
  float* zt = (float*)malloc(sizeof(float) * (size_t)G * d);
  for (int t = 0; t < G; ++t) {
    int tok = t_begin + t;
    const uint16_t* rrow = ring + (sl * ringsz + (size_t)(tok % ringsz)) * d;
    for (int c = 0; c < d; ++c) x[c] = orc_bf16_to_f32(rrow[c]);
    orc_gauge_apply(d, o->g, Gs, x, zt + (size_t)t * d);
  }
  if (s == 0) {
    int grp = t_begin / G, cb = G * o->bits / 8;
    size_t gbase = sl * (o->T_cap / G) + grp;
    flags |= encode_key_group(zt, G, d, o->bits, codes + gbase * d * cb, side + gbase * d * 2);
  } else {
    int row_bytes = d * o->bits / 8, nb = d / o->kvc;
    for (int t = 0; t < G; ++t) {
      size_t row = sl * o->T_cap + (size_t)(t_begin + t);
      flags |= encode_row(zt + (size_t)t * d, d, o->kvc, o->bits, codes + row * row_bytes, side + row * nb * 2);
    }
  }
  free(x); free(zt);
  return flags;
}

/* Quantise the staged tokens [t_begin, t_begin + Tb) of one slice as one tile. */
static int tile_flush(const orc_layout* o, size_t sl, const float* Gs, int t_begin, uint8_t* codes, uint16_t* side,
                      const uint16_t* staging) {
  int d = o->d, bt = o->bt, flags = 0;
  float* x = (float*)malloc(sizeof(float) * d);
  float* zt = (float*)malloc(sizeof(float) * (size_t)bt * d);
  for (int u = 0; u < bt; ++u) {
    const uint16_t* srow = staging + (sl * bt + (size_t)((t_begin + u) % bt)) * d;
    for (int c = 0; c < d; ++c) {
      x[c] = orc_bf16_to_f32(srow[c]);
      if (!isfinite(x[c])) flags |= ORC_FLAG_NONFINITE;
    }
    orc_gauge_apply(d, o->g, Gs, x, zt + (size_t)u * d);
  }
  int row_bytes = d * o->bits / 8, nb = d / o->n;
  flags |= encode_tile(zt, bt, d, o->n, o->bits, codes + (sl * o->T_cap + (size_t)t_begin) * row_bytes,
                       side + (sl * (o->T_cap / bt) + (size_t)(t_begin / bt)) * nb * 2);
  free(x); free(zt);
  return flags;
}

/* Encode tokens [t0, t0 + T) of X (s: 0 = keys, 1 = values) into the cache.  KIVI requires
 * t0 == 0: the T tokens form the whole cache, T_q of them quantised, the rest in the ring.
 * Returns the OR of ORC_FLAG_* over all blocks, or a negative error. */
int orc_kv_encode(int backend, int bits, int n, int kg, int kvc, int win, int bt, int s, int L, int B, int H, int T,
                  int d, int g, int x_bf16, const void* X, const float* Gall, int T_cap, void* codes, void* side,
                  void* residual, int t0) {
  orc_layout o = {backend, bits, n, kg, kvc, win, bt, L, B, H, d, g, T_cap};
  if (check_layout(&o) || s < 0 || s > 1 || T < 0 || t0 < 0 || t0 + T > T_cap) return ORC_EARG;
  if (backend == ORC_BACKEND_KIVI && (t0 != 0 || !x_bf16)) return ORC_EARG;
  const int tile = backend == ORC_BACKEND_BLOCK_UNIFORM && bt > 1;
  if (tile && (t0 % bt || !x_bf16)) return ORC_EARG;
  if (backend == ORC_BACKEND_ZFP && (t0 % 4 || T % 4)) return ORC_EARG;
  int R = d / g, flags = 0;
  size_t gsz = (size_t)R * g * g;
  float* x = (float*)malloc(sizeof(float) * d);
  float* z = (float*)malloc(sizeof(float) * d);
  for (int l = 0; l < L; ++l)
    for (int b = 0; b < B; ++b)
      for (int h = 0; h < H; ++h) {
        size_t sl = slice_index(&o, l, b, h);
        const float* Gs = Gall + (((size_t)l * 2 + s) * H + h) * gsz;
        size_t xbase = sl * (size_t)T * d;
        if (backend == ORC_BACKEND_KIVI) {
          int tq = kivi_tq(T, win, kg), ringsz = win + kg;
          uint16_t* ring = (uint16_t*)residual;
          for (int t = tq; t < T; ++t)
            memcpy(ring + (sl * ringsz + (size_t)(t % ringsz)) * d, (const uint16_t*)X + xbase + (size_t)t * d,
                   sizeof(uint16_t) * d);
          /* quantised part: same arithmetic as a flush, reading X instead of the ring */
          float* zt = (float*)malloc(sizeof(float) * (size_t)kg * d);
          for (int t = 0; t < tq; t += kg) {
            for (int u = 0; u < kg; ++u) {
              for (int c = 0; c < d; ++c) x[c] = load_x(X, 1, xbase + (size_t)(t + u) * d + c);
              orc_gauge_apply(d, g, Gs, x, zt + (size_t)u * d);
            }
            if (s == 0) {
              int cb = kg * bits / 8;
              size_t gbase = sl * (T_cap / kg) + t / kg;
              flags |= encode_key_group(zt, kg, d, bits, (uint8_t*)codes + gbase * d * cb,
                                        (uint16_t*)side + gbase * d * 2);
            } else {
              int row_bytes = d * bits / 8, nb = d / kvc;
              for (int u = 0; u < kg; ++u) {
                size_t row = sl * T_cap + (size_t)(t + u);
                flags |= encode_row(zt + (size_t)u * d, d, kvc, bits, (uint8_t*)codes + row * row_bytes,
                                    (uint16_t*)side + row * nb * 2);
              }
            }
          }
          free(zt);
          continue;
        }
        if (tile) {
          /* whole tiles quantised (positions t0 + [0, T_q)), the unfinished one staged raw;
           * as for the KIVI window, staged tokens are checked when their tile is quantised */
          int tq = (T / bt) * bt;
          uint16_t* staging = (uint16_t*)residual;
          for (int t = tq; t < T; ++t)
            memcpy(staging + (sl * bt + (size_t)((t0 + t) % bt)) * d, (const uint16_t*)X + xbase + (size_t)t * d,
                   sizeof(uint16_t) * d);
          float* zt = (float*)malloc(sizeof(float) * (size_t)bt * d);
          for (int t = 0; t < tq; t += bt) {
            for (int u = 0; u < bt; ++u) {
              for (int c = 0; c < d; ++c) x[c] = load_x(X, 1, xbase + (size_t)(t + u) * d + c);
              for (int c = 0; c < d; ++c)
                if (!isfinite(x[c])) flags |= ORC_FLAG_NONFINITE;
              orc_gauge_apply(d, g, Gs, x, zt + (size_t)u * d);
            }
            int row_bytes = d * bits / 8, nb = d / n;
            flags |= encode_tile(zt, bt, d, n, bits, (uint8_t*)codes + (sl * T_cap + (size_t)(t0 + t)) * row_bytes,
                                 (uint16_t*)side + (sl * (T_cap / bt) + (size_t)((t0 + t) / bt)) * nb * 2);
          }
          free(zt);
          continue;
        }
        if (backend == ORC_BACKEND_ZFP) {
          /* 4-token groups: gauge each token, then one block per 4 channels */
          float* zt = (float*)malloc(sizeof(float) * 4 * (size_t)d);
          const int bb = 2 * bits;
          for (int t = 0; t < T; t += 4) {
            for (int u = 0; u < 4; ++u) {
              for (int c = 0; c < d; ++c) x[c] = load_x(X, x_bf16, xbase + (size_t)(t + u) * d + c);
              orc_gauge_apply(d, g, Gs, x, zt + (size_t)u * d);
            }
            size_t grp = sl * (T_cap / 4) + (size_t)((t0 + t) / 4);
            for (int cb = 0; cb < d / 4; ++cb) {
              float v[16];
              for (int j = 0; j < 4; ++j)
                for (int i = 0; i < 4; ++i) v[4 * j + i] = zt[(size_t)j * d + 4 * cb + i];
              flags |= orc_zfp_encode_block(v, bits, (uint8_t*)codes + (grp * (d / 4) + cb) * bb);
            }
          }
          free(zt);
          continue;
        }
        for (int t = 0; t < T; ++t) {
          for (int c = 0; c < d; ++c) x[c] = load_x(X, x_bf16, xbase + (size_t)t * d + c);
          for (int c = 0; c < d; ++c)
            if (!isfinite(x[c])) flags |= ORC_FLAG_NONFINITE;
          orc_gauge_apply(d, g, Gs, x, z);
          size_t row = sl * T_cap + (size_t)(t0 + t);
          if (backend == ORC_BACKEND_PASSTHROUGH) {
            memcpy((float*)codes + row * d, z, sizeof(float) * d);
          } else {
            int row_bytes = d * bits / 8, nb = d / n;
            flags |= encode_row(z, d, n, bits, (uint8_t*)codes + row * row_bytes, (uint16_t*)side + row * nb * 2);
          }
        }
      }
  free(x); free(z);
  return flags;
}

/* Decode tokens [t0, t0 + Tout) of every slice into Xhat[L][B][H][Tout][d] (bf16 bits when
 * out_bf16, else binary32).  KIVI and token-channel tiles need the number of tokens the cache
 * holds for each batch row, lens[b]; tokens at or beyond lens[b] are left untouched.  lens
 * may be NULL for the other backends. */
int orc_kv_decode(int backend, int bits, int n, int kg, int kvc, int win, int bt, int s, int L, int B, int H, int d,
                  int g, const float* Gall, int T_cap, const void* codes, const void* side, const void* residual,
                  const int* lens, int t0, int Tout, int out_bf16, void* Xhat) {
  orc_layout o = {backend, bits, n, kg, kvc, win, bt, L, B, H, d, g, T_cap};
  if (check_layout(&o) || s < 0 || s > 1 || t0 < 0 || Tout < 0 || t0 + Tout > T_cap) return ORC_EARG;
  const int tile = backend == ORC_BACKEND_BLOCK_UNIFORM && bt > 1;
  if ((backend == ORC_BACKEND_KIVI || tile) && !lens) return ORC_EARG;
  if (backend == ORC_BACKEND_ZFP && (t0 % 4 || Tout % 4)) return ORC_EARG;
  int R = d / g;
  size_t gsz = (size_t)R * g * g;
  float* zh = (float*)malloc(sizeof(float) * d);
  float* xh = (float*)malloc(sizeof(float) * d);
  if (backend == ORC_BACKEND_ZFP) {
    float* zt = (float*)malloc(sizeof(float) * 4 * (size_t)d);
    const int bb = 2 * bits;
    for (int l = 0; l < L; ++l)
      for (int b = 0; b < B; ++b)
        for (int h = 0; h < H; ++h) {
          size_t sl = slice_index(&o, l, b, h);
          const float* Gs = Gall + (((size_t)l * 2 + s) * H + h) * gsz;
          int len = lens ? lens[b] : T_cap;
          for (int u0 = 0; u0 < Tout; u0 += 4) {
            size_t grp = sl * (T_cap / 4) + (size_t)((t0 + u0) / 4);
            for (int cb = 0; cb < d / 4; ++cb) {
              float v[16];
              orc_zfp_decode_block((const uint8_t*)codes + (grp * (d / 4) + cb) * bb, bits, v);
              for (int j = 0; j < 4; ++j)
                for (int i = 0; i < 4; ++i) zt[(size_t)j * d + 4 * cb + i] = v[4 * j + i];
            }
            for (int j = 0; j < 4; ++j) {
              if (t0 + u0 + j >= len) continue;
              orc_gauge_inverse(d, g, Gs, zt + (size_t)j * d, xh);
              size_t obase = (sl * (size_t)Tout + u0 + j) * d;
              for (int c = 0; c < d; ++c) {
                if (out_bf16) ((uint16_t*)Xhat)[obase + c] = orc_f32_to_bf16(xh[c]);
                else ((float*)Xhat)[obase + c] = xh[c];
              }
            }
          }
        }
    free(zt); free(zh); free(xh);
    return 0;
  }
  for (int l = 0; l < L; ++l)
    for (int b = 0; b < B; ++b)
      for (int h = 0; h < H; ++h) {
        size_t sl = slice_index(&o, l, b, h);
        const float* Gs = Gall + (((size_t)l * 2 + s) * H + h) * gsz;
        int len = lens ? lens[b] : T_cap;
        int tq = backend == ORC_BACKEND_KIVI ? kivi_tq(len, win, kg) : (tile ? (len / bt) * bt : len);
        for (int u = 0; u < Tout; ++u) {
          int t = t0 + u;
          if (t >= len) continue;
          size_t obase = (sl * (size_t)Tout + u) * d;
          if ((backend == ORC_BACKEND_KIVI || tile) && t >= tq) {
            const int slots = tile ? bt : win + kg;
            const uint16_t* rrow = (const uint16_t*)residual + (sl * (size_t)slots + (size_t)(t % slots)) * d;
            for (int c = 0; c < d; ++c) {
              if (out_bf16) ((uint16_t*)Xhat)[obase + c] = rrow[c];
              else ((float*)Xhat)[obase + c] = orc_bf16_to_f32(rrow[c]);
            }
            continue;
          }
          size_t row = sl * T_cap + (size_t)t;
          if (backend == ORC_BACKEND_PASSTHROUGH) {
            memcpy(zh, (const float*)codes + row * d, sizeof(float) * d);
          } else if (backend == ORC_BACKEND_BLOCK_UNIFORM) {
            int row_bytes = d * bits / 8, nb = d / n;
            size_t srow = sl * (T_cap / bt) + (size_t)(t / bt);
            decode_row((const uint8_t*)codes + row * row_bytes, (const uint16_t*)side + srow * nb * 2, d, n, bits, zh);
          } else if (s == 0) {
            int cb = kg * bits / 8;
            size_t gbase = sl * (T_cap / kg) + t / kg;
            decode_key_token((const uint8_t*)codes + gbase * d * cb, (const uint16_t*)side + gbase * d * 2, kg, d,
                             bits, t % kg, zh);
          } else {
            int row_bytes = d * bits / 8, nb = d / kvc;
            decode_row((const uint8_t*)codes + row * row_bytes, (const uint16_t*)side + row * nb * 2, d, kvc, bits,
                       zh);
          }
          orc_gauge_inverse(d, g, Gs, zh, xh);
          for (int c = 0; c < d; ++c) {
            if (out_bf16) ((uint16_t*)Xhat)[obase + c] = orc_f32_to_bf16(xh[c]);
            else ((float*)Xhat)[obase + c] = xh[c];
          }
        }
      }
  free(zh); free(xh);
  return 0;
}

/* Rolling step (section 4.4: every new KV token passes through gauge, backend, decode and
 * inverse gauge): append the token Xnew[L][B][H][d] at position pos[b] of each batch row.
 * Block-uniform (one token per block) / passthrough encode it in place; KIVI puts it in the
 * ring and, when the cache then holds T = pos + 1 tokens with T - W a positive multiple of G,
 * gauges and quantises the G oldest ring tokens [T - W - G, T - W); token-channel tiles stage
 * it and quantise the tile once its Tb-th token arrives. */
int orc_kv_append(int backend, int bits, int n, int kg, int kvc, int win, int bt, int s, int L, int B, int H, int d,
                  int g, int x_bf16, const void* Xnew, const float* Gall, int T_cap, void* codes, void* side,
                  void* residual, const int* pos) {
  orc_layout o = {backend, bits, n, kg, kvc, win, bt, L, B, H, d, g, T_cap};
  if (check_layout(&o) || s < 0 || s > 1) return ORC_EARG;
  const int tile = backend == ORC_BACKEND_BLOCK_UNIFORM && bt > 1;
  if ((backend == ORC_BACKEND_KIVI || tile) && !x_bf16) return ORC_EARG;
  if (backend == ORC_BACKEND_ZFP) return ORC_EARG;  /* whole 4-token groups only */
  for (int b = 0; b < B; ++b)
    if (pos[b] < 0 || pos[b] >= T_cap) return ORC_EARG;
  int R = d / g, flags = 0;
  size_t gsz = (size_t)R * g * g;
  float* x = (float*)malloc(sizeof(float) * d);
  float* z = (float*)malloc(sizeof(float) * d);
  for (int l = 0; l < L; ++l)
    for (int b = 0; b < B; ++b)
      for (int h = 0; h < H; ++h) {
        size_t sl = slice_index(&o, l, b, h);
        const float* Gs = Gall + (((size_t)l * 2 + s) * H + h) * gsz;
        size_t xin = sl * (size_t)d;
        int t = pos[b];
        if (backend == ORC_BACKEND_KIVI) {
          int ringsz = win + kg;
          uint16_t* ring = (uint16_t*)residual;
          memcpy(ring + (sl * ringsz + (size_t)(t % ringsz)) * d, (const uint16_t*)Xnew + xin, sizeof(uint16_t) * d);
          int T = t + 1;
          if (T - win >= kg && (T - win) % kg == 0)
            flags |= kivi_flush(&o, s, sl, Gs, T - win - kg, (uint8_t*)codes, (uint16_t*)side, ring);
          continue;
        }
        if (tile) {
          uint16_t* staging = (uint16_t*)residual;
          memcpy(staging + (sl * bt + (size_t)(t % bt)) * d, (const uint16_t*)Xnew + xin, sizeof(uint16_t) * d);
          if ((t + 1) % bt == 0) flags |= tile_flush(&o, sl, Gs, t + 1 - bt, (uint8_t*)codes, (uint16_t*)side, staging);
          continue;
        }
        for (int c = 0; c < d; ++c) x[c] = load_x(Xnew, x_bf16, xin + c);
        for (int c = 0; c < d; ++c)
          if (!isfinite(x[c])) flags |= ORC_FLAG_NONFINITE;
        orc_gauge_apply(d, g, Gs, x, z);
        size_t row = sl * T_cap + (size_t)t;
        if (backend == ORC_BACKEND_PASSTHROUGH) {
          memcpy((float*)codes + row * d, z, sizeof(float) * d);
        } else {
          int row_bytes = d * bits / 8, nb = d / n;
          flags |= encode_row(z, d, n, bits, (uint8_t*)codes + row * row_bytes, (uint16_t*)side + row * nb * 2);
        }
      }
  free(x); free(z);
  return flags;
}
