/* Driver for the sanitizer build of the CPU oracle (test infrastructure): exercises every oracle
 * entry point on small ragged inputs (all gauge kinds, every backend, sub-range decodes, rolling
 * appends, the zfp-style block coder) so that an AddressSanitizer / UndefinedBehaviorSanitizer
 * build reports any out-of-bounds access, leak or undefined operation.  Exits 0 when every call
 * returned as expected. */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

int orc_gauge_make(int kind, int L, int H, int d, int g, uint64_t seed, const float* params, float* G);
double orc_orthogonality_error(int g, const float* G);
int orc_quantize_block(const float* z, int n, int bits, uint8_t* q, uint16_t* mn_bits, uint16_t* sc_bits);
void orc_dequantize_block(const uint8_t* q, int n, uint16_t mn_bits, uint16_t sc_bits, float* zhat);
void orc_pack_codes(const uint8_t* q, int n, int bits, uint8_t* out);
void orc_unpack_codes(const uint8_t* in, int n, int bits, uint8_t* q);
int orc_zfp_encode_block(const float* v, int rate, uint8_t* out);
void orc_zfp_decode_block(const uint8_t* in, int rate, float* v);
int orc_kv_encode(int backend, int bits, int n, int kg, int kvc, int win, int bt, int s, int L, int B, int H, int T,
                  int d, int g, int x_bf16, const void* X, const float* Gall, int T_cap, void* codes, void* side,
                  void* residual, int t0);
int orc_kv_decode(int backend, int bits, int n, int kg, int kvc, int win, int bt, int s, int L, int B, int H, int d,
                  int g, const float* Gall, int T_cap, const void* codes, const void* side, const void* residual,
                  const int* lens, int t0, int Tout, int out_bf16, void* Xhat);
int orc_kv_append(int backend, int bits, int n, int kg, int kvc, int win, int bt, int s, int L, int B, int H, int d,
                  int g, int x_bf16, const void* Xnew, const float* Gall, int T_cap, void* codes, void* side,
                  void* residual, const int* pos);

static uint64_t rng = 0x9E3779B97F4A7C15ull;
static double uniform(void) {
  rng ^= rng << 13; rng ^= rng >> 7; rng ^= rng << 17;
  return (double)(rng >> 11) * (1.0 / 9007199254740992.0);
}
static uint16_t bf16_of(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  return (uint16_t)(u >> 16);
}

static int failures = 0;
#define EXPECT(c) do { if (!(c)) { fprintf(stderr, "line %d: %s\n", __LINE__, #c); ++failures; } } while (0)

/* one cache of each backend: encode T tokens (twice: whole and from an offset), decode a
 * sub-range with per-row lengths, append a few tokens at per-row positions */
static void codec_case(int backend, int bits, int n, int bt, int d, int g, int T, int T_cap, int x_bf16) {
  const int L = 2, B = 2, H = 2, kg = 32, kvc = 64 < d ? 64 : d, win = 64;
  const int R = d / g;
  float* G = malloc(sizeof(float) * (size_t)L * 2 * H * R * g * g);
  EXPECT(orc_gauge_make(1, L, H, d, g, 7, NULL, G) == 0);
  const size_t nel = (size_t)L * B * H * T * d;
  void* X = malloc(nel * 4);
  for (size_t i = 0; i < nel; ++i) {
    const float v = (float)(uniform() * 4.0 - 2.0);
    if (x_bf16) ((uint16_t*)X)[i] = bf16_of(v);
    else ((float*)X)[i] = v;
  }
  for (int s = 0; s < 2; ++s) {
    const size_t slices = (size_t)L * B * H;
    size_t ncodes, nside = 0, nres = 0;
    if (backend == 0) ncodes = slices * T_cap * d * 4;
    else if (backend == 3) ncodes = slices * (T_cap / 4) * (d / 4) * 2 * bits;
    else if (backend == 2 && s == 0) ncodes = slices * (T_cap / kg) * d * kg * bits / 8;
    else ncodes = slices * T_cap * d * bits / 8;
    if (backend == 1) nside = slices * (T_cap / bt) * (d / n) * 4;
    if (backend == 2) nside = s == 0 ? slices * (T_cap / kg) * d * 4 : slices * T_cap * (d / kvc) * 4;
    if (backend == 2) nres = slices * (win + kg) * d * 2;
    if (backend == 1 && bt > 1) nres = slices * bt * d * 2;
    uint8_t* codes = calloc(ncodes, 1);
    uint8_t* side = nside ? calloc(nside, 1) : NULL;
    uint8_t* res = nres ? calloc(nres, 1) : NULL;
    EXPECT(orc_kv_encode(backend, bits, n, kg, kvc, win, bt, s, L, B, H, T, d, g, x_bf16, X, G, T_cap, codes, side,
                         res, 0) >= 0);
    if (backend != 2) {  /* a second encode from an offset (KIVI encodes whole caches) */
      const int t0 = backend == 3 ? 4 : bt;
      const size_t part = (size_t)L * B * H * (T - t0 - (backend == 3 ? (T - t0) % 4 : 0));
      (void)part;
      int T2 = T - t0;
      if (backend == 3) T2 -= T2 % 4;
      if (bt > 1) T2 -= 0;
      void* X2 = malloc((size_t)L * B * H * T2 * d * (x_bf16 ? 2 : 4));
      for (size_t i = 0; i < (size_t)L * B * H * T2 * d; ++i) {
        if (x_bf16) ((uint16_t*)X2)[i] = ((uint16_t*)X)[i];
        else ((float*)X2)[i] = ((float*)X)[i];
      }
      EXPECT(orc_kv_encode(backend, bits, n, kg, kvc, win, bt, s, L, B, H, T2, d, g, x_bf16, X2, G, T_cap, codes,
                           side, res, t0) >= 0);
      free(X2);
    }
    const int lens[2] = {T, T - 9};
    const int t0 = backend == 3 ? 4 : 5, Tout = backend == 3 ? 16 : T - 7;
    void* Y = malloc((size_t)L * B * H * Tout * d * 4);
    EXPECT(orc_kv_decode(backend, bits, n, kg, kvc, win, bt, s, L, B, H, d, g, G, T_cap, codes, side, res,
                         backend == 3 ? NULL : lens, t0, Tout, 0, Y) == 0);
    EXPECT(orc_kv_decode(backend, bits, n, kg, kvc, win, bt, s, L, B, H, d, g, G, T_cap, codes, side, res,
                         backend == 3 ? NULL : lens, t0, Tout, 1, Y) == 0);
    free(Y);
    if (backend != 3 && T + 3 <= T_cap) {
      uint16_t* xn = malloc((size_t)L * B * H * d * 2);
      float* xf = malloc((size_t)L * B * H * d * 4);
      for (size_t i = 0; i < (size_t)L * B * H * d; ++i) {
        xf[i] = (float)(uniform() - 0.5);
        xn[i] = bf16_of(xf[i]);
      }
      for (int k = 0; k < 3; ++k) {
        const int pos[2] = {T + k, T - 1 + k};
        EXPECT(orc_kv_append(backend, bits, n, kg, kvc, win, bt, s, L, B, H, d, g, x_bf16, x_bf16 ? (void*)xn : (void*)xf,
                             G, T_cap, codes, side, res, pos) >= 0);
      }
      free(xn);
      free(xf);
    }
    free(codes);
    free(side);
    free(res);
  }
  free(X);
  free(G);
}

int main(void) {
  /* gauges */
  for (int kind = 0; kind <= 3; ++kind) {
    float* G = malloc(sizeof(float) * 2 * 2 * 2 * 4 * 16 * 16);
    EXPECT(orc_gauge_make(kind, 2, 2, 64, 16, 3, NULL, G) == 0);
    EXPECT(orc_orthogonality_error(16, G) < 1e-6);
    free(G);
  }
  {
    float* A = calloc(2 * 2 * 4 * 8 * 8, sizeof(float));
    float* G = malloc(sizeof(float) * 2 * 2 * 4 * 8 * 8);
    for (int i = 0; i < 2 * 2 * 4 * 64; ++i) A[i] = (float)(uniform() - 0.5);
    EXPECT(orc_gauge_make(4, 1, 2, 32, 8, 0, A, G) == 0);
    EXPECT(orc_gauge_make(5, 1, 2, 32, 8, 0, G, A) == 0);
    free(A);
    free(G);
  }
  /* quantiser and packing at every width, ragged n */
  const int widths[5] = {2, 3, 4, 6, 8};
  for (int wi = 0; wi < 5; ++wi) {
    float z[37], zh[37];
    uint8_t q[37], q2[37], packed[64];
    uint16_t mn, sc;
    for (int i = 0; i < 37; ++i) z[i] = (float)(uniform() * 10.0 - 5.0);
    orc_quantize_block(z, 32, widths[wi], q, &mn, &sc);
    orc_dequantize_block(q, 32, mn, sc, zh);
    orc_pack_codes(q, 32, widths[wi], packed);
    orc_unpack_codes(packed, 32, widths[wi], q2);
    EXPECT(memcmp(q, q2, 32) == 0);
  }
  /* zfp-style block coder at every rate */
  for (int rate = 1; rate <= 32; ++rate) {
    float v[16], w[16];
    uint8_t code[64];
    for (int i = 0; i < 16; ++i) v[i] = (float)(uniform() * 100.0 - 50.0);
    orc_zfp_encode_block(v, rate, code);
    orc_zfp_decode_block(code, rate, w);
  }
  /* codec round trips: passthrough, block-uniform (per token, tiles), KIVI, zfp-style */
  codec_case(0, 8, 64, 1, 64, 16, 37, 48, 0);
  codec_case(1, 4, 32, 1, 64, 16, 37, 48, 0);
  codec_case(1, 3, 64, 1, 128, 32, 45, 64, 1);
  codec_case(1, 6, 64, 1, 128, 128, 45, 64, 1);
  codec_case(1, 4, 64, 16, 128, 32, 40, 64, 1);
  codec_case(2, 3, 64, 1, 128, 32, 150, 192, 1);
  codec_case(2, 4, 64, 1, 128, 8, 70, 128, 1);
  codec_case(3, 4, 64, 1, 128, 128, 36, 48, 1);
  if (failures) return 1;
  printf("oracle sanitizer driver: ok\n");
  return 0;
}
