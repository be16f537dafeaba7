/*
 * codec_gauge.h - C ABI of the MI355X (gfx950) gauge-coded KV-cache codec.
 *
 * The library implements the codec wrapper of Codec-Gauge ("Learning Compression-Friendly
 * Gauges for Transformer KV Caches"), section 3 (Problem Statement):
 *
 *     Z = G X,   B_c = C(Z),   Zhat = D(B_c),   Xhat = G^{-1} Zhat = G^T Zhat
 *
 * where X is a layer's key or value cache K_l, V_l in R^{B x H x T x d} (section 3), G is a
 * block-diagonal orthogonal gauge with one g x g block G_{l,s,h,r} per (layer l, cache type
 * s in {K, V}, head h, channel group r), R = d / g (section 3, Table 1), G^{-1} = G^T
 * (section 4.1 eq.), and C / D are the compression and decompression maps of a fixed
 * quantisation backend (section 4.3, Compression Conditions): block-uniform ranges, or
 * KIVI-style per-channel key and per-token value ranges.  The gauge mixes channels inside
 * one group of one cached vector only; it never mixes tokens, heads or layers.
 *
 * Conventions shared by every entry point
 *   - Every function returns an int32 status (CG_OK = 0 on success) and never throws.
 *     cg_status_str() names a status.
 *   - All arguments are validated on the host before anything is enqueued; on an error
 *     nothing is launched and nothing is written.
 *   - Device work is enqueued on the caller's HIP stream (`stream`, a hipStream_t; NULL is
 *     the null stream) and the call returns without synchronising.  Kernel faults surface
 *     at the caller's next synchronisation.
 *   - Ownership: every buffer is allocated and freed by the caller.  The library keeps no
 *     pointer after a call returns, allocates no device memory in these entry points and
 *     holds no global state, so calls are reentrant; calls that write the same cache
 *     buffers on different streams race.
 *   - err_flag (optional, may be NULL): a caller-owned device int32 that kernels OR with
 *     CG_FLAG_* bits when they meet a non-finite input, a side-info value that overflows
 *     binary16, or an append position outside the cache.  The library never clears it.
 *   - Device pointers must be 16-byte aligned (CG_ERR_ALIGN otherwise).  A view with T = 0
 *     touches no memory and may carry a NULL pointer.
 *   - Tensors: element (l, b, h, t, c) of a cg_kv_view sits at
 *     ptr + l*stride_l + b*stride_b + h*stride_h + t*stride_t + c (strides in elements,
 *     channel stride 1); strides must keep 16-byte alignment of every row.
 *
 * Byte layouts of a compressed cache (one cg_cache per cache type s; a library contract,
 * the paper leaves the packing format unstated):
 *   block-uniform   codes [L][B][H][T_cap][d*b/8] bytes: the d/n blocks of one token in
 *                   channel order, each an LSB-first stream of n b-bit codes (bit k of a
 *                   stream is bit k mod b of code floor(k/b); stream bit k is bit k%8 of
 *                   byte k/8); side [L][B][H][T_cap/Tb][d/n][2] binary16 (min, scale), one
 *                   pair per block of n channels over Tb consecutive tokens (Tb = block_t;
 *                   Tb = 1: per token).  With Tb > 1, staging [L][B][H][Tb][d] raw bf16
 *                   (the residual buffer) holds the tokens of the unfinished tile, token t
 *                   in slot t mod Tb: a cache holding T tokens quantises the first
 *                   floor(T/Tb) * Tb of them.
 *   KIVI keys       codes [L][B][H][T_cap/Gk][d][Gk*b/8]: per channel, the LSB-first stream
 *                   of the Gk tokens of one token group; side [L][B][H][T_cap/Gk][d][2].
 *   KIVI values     as block-uniform with n = val_channels.
 *   KIVI window     residual [L][B][H][W+Gk][d] raw bf16, token t in slot t mod (W+Gk).
 *                   A KIVI cache holding T tokens quantises the first
 *                   T_q = floor((T - W)/Gk) * Gk of them (0 when T < W); the rest stay in
 *                   the window.
 *   passthrough     codes [L][B][H][T_cap][d] binary32 z (the error-free backend of the
 *                   paper's no-compression sanity rows, section 4.4).
 *   zfp-style       codes [L][B][H][T_cap/4][d/4][2*b] bytes: one fixed-rate block of 16*b
 *                   bits (LSB-first) per 4 consecutive tokens x 4 consecutive channels of z,
 *                   the 2-D field with x = channel and y = token of the paper's zfp setup
 *                   (section 4.3: n_x = d_l); no side or residual buffer.  A block is coded
 *                   as zfp's published algorithm describes: a 0 bit for an all-zero block,
 *                   else a 1 bit and the 8-bit biased block exponent e (|z| < 2^e, e >= -126),
 *                   the values as 30-bit integers trunc(z 2^(30-e)), the 4-point transform
 *                   1/16 [[4 4 4 4] [5 1 -1 -5] [-4 4 4 -4] [-2 6 -6 2]] by integer lifting
 *                   along channels then tokens, coefficients in sequency order (i + j, then
 *                   i^2 + j^2, then the token index), negabinary, and bit planes from the top
 *                   (bits of significant coefficients, then group tests with the last
 *                   candidate's 1 implied) until the 16*b bits are spent.  T_cap, t0 and the
 *                   token counts of kv_encode / kv_decode must be multiples of 4; no append,
 *                   no attention.
 *
 * Quantiser (section 4.3; every fp32 operation rounds to nearest even, no fused
 * multiply-add):  mn_h = binary16 rounded toward -inf of the block minimum (+0 for zero),
 * sc_h = binary16 rounded toward +inf of fl32(fl32(max - mn_h) / (2^b - 1)),
 * inv = fl32(1 / sc_h) (0 when sc_h is 0), q = clamp(rint(fl32(fl32(z - mn_h) * inv)),
 * 0, 2^b - 1); decode zhat = fl32(mn_h + q * sc_h).
 */
#ifndef CODEC_GAUGE_H
#define CODEC_GAUGE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* status codes */
enum {
  CG_OK = 0,
  CG_ERR_ARG = 1,             /* NULL pointer, bad enum, inconsistent dimensions */
  CG_ERR_SHAPE = 2,           /* view / cache / gauge shapes disagree */
  CG_ERR_ALIGN = 3,           /* pointer or stride breaks 16-byte alignment */
  CG_ERR_UNSUPPORTED = 4,     /* valid but not implemented (g, b, n, d combination) */
  CG_ERR_NOT_ORTHOGONAL = 5,  /* CG_GAUGE_USER block with max |G G^T - I| > 1e-5 */
  CG_ERR_CAPACITY = 6,        /* token range beyond the cache capacity */
  CG_ERR_DEVICE = 7           /* a HIP runtime call failed */
};

/* device error-flag bits */
enum { CG_FLAG_NONFINITE = 1, CG_FLAG_SIDE_OVERFLOW = 2, CG_FLAG_POS_RANGE = 4 };

/* gauge kinds (section 4.1 and the controls of section 4.3) */
enum {
  CG_GAUGE_IDENTITY = 0,  /* raw coordinates */
  CG_GAUGE_HAAR = 1,      /* sampled orthogonal gauge with the learned gauge's block structure */
  CG_GAUGE_DCT2 = 2,      /* orthonormal DCT-II, row k = frequency k */
  CG_GAUGE_HADAMARD = 3,  /* Sylvester-ordered Hadamard / sqrt(g); g a power of two */
  CG_GAUGE_EXPM = 4,      /* G = exp(A - A^T), params = A (section 4.1 eq.) */
  CG_GAUGE_USER = 5       /* params = G itself (e.g. a trained gauge) */
};

/* backends (section 4.3; ZFP: the zfp-style fixed-rate transform codec, rate = bits) */
enum { CG_BACKEND_PASSTHROUGH = 0, CG_BACKEND_BLOCK_UNIFORM = 1, CG_BACKEND_KIVI = 2, CG_BACKEND_ZFP = 3 };

/* element types of a cg_kv_view */
enum { CG_DTYPE_BF16 = 0, CG_DTYPE_F32 = 1 };

/* Gauge shape: L layers, H KV heads, head dimension d, group size g (R = d / g groups). */
typedef struct cg_gauge_shape {
  int32_t L, H, d, g;
} cg_gauge_shape;

/* Backend parameters.  bits: b in {2,3,4,6,8} (zfp-style: the rate in bits per value).  block_c: block-uniform channel block n
 * (n | d, n * b % 32 == 0).  key_tokens (Gk, KIVI keys: channel ranges over Gk tokens),
 * val_channels (KIVI values: token ranges over that many channels), residual (W, KIVI
 * full-precision window of recent tokens).  block_t: block-uniform tile tokens Tb in
 * {1, 2, 4, 8, 16, 32}; 1 gives one range per n channels of each token vector, Tb > 1 one
 * range per n channels of Tb consecutive tokens (the token-channel tiles of section 4.3,
 * Tb = 16 in the paper's setup), quantised once the tile's last token is there (bf16 input
 * only).  Unused fields are ignored. */
typedef struct cg_codec {
  int32_t backend, bits, block_c, key_tokens, val_channels, residual;
  int32_t block_t;
} cg_codec;

/* A strided view of a KV tensor [L][B][H][T][d] in device memory. */
typedef struct cg_kv_view {
  void* ptr;
  int32_t dtype;                               /* CG_DTYPE_* */
  int32_t L, B, H, T, d;
  int64_t stride_l, stride_b, stride_h, stride_t;  /* in elements */
} cg_kv_view;

/* One compressed K or V cache (device buffers sized by cache_bytes()).  len: tokens every
 * batch row of the cache currently holds (host value, read by kv_decode for KIVI and
 * block-uniform tiles when it is given no per-row lengths, and by kv_attend without lens). */
typedef struct cg_cache {
  void* codes;
  void* side;      /* NULL for passthrough */
  void* residual;  /* KIVI window or tile staging; NULL otherwise */
  int32_t L, B, H, T_cap, d;
  int32_t len;
} cg_cache;

/* Page table of paged caches: batch row b's positions [i P, (i + 1) P) live in cache batch row
 * (pool page) pages[b * max_pages + i], positions [0, P), P = page_size; the cache's batch
 * dimension counts pool pages and its T_cap equals P.  pages: device int32. */
typedef struct cg_page_table {
  const int32_t* pages;
  int32_t max_pages, page_size;
} cg_page_table;

/* Static message for a status code. */
const char* cg_status_str(int32_t status);

/* Bytes of the device gauge buffer gauge_make() fills for this shape (0 if invalid). */
size_t gauge_device_bytes(cg_gauge_shape shp);

/* Builds every gauge block G_{l,s,h,r} (section 3, Table 1) on the host in binary64 and
 * rounds it once to binary32.  kind: CG_GAUGE_*.  seed: random gauges draw block
 * ((l*2+s)*H+h)*R+r from a Philox4x32-10 stream (Box-Muller normals, QR with the sign of
 * R's diagonal folded in).  params: [L][2][H][R][g][g] binary32 host array for EXPM (A) and
 * USER (G), else ignored.  G_host (optional): host array of the same shape receiving G.
 * G_dev (optional): device buffer of gauge_device_bytes(shp) bytes receiving G and the
 * derived forms the kernels read; the copy is enqueued on `stream` and completed before
 * return.  At least one of G_host, G_dev must be non-NULL.
 * Errors: CG_ERR_ARG, CG_ERR_UNSUPPORTED (g must divide d; Hadamard needs a power of two),
 * CG_ERR_NOT_ORTHOGONAL (USER), CG_ERR_ALIGN, CG_ERR_DEVICE. */
int32_t gauge_make(int32_t kind, cg_gauge_shape shp, uint64_t seed, const float* params, float* G_host,
                   void* G_dev, void* stream);

/* Byte sizes of the codes / side / residual buffers of one cache of type s (0 = K,
 * 1 = V) with capacity T_cap tokens (T_cap a multiple of key_tokens for KIVI, of block_t
 * for block-uniform tiles).  Any output pointer may be NULL. */
int32_t cache_bytes(const cg_codec* codec, int32_t s, int32_t L, int32_t B, int32_t H, int32_t T_cap, int32_t d,
                    size_t* codes, size_t* side, size_t* residual);

/* Encode: Z = G X, B_c = C(Z) (section 3) for the X->T tokens of X_s, written at cache
 * positions [t0, t0 + X->T).  s: 0 keys, 1 values.  G_dev: from gauge_make with the same
 * shape.  KIVI requires t0 == 0 and bf16 input: X is the whole cache (T_q tokens
 * quantised, the rest copied to the window).  Block-uniform tiles (block_t = Tb > 1)
 * require t0 % Tb == 0 and bf16 input: the floor(X->T / Tb) whole tiles are quantised and
 * the remaining tokens staged.  out->len is not modified.
 * Errors: CG_ERR_ARG, CG_ERR_SHAPE, CG_ERR_ALIGN, CG_ERR_UNSUPPORTED, CG_ERR_CAPACITY,
 * CG_ERR_DEVICE. */
int32_t kv_encode(int32_t s, const cg_kv_view* X, const void* G_dev, cg_gauge_shape shp, const cg_codec* codec,
                  const cg_cache* out, int32_t t0, int32_t* err_flag, void* stream);

/* Decode: Zhat = D(B_c), Xhat = G^T Zhat (section 3) for cache positions
 * [t0, t0 + Xhat->T) into Xhat (bf16 rounded to nearest even, or binary32).
 * lens (optional): device int32[B], the positions batch row b of the cache holds (the rows of
 * one layer's [B x H x T x d] cache may hold different lengths, section 3), read on the
 * device only: row b writes view rows for positions [t0, min(t0 + Xhat->T, lens[b])) and leaves
 * the rest of its view rows untouched; a length outside [0, T_cap] sets CG_FLAG_POS_RANGE and
 * the row writes nothing.  NULL: every row holds in->len positions.  A KIVI cache of length T
 * quantises its first T_q(T) positions and keeps the rest in the window, a block-uniform tile
 * cache its first floor(T / Tb) * Tb; window and staged positions come back bit for bit.
 * Without lens, KIVI and tile caches require t0 + Xhat->T <= in->len (CG_ERR_CAPACITY).  The
 * zfp-style backend takes no lens (CG_ERR_UNSUPPORTED).  Errors: as kv_encode. */
int32_t kv_decode(int32_t s, const cg_cache* in, const void* G_dev, cg_gauge_shape shp, const cg_codec* codec,
                  const int32_t* lens, int32_t t0, const cg_kv_view* Xhat, int32_t* err_flag, void* stream);

/* Rolling compressed-history step (section 4.4: every new KV token passes through gauge,
 * backend, decode and inverse gauge), for layers [l0, l1):
 *   1. encode the new key and value token of every (layer, b, h) at position pos[b]
 *      (pos: device int32[B], read on the device, never by the host);  KIVI puts it in
 *      the window and, when the cache then holds T = pos[b] + 1 tokens with T - W a
 *      positive multiple of Gk, gauges and quantises the Gk oldest window tokens;
 *      block-uniform tiles stage it and, when it is the last token of its tile
 *      (pos[b] + 1 a multiple of Tb), gauge and quantise the tile;
 *   2. if k_hist / v_hist are non-NULL, decode the history [0, pos[b]] of those layers
 *      into them (tokens beyond pos[b] are left untouched).
 * k_new / v_new: views with L = l1 - l0 and T = 1 (view layer i is cache layer l0 + i).
 * k_hist / v_hist: views with L = l1 - l0 and T = the number of token slots to cover;
 * positions with pos[b] >= T_cap set CG_FLAG_POS_RANGE and skip that batch row.
 * Errors: as kv_encode. */
int32_t kv_append_step(int32_t l0, int32_t l1, const cg_kv_view* k_new, const cg_kv_view* v_new, const int32_t* pos,
                       const void* G_dev, cg_gauge_shape shp, const cg_codec* codec, const cg_cache* kc,
                       const cg_cache* vc, const cg_kv_view* k_hist, const cg_kv_view* v_hist, int32_t* err_flag,
                       void* stream);

/* Bytes of the device workspace kv_spectral_stats needs for this shape and token block
 * (0 if either is invalid). */
size_t spectral_workspace_bytes(cg_gauge_shape shp, int32_t block_t);

/* Codec-facing spectral statistics of the gauge training objective (section 4.2) for the
 * gauge-transformed cache X' = G X of type s (G from G_dev, cache type s = 0 keys, 1 values).
 * X: a view [L][B][H][T][d] with L = shp.L (bf16 or binary32).  The token axis is cut into
 * blocks of block_t = Tb tokens (Tb in {2, 4, 8, 16, 32}; tokens past the last whole block are
 * not used) and every Tb x d block of X' goes through the orthonormal 2-D DCT-II
 * U = C_Tb Z C_d^T (u: token frequency, v: channel-layout frequency; C_N[k][n] =
 * sqrt((k == 0 ? 1 : 2) / N) cos(pi (2n + 1) k / (2N))).  With E_uv the sum of U_uv^2 over a
 * layer's blocks (all batch rows, heads and token blocks) and
 * rho(u, v) = sqrt((u / (Tb - 1))^2 + (v / (d - 1))^2) / sqrt(2), writes per layer l
 *   stats[4 l + 0] = L_freq = sum E rho / (sum E + 1e-12)
 *   stats[4 l + 1] = L_rate = mean over the layer's coefficients of log(1 + |U| / tau)
 *   stats[4 l + 2] = 1 - L_freq (spectral concentration)
 *   stats[4 l + 3] = sum E (the energy of the used tokens of X', G and the DCT being orthogonal)
 * stats: device binary64 [L][4].  energy (optional, may be NULL): device binary64 [L][Tb][d]
 * receiving the energy maps E.  workspace: caller-owned device buffer of
 * spectral_workspace_bytes(shp, block_t) bytes, 16-byte aligned, whose contents the call
 * overwrites (calls sharing one workspace on different streams race).  tau > 0 (the paper
 * uses 0.04).  Errors: CG_ERR_ARG, CG_ERR_SHAPE, CG_ERR_ALIGN, CG_ERR_UNSUPPORTED,
 * CG_ERR_DEVICE. */
int32_t kv_spectral_stats(int32_t s, const cg_kv_view* X, const void* G_dev, cg_gauge_shape shp, int32_t block_t,
                          float tau, void* workspace, double* stats, double* energy, void* stream);

/* Bytes of the device workspace kv_gauge_grad needs for this shape, B batch rows, T tokens and
 * token block (0 if any is invalid or unsupported). */
size_t gauge_grad_workspace_bytes(cg_gauge_shape shp, int32_t B, int32_t T, int32_t block_t);

/* Gradient of the gauge training objective (section 4.2) with respect to the gauge generators
 * of section 4.1 (G = exp(A - A^T) per (layer, cache type, head, group)), for cache type s:
 *   L_train(l) = lambda_f L_freq(l) + lambda_r L_rate(l)   (the statistics of kv_spectral_stats
 *                                                          of X' = G X, per layer l)
 *   grad[l][h][r][i][j] = d L_train(l) / d A[l][s][h][r][i][j]
 * X: a view [L][B][H][T][d] with L = shp.L (bf16 or binary32).  A: device binary32
 * [L][2][H][R][g][g], the generators; G_dev: the gauge buffer gauge_make built from them
 * (CG_GAUGE_EXPM with params A), which the statistics and the pass over X read.  The sign of a
 * coefficient that is exactly 0 counts as 0 in the derivative of |U|.  stats: device binary64
 * [L][4] receiving the statistics as kv_spectral_stats writes them.  grad: device binary64
 * [L][H][R][g][g] (antisymmetric per block).  workspace: caller-owned device buffer of
 * gauge_grad_workspace_bytes(shp, X->B, X->T, block_t) bytes, 16-byte aligned, whose contents
 * the call overwrites (calls sharing one workspace on different streams race).  d a multiple of
 * 16 and at most 128 (CG_ERR_UNSUPPORTED otherwise); block_t and tau as kv_spectral_stats;
 * lambda_f, lambda_r finite (the paper uses 1.0 and 0.02).  Errors: CG_ERR_ARG, CG_ERR_SHAPE,
 * CG_ERR_ALIGN, CG_ERR_UNSUPPORTED, CG_ERR_DEVICE. */
int32_t kv_gauge_grad(int32_t s, const cg_kv_view* X, const float* A, const void* G_dev, cg_gauge_shape shp,
                      int32_t block_t, float tau, float lambda_f, float lambda_r, void* workspace, double* stats,
                      double* grad, void* stream);

/* Bytes of the device workspace kv_attend needs for nl layers, B batch rows, Hq query heads
 * and caches of capacity T_cap (0: no workspace needed, or invalid arguments). */
size_t attend_workspace_bytes(cg_gauge_shape shp, int32_t nl, int32_t B, int32_t Hq, int32_t T_cap);

/* Decode-phase attention over the compressed caches, with the inverse gauge of section 3
 * folded into the consumer instead of decoding Xhat (section 4.1 on where the recovery can go;
 * section 6: the paper times explicit recovery and leaves kernel fusion to deployments).  For
 * layers [l0, l1), batch
 * row b and query head j (KV head h = j / (Hq / H), grouped-query attention):
 *     o = softmax(scale q Khat^T) Vhat  over the positions [0, n_b) the row holds,
 * with Khat, Vhat the caches as kv_decode would return them in binary32.  Computed as
 * s_t = (scale G_K q) . zhat^K_t and o = G_V^T sum_t p_t zhat^V_t (KIVI window and staged tile
 * tokens enter raw), all in binary32; the cached codes are read once and nothing of size T is
 * written.
 * q, out: views [l1 - l0][B][Hq][1][d] (bf16 or binary32; Hq a positive multiple of shp.H);
 * view layer i is cache layer l0 + i.  kc, vc: the K and V caches (same T_cap).  lens: device
 * int32 [B] with n_b = lens[b] (a KIVI or tile cache then quantises the positions a cache of
 * n_b tokens quantises; rows with lens[b] outside [0, T_cap] set CG_FLAG_POS_RANGE and attend
 * to nothing), or NULL: every row holds kc->len (= vc->len) positions.  A row with no positions
 * gets a zero output.  workspace: caller-owned device buffer of
 * attend_workspace_bytes(shp, l1 - l0, B, Hq, T_cap) bytes, 16-byte aligned (may be NULL when
 * that is 0); calls sharing one workspace on different streams race.
 * Errors: CG_ERR_ARG, CG_ERR_SHAPE, CG_ERR_ALIGN, CG_ERR_UNSUPPORTED, CG_ERR_CAPACITY,
 * CG_ERR_DEVICE. */
int32_t kv_attend(int32_t l0, int32_t l1, const cg_kv_view* q, const cg_cache* kc, const cg_cache* vc,
                  const void* G_dev, cg_gauge_shape shp, const cg_codec* codec, const int32_t* lens, float scale,
                  const cg_kv_view* out, void* workspace, int32_t* err_flag, void* stream);

/* kv_attend for callers that cannot allocate device memory (code under HIP graph capture,
 * tight serving loops, harnesses that forbid allocation): the same arguments without the
 * workspace, the same validation, split plan and results (bit for bit).  The partial results of
 * split rows go to a device array the library owns: CG_ATTEND_NOALLOC_SCRATCH_BYTES (32 MiB) per
 * device, created with the library's code object on a device and held until the process ends;
 * the call allocates nothing.  A call whose split plan needs more than that
 * (attend_workspace_bytes over the rows' span) returns CG_ERR_CAPACITY before anything is
 * enqueued.  Every call on a device shares that device's array and every split writes its whole
 * partial before the combine reads it, so nothing carries over between calls, but calls that
 * overlap on one device (different streams, or host threads) race: serialise them.  The device
 * address of the array is looked up once per device on the first call (CG_ERR_DEVICE if that
 * fails).  Errors: as kv_attend, plus CG_ERR_CAPACITY for a plan beyond the scratch. */
#define CG_ATTEND_NOALLOC_SCRATCH_BYTES ((size_t)32 << 20)
int32_t kv_attend_noalloc(int32_t l0, int32_t l1, const cg_kv_view* q, const cg_cache* kc, const cg_cache* vc,
                          const void* G_dev, cg_gauge_shape shp, const cg_codec* codec, const int32_t* lens,
                          float scale, const cg_kv_view* out, int32_t* err_flag, void* stream);

/* Workspace bytes of kv_attend_paged: as attend_workspace_bytes for rows of
 * max_pages * page_size positions. */
size_t attend_paged_workspace_bytes(cg_gauge_shape shp, int32_t nl, int32_t B, int32_t Hq, int32_t max_pages,
                                    int32_t page_size);

/* kv_attend over paged caches (section 6 names paged-KV integration among the deployment
 * specialisations): kc / vc are page pools (block-uniform with block_t = 1, or passthrough;
 * their B counts pages, T_cap = page size, a multiple of 64), batch row b of q reads its
 * positions [0, lens[b]) through the page table (lens: device int32 [B], required).  A row
 * whose length exceeds max_pages * page_size, or whose table sends a position outside the
 * pool, sets CG_FLAG_POS_RANGE (a page outside the pool contributes nothing).  Otherwise as
 * kv_attend.  workspace: attend_paged_workspace_bytes bytes. */
int32_t kv_attend_paged(int32_t l0, int32_t l1, const cg_kv_view* q, const cg_cache* kc, const cg_cache* vc,
                        const cg_page_table* pages, const void* G_dev, cg_gauge_shape shp, const cg_codec* codec,
                        const int32_t* lens, float scale, const cg_kv_view* out, void* workspace, int32_t* err_flag,
                        void* stream);

/* Encode into paged caches: Z = G X, B_c = C(Z) (section 3) for the X->T tokens of every batch
 * row b of X (shape [L][B][H][T][d]), written at row b's positions [t0, t0 + X->T), i.e. into
 * the pool pages the table assigns to them.  t0 % 32 == 0; block-uniform with block_t = 1, or
 * passthrough; runs on the general kernels.  Positions past the table or pages outside the
 * pool set CG_FLAG_POS_RANGE and skip that 32-position tile.  Errors: as kv_encode. */
int32_t kv_encode_paged(int32_t s, const cg_kv_view* X, const cg_page_table* pages, const void* G_dev,
                        cg_gauge_shape shp, const cg_codec* codec, const cg_cache* out, int32_t t0, int32_t* err_flag,
                        void* stream);

/* Rolling append into paged caches (section 4.4 step 1, through the page table): the new key
 * and value token of every (layer, b, h) is encoded at position pos[b] of row b, i.e. at
 * position pos[b] mod page_size of pool page pages[b * max_pages + pos[b] / page_size].
 * Block-uniform with block_t = 1, or passthrough.  Positions past the table or pages outside
 * the pool set CG_FLAG_POS_RANGE and skip that row.  Errors: as kv_append_step. */
int32_t kv_append_paged(int32_t l0, int32_t l1, const cg_kv_view* k_new, const cg_kv_view* v_new, const int32_t* pos,
                        const cg_page_table* pages, const void* G_dev, cg_gauge_shape shp, const cg_codec* codec,
                        const cg_cache* kc, const cg_cache* vc, int32_t* err_flag, void* stream);

/* Device self-test of the two binary32 steps of the quantiser the kernels compute without a
 * division (section 4.3 block range; the oracle divides): which = 0 compares the reciprocal
 * of every positive finite binary16 scale with correctly rounded 1/s; which = 1 compares the
 * block range divided by 2^b - 1, b in {2,3,4,6,8}, with correctly rounded division for every
 * binary32 significand in the lowest four binades, binades 100..103, binade 127 and the top
 * five, and counts the ranges whose binary16 scale (rounded up) would differ; which = 2
 * compares the binary16 roundings toward -inf and +inf (block minimum and scale) that the
 * matrix-core encoder takes from the hardware conversion under a directed rounding mode with
 * the exact software rounding, for every binary32 bit pattern (zeros, subnormals, normals,
 * infinities and NaNs of both signs), and counts the values where either differs.  Adds the
 * number of mismatches to the caller-zeroed device uint64 *mismatches_dev (8-byte aligned)
 * on `stream`; a correct build adds 0.  Errors: CG_ERR_ARG, CG_ERR_ALIGN, CG_ERR_DEVICE. */
int32_t cg_selftest(int32_t which, uint64_t* mismatches_dev, void* stream);

/* Measurement aid, not part of the codec: the HBM ceiling against which the memory-bound
 * kernels' rates are read.  Streams `read_bytes` (a positive multiple of 8192) from device
 * buffer `src` through LDS with the LDS-direct loads and tile ring of the encoder, and writes
 * `write_bytes` (a multiple of 16, may be 0) of data read back from those tiles to device
 * buffer `dst`, the writes spread evenly over the reads, in one kernel on `stream`.  Both
 * buffers are the caller's and 16-byte aligned; `dst`'s contents afterwards are unspecified.
 * Timing the call with events on `stream` gives the rate one pass with that read / write mix
 * can reach.  Errors: CG_ERR_ARG, CG_ERR_ALIGN, CG_ERR_DEVICE. */
int32_t cg_stream_probe(const void* src, int64_t read_bytes, void* dst, int64_t write_bytes, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* CODEC_GAUGE_H */
