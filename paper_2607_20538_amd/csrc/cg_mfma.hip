// Matrix-core codec kernels for bf16 caches with head dimension 128 and the block-uniform
// backend (the configuration the paper's Llama-class KV caches take).
//
// The gauge (section 3: z = G_{l,s,h,r} x per channel group) is a dense contraction over the
// channel axis, so it runs on the gfx950 matrix cores with v_mfma_f32_32x32x16_bf16.  The
// input x is exact in bf16; the binary32 gauge enters as kNP bf16 planes G0 + G1 (+ G2) of
// its split (the gauge buffer holds three), each multiplied on the matrix core with a
// binary32 accumulator.  Two planes carry 16 significant bits of every entry (entry error at
// most 2^-16 relative), which keeps z within a few 1e-6 of the binary32 gauge per group,
// inside the 1e-5 gauge tolerance, at two thirds of the matrix-core work of three planes.
//
// Work split: a workgroup of four wave64s owns a range of 32-token tiles of one
// (layer, batch, head) slice; wave w computes output channels [32w, 32w+32) (one 32-row MFMA
// tile) for the tile's 32 tokens.  The wave keeps its 32 rows of every split plane in VGPRs
// for the whole range, so the matrix core never re-reads G.  Output rows are permuted so
// that lane (token n, half hc) ends up with the 16 consecutive channels 32w + 16hc + [0, 16):
// its codes form one contiguous stretch of the packed row.  Tokens are staged through LDS
// with an XOR swizzle of the 16-byte granules of each 256-byte row, so the B-operand reads
// (lane n reads granule j of row n) hit distinct banks.
//
// Encode epilogue (section 4.3 block-uniform): block minimum / maximum in-lane, across the
// two lane halves (n = 32) and across the wave pair through LDS (n = 64); binary16 side
// information; binary32 quantisation without contraction; LSB-first packing; stores.
//
// Decode: the B operand is the centred integer code q - c, c = 2^(b-1) (exact in bf16), so
// per block k, with the grid midpoint m_k = mn_k + c sc_k,
//   xhat_i = sum_k ( m_k * colsum_k(G^T)_i + sc_k * (G^T (q - c))_{k,i} )
// with block-local accumulation on the matrix core and the column sums of each block
// computed once per workgroup in binary64.  Centring keeps the two terms small when a block
// spans a group whose values sit far from the block's minimum (an outlier in another group
// of the same block), where mn * colsum and sc * G^T q would cancel.
#include <cstdlib>
#include <type_traits>

#include "cg_internal.h"
#include "cg_device.h"
#include "cg_mfma_util.h"
#include "cg_zfp.h"

namespace cg {

namespace {

constexpr int kStages = 5;       // encoder LDS ring: tiles in flight + the one being read

struct MfmaArgs {
  // view (input for encode, output for decode)
  char* x;
  int64_t sl, sb, sh, st;        // element strides
  int L, B, H, T;                // view dims (L = layers of the view)
  int l0;                        // cache layer of view layer 0
  int s;                         // 0 keys, 1 values
  int t0;                        // cache position of view token 0
  // gauge planes ([nblk][g][g] bf16) and binary32 blocks
  const uint16_t* gp[3];
  const float* g32;
  const float* cs8;              // decoder column sums per 8-channel segment [head][d/8][d]
  int g, R;                      // group size, groups per head
  int Hg;                        // heads of the gauge shape
  // cache
  uint8_t* codes;
  uint32_t* side;
  int T_cap, cB, cH;             // cache capacity and dims
  // KIVI: tokens [0, tq) are quantised, [tq, T) go raw into the ring of ring_slots rows;
  // the decoders derive tq from the positions the cache holds (len, or pos[b] + 1)
  int tq, ring_slots;
  uint16_t* ring;
  int kivi, win, kg, len;
  // work split
  int nslices, chunks, tiles_per_wg;
  // decode only: batch row b holds positions [0, pos[b] + pos_add) (rolling step: pos_add = 1,
  // the row's newest position; per-row lengths: pos_add = 0); NULL: every row holds `len`
  const int* pos;
  int pos_add;
  int* err;
};


// Load the wave's A fragments: plane p, K-step kk: 8 bf16 of row `ch` (an output channel of
// this wave) at input channels j0..j0+7 of the full block-diagonal matrix (zero outside the
// row's group).  `tr` selects G^T planes (decode).
template <int NP, int KS>
__device__ void load_a(bf16x8_t (&A)[NP][KS], const MfmaArgs& a, int l, int h, int ch, int kbase, int kh) {
  const int g = a.g;
  const int r = ch / g;
  const size_t blk = ((size_t(l) * 2 + a.s) * a.Hg + h) * a.R + r;
#pragma unroll
  for (int kk = 0; kk < KS; ++kk) {
    const int j0 = kbase + 16 * kk + 8 * kh;
    const bool in_group = (j0 / g) == r;
#pragma unroll
    for (int p = 0; p < NP; ++p) {
      u32x4_t v = {0u, 0u, 0u, 0u};
      if (in_group) v = *(const u32x4_t*)(a.gp[p] + blk * g * g + size_t(ch % g) * g + (j0 % g));
      A[p][kk] = as_bf16x8(v);
    }
  }
}

// Packs 16 codes of BITS bits into 16*BITS/32 words (BITS even) LSB-first.
template <int BITS>
__device__ __forceinline__ void pack16(const uint32_t (&q)[16], uint32_t* out) {
  constexpr int NW = (16 * BITS + 31) / 32;
#pragma unroll
  for (int w = 0; w < NW; ++w) out[w] = 0;
#pragma unroll
  for (int e = 0; e < 16; ++e) {
    const int bit = e * BITS, w = bit >> 5, off = bit & 31;
    out[w] |= q[e] << off;
    if (off + BITS > 32) out[w + 1] |= q[e] >> (32 - off);
  }
}

template <int NW>
__device__ __forceinline__ void store_words(uint32_t* dst, const uint32_t* v) {
  // dst is 4-byte aligned; use the widest aligned vector stores available
  if constexpr (NW == 4) {
    *(u32x4_t*)dst = u32x4_t{v[0], v[1], v[2], v[3]};
  } else if constexpr (NW == 2) {
    *(uint2*)dst = make_uint2(v[0], v[1]);
  } else {
#pragma unroll
    for (int i = 0; i < NW; ++i) dst[i] = v[i];
  }
}

// ------------------------------------------------------------------------------------------
// encode
// ------------------------------------------------------------------------------------------

// z (32 rows x 32 tokens) of one tile: the NP split planes times the tile, one chain.
// TR: the tile as the A operand and the gauge rows as the B operand, so the accumulator holds
// z transposed (lane (n, hc): tokens 8i + 4hc + j of channel row n).
template <int NP, int KS, bool TR = false>
__device__ __forceinline__ f32x16_t mfma_chain(const bf16x8_t (&A)[NP][KS], const bf16x8_t (&Bf)[KS]) {
  f32x16_t acc = {};
#pragma unroll
  for (int kk = 0; kk < KS; ++kk)
#pragma unroll
    for (int p = 0; p < NP; ++p) acc = TR ? mfma(Bf[kk], A[p][kk], acc) : mfma(A[p][kk], Bf[kk], acc);
  return acc;
}


// min / max over the 16 lanes of a DPP row (quad swaps, then rotations by 4 and 8 lanes)
__device__ __forceinline__ float row16_min(float v) {
  v = min_nan(v, dpp_mov<0xB1>(v));   // quad_perm [1,0,3,2]
  v = min_nan(v, dpp_mov<0x4E>(v));   // quad_perm [2,3,0,1]
  v = min_nan(v, dpp_mov<0x124>(v));  // row_ror:4
  return min_nan(v, dpp_mov<0x128>(v));  // row_ror:8
}
__device__ __forceinline__ float row16_max(float v) {
  v = max_nan(v, dpp_mov<0xB1>(v));
  v = max_nan(v, dpp_mov<0x4E>(v));
  v = max_nan(v, dpp_mov<0x124>(v));
  return max_nan(v, dpp_mov<0x128>(v));
}


// 4 x 4 transpose of four-value groups across a DPP quad: lane r (= lane % 4) holds groups
// M[r][c] = z[4c .. 4c+3]; afterwards v[4j .. 4j+3] = M[j][r] (lane j's group r).  Two
// exchanges: slot c takes the partner's slot c ^ d from lane r ^ d where bit d of c ^ r is set
// (d = 1, then 2), which moves M[r ^ (c ^ r)][c ^ (c ^ r)] = M[c][r] into slot c.
__device__ __forceinline__ void quad_transpose(const float (&z)[16], int r, float (&v)[16]) {
  float t[16];
#pragma unroll
  for (int c = 0; c < 4; ++c)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float o = dpp_mov<0xB1>(z[4 * (c ^ 1) + i]);  // quad_perm [1,0,3,2]
      t[4 * c + i] = ((c ^ r) & 1) ? o : z[4 * c + i];
    }
#pragma unroll
  for (int c = 0; c < 4; ++c)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float o = dpp_mov<0x4E>(t[4 * (c ^ 2) + i]);  // quad_perm [2,3,0,1]
      v[4 * c + i] = ((c ^ r) & 2) ? o : t[4 * c + i];
    }
}

// encoder modes
constexpr int kModeBU = 0;     // block-uniform (or KIVI values: n = value channel group)
constexpr int kModePass = 1;   // error-free backend: binary32 z
constexpr int kModeKeys = 2;   // KIVI keys: one block per channel over a 32-token group
constexpr int kModeZfp = 3;    // zfp-style fixed-rate blocks of 4 tokens x 4 channels (BITS = rate)

// Software pipeline over 32-token tiles, one barrier per tile.  Iteration t:
//   1. block-range partials of tile t from its accumulator (64-channel blocks: wave-pair
//      exchange through red[t & 1]);
//   2. wait for tile t+1's LDS-direct loads, barrier, issue the loads of tile t+kStages-1
//      into the buffer tile t-1 used, read the B fragments of tile t+1, write tile t-1's
//      staged codes and side words to the cache as contiguous runs;
//   3. matrix-core chain of tile t+1 interleaved with side info, quantisation and packing of
//      tile t into the staging buffers.
// kStages - 1 tiles are in flight between global memory and LDS.  The codes of a tile are one
// contiguous run of 32 RB bytes in the cache and its side words one run of 32 NBK words, so
// the staged copy leaves with whole-line stores instead of 32 scattered row pieces.
template <int NP, int KS, int BITS, int NB, int MODE, int TB = 1>
__global__ __launch_bounds__(kThreads, NP == 2 ? 3 : 2) void enc_mfma(MfmaArgs a) {
  constexpr bool PASS = MODE == kModePass, KEYS = MODE == kModeKeys, ZFP = MODE == kModeZfp;
  constexpr bool QUANT = !PASS && !ZFP;  // block ranges, staged codes and side words
  // token-channel tiles: one range per TB tokens x NB channels (NB spans whole waves)
  constexpr bool TILE = TB > 1;
  static_assert(!TILE || (TB == 16 && MODE == kModeBU && (NB == 64 || NB == 128)), "tile shape");
  constexpr int RB = kD * BITS / 8;   // packed code bytes per token row
  constexpr int NBK = kD / NB;        // side words per token row (per tile row of tiles)
  // ring depth: the zfp-style coder is bound by its VALU work, so it keeps one tile fewer in
  // flight and gives the LDS to the block transpose below (three workgroups per CU either way)
  constexpr int ST = ZFP ? kStages - 1 : kStages;
  __shared__ __attribute__((aligned(16))) uint8_t xtile[ST][kTok * kRowBytes];
  __shared__ float2 red[2][4][kTok];  // per-wave (min, max) of each token, for 64-channel blocks
  // a tile's packed rows and side words, staged so that they leave as contiguous stores
  __shared__ __attribute__((aligned(16))) uint8_t cstage[2][QUANT ? kTok * RB : 16];
  __shared__ uint32_t sstage[2][QUANT ? kTok * NBK : 1];  // KIVI keys: NB = 32, one word per channel
  __shared__ std::conditional_t<ZFP, ZfpTables, char> ztab;
  // zfp-style: each wave's 32 tokens x 32 channels of z, written by token rows and read back as
  // 4 x 4 blocks by the same wave (LDS operations of a wave complete in order, so no barrier)
  constexpr int QP = 36;  // row pitch in floats (16-byte rows, rows 4 banks apart)
  __shared__ __attribute__((aligned(16))) float zq[ZFP ? 4 : 1][ZFP ? kTok * QP : 4];

  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int n = lane & 31, hc = lane >> 5;
  const int logical = xcd_remap(blockIdx.x, gridDim.x);
  const int slice = logical / a.chunks, chunk = logical - slice * a.chunks;
  if (slice >= a.nslices) return;
  const int h = slice % a.H, b = (slice / a.H) % a.B, lv = slice / (a.H * a.B);
  const int l = lv + a.l0;
  const int ntiles = (a.T + kTok - 1) / kTok;
  const int tb = chunk * a.tiles_per_wg;
  const int te_all = min(ntiles, tb + a.tiles_per_wg);
  if (tb >= te_all) return;
  // tiles below tq / 32 are quantised (tq is a multiple of 32 for KIVI, T otherwise)
  const int te = min(te_all, (a.tq + kTok - 1) / kTok);

  const char* xs = a.x + 2 * (size_t(lv) * a.sl + size_t(b) * a.sb + size_t(h) * a.sh);
  const size_t cslice = (size_t(l) * a.cB + b) * a.cH + h;
  const int64_t tstride = 2 * a.st;  // bytes between tokens

  // KIVI full-precision window / staged tokens of an unfinished tile: this workgroup's rows
  // at or past tq copied raw into the ring (slot = cache position mod ring_slots)
  auto ring_copy = [&]() {
    constexpr int GR = kRowBytes / 16;  // granules per row
    const int r0 = max(a.tq, tb * kTok), r1 = min(a.T, te_all * kTok);
    for (int gi = r0 * GR + int(threadIdx.x); gi < r1 * GR; gi += kThreads) {
      const int row = gi / GR, j = gi % GR;
      uint16_t* dst = a.ring + (cslice * a.ring_slots + (a.t0 + row) % a.ring_slots) * kD;
      *(u32x4_t*)((char*)dst + 16 * j) = *(const u32x4_t*)(xs + int64_t(row) * tstride + 16 * j);
    }
  };
  if (tb >= te) {
    ring_copy();
    return;
  }
  if constexpr (ZFP) zfp_tables_init(ztab);  // read after the prologue's barrier

  // K range of this wave's rows: the group of channels 32w.. (whole head for g = 128)
  const int kbase = a.g >= 32 ? (32 * w / a.g) * a.g : 32 * w;
  // A row m of this wave computes output channel 32w + 16*((m/4)%2) + 4*(m/8) + m%4
  const int chA = 32 * w + 16 * ((n >> 2) & 1) + 4 * (n >> 3) + (n & 3);
  bf16x8_t A[NP][KS];
  load_a<NP, KS>(A, a, l, h, chA, kbase, hc);

  // Tiles stream global -> LDS without VGPRs (LDS-direct loads): wave w moves rows
  // 8w .. 8w+7 of a tile with two 1 KB instructions whose lanes write consecutive 16-byte
  // LDS granules; lane l of instruction q fetches the logical granule that the XOR swizzle
  // puts at physical granule l % 16 of row 8w + 4q + l / 16.
  const int wu = __builtin_amdgcn_readfirstlane(w);  // the wave index as a scalar
  int drow[2];
  const char* dsrc[2];  // this lane's source granule in tile 0
#pragma unroll
  for (int q = 0; q < 2; ++q) {
    drow[q] = 8 * w + 4 * q + (lane >> 4);
    dsrc[q] = xs + drow[q] * tstride + 16 * swz(drow[q], lane & 15);
  }
  auto issue = [&](int tile) {
    uint8_t* dst = xtile[(tile - tb) % ST] + 8 * wu * kRowBytes;
    if ((tile + 1) * kTok <= a.T) {
      const int64_t off = int64_t(tile) * kTok * tstride;
#pragma unroll
      for (int q = 0; q < 2; ++q)
        __builtin_amdgcn_global_load_lds(dsrc[q] + off, (__attribute__((address_space(3))) void*)(dst + 4 * q * kRowBytes),
                                         16, 0, kLoadStreamPolicy);
    } else {
      // ragged last tile: rows past the view repeat its last token
#pragma unroll
      for (int q = 0; q < 2; ++q) {
        const int tok = min(tile * kTok + drow[q], a.T - 1);
        __builtin_amdgcn_global_load_lds(dsrc[q] + (int64_t(tok) - drow[q]) * tstride,
                                         (__attribute__((address_space(3))) void*)(dst + 4 * q * kRowBytes), 16, 0,
                                         kLoadStreamPolicy);
      }
    }
  };
  // Before a barrier: wait until this wave's loads of tile X have landed while the loads of
  // tiles X+1 .. I (the last one issued) may stay in flight, and until its LDS writes are
  // done.  VMEM operations complete in issue order; stores issued after those loads only make
  // the count stricter.
  auto wait_tile = [&](int X, int I) {
    switch (I - X) {
      case 0: __builtin_amdgcn_s_waitcnt(waitcnt_imm(0)); break;
      case 1: __builtin_amdgcn_s_waitcnt(waitcnt_imm(2)); break;
      case 2: __builtin_amdgcn_s_waitcnt(waitcnt_imm(4)); break;
      case 3: __builtin_amdgcn_s_waitcnt(waitcnt_imm(6)); break;
      default: __builtin_amdgcn_s_waitcnt(waitcnt_imm(8)); break;
    }
  };
  int boff[KS];
#pragma unroll
  for (int kk = 0; kk < KS; ++kk) boff[kk] = n * kRowBytes + 16 * swz(n, (kbase >> 3) + 2 * kk + hc);
  bf16x8_t Bf[KS];
  auto bfrags = [&](int tile) {
    const uint8_t* src = xtile[(tile - tb) % ST];
#pragma unroll
    for (int kk = 0; kk < KS; ++kk) Bf[kk] = as_bf16x8(*(const u32x4_t*)(src + boff[kk]));
  };

  // prologue: tiles tb .. tb+ST-2 in flight, tile tb on the matrix core
  for (int t = tb; t < min(te, tb + ST - 1); ++t) issue(t);
  wait_tile(tb, min(te - 1, tb + ST - 2));
  __builtin_amdgcn_s_barrier();
  bfrags(tb);
  f32x16_t acc[2];
  acc[0] = mfma_chain<NP, KS, KEYS>(A, Bf);
  int flags = 0;
  // staged tile -> cache: thread i stores 16-byte granule i of the codes (row i / BITS) and,
  // counting from the last thread, side word i (row i / NBK); rows past the view are skipped
  auto flush = [&](int tile, auto parity) {
    constexpr int P = decltype(parity)::value;
    const int tid = int(threadIdx.x);
    const int nlive = min(a.T, a.tq) - tile * kTok;  // quantised rows of the tile
    const size_t crow0 = cslice * a.T_cap + size_t(a.t0 + tile * kTok);
    if (tid < kTok * BITS && tid / BITS < nlive)
      *(u32x4_t*)(a.codes + crow0 * RB + 16 * tid) = *(const u32x4_t*)(cstage[P] + 16 * tid);
    // side words: one per (row, block), or per (tile of TB rows, block); t0 % TB == 0
    const int si = kThreads - 1 - tid;
    if (si < (kTok / TB) * NBK && (si / NBK) * TB < nlive) a.side[crow0 / TB * NBK + si] = sstage[P][si];
  };
  // one pipeline step; P = parity of (tile - tb) selects the accumulator, LDS buffer, register
  // stage and exchange slot at compile time
  auto step = [&](int tile, auto parity) {
    constexpr int P = decltype(parity)::value;
    float z[16];
#pragma unroll
    for (int e = 0; e < 16; ++e) z[e] = acc[P][e];
    const int tok = tile * kTok + n;
    const bool live = tok < (TILE ? a.tq : a.T);
    const size_t crow = cslice * a.T_cap + size_t(a.t0 + tok);

    // 1. block-range partials (NaN-propagating: a NaN anywhere in the block reaches the range)
    float mn = z[0], mx = z[0];
    if constexpr (QUANT) {
#pragma unroll
      for (int e = 1; e < 16; ++e) {
        mn = min_nan(mn, z[e]);
        mx = max_nan(mx, z[e]);
      }
      if constexpr (TILE) {  // the 16 tokens of the lane's tile: one DPP row
        mn = row16_min(mn);
        mx = row16_max(mx);
      }
      if constexpr (NB >= 32) halves_minmax(mn, mx);
      if constexpr (TILE) {
        if (hc == 0 && (n & 15) == 0) red[P][w][n >> 4] = make_float2(mn, mx);
      } else if constexpr (NB == 64) {
        if (hc == 0) red[P][w][n] = make_float2(mn, mx);
      }
    }
    // 2. tile+1 landed in every wave (and every wave is done with tile-1's buffer), refill
    //    that buffer with tile+ST-1, read tile+1's B fragments
    if (tile + 1 < te) wait_tile(tile + 1, min(te - 1, tile + ST - 2));
    else __builtin_amdgcn_s_waitcnt(waitcnt_imm(63));  // LDS writes only
    __builtin_amdgcn_s_barrier();
    if (tile + ST - 1 < te) issue(tile + ST - 1);
    bfrags(tile + 1);
    if constexpr (QUANT) {
      if (tile > tb) flush(tile - 1, std::integral_constant<int, P ^ 1>());
    }
    // 5. next tile on the matrix core (past the range it reads a stale buffer and is unused),
    //    this tile's epilogue on the VALU; no branch until the stores
    acc[P ^ 1] = mfma_chain<NP, KS, KEYS>(A, Bf);

    if constexpr (ZFP) {
      // the lane's 4 x 4 block of this tile, through the wave's LDS region: tokens
      // 4(n/4) .. +3 x channels 32w + 16hc + 4(n%4) .. +3; range, transform and top planes
      // alongside the chain, then the planes (blocks past the view, at token counts that are
      // multiples of 4, are skipped)
      (void)live;
      float* zw = zq[w];
#pragma unroll
      for (int q = 0; q < 4; ++q)
        *(float4*)(zw + n * QP + 16 * hc + 4 * q) = make_float4(z[4 * q], z[4 * q + 1], z[4 * q + 2], z[4 * q + 3]);
      __builtin_amdgcn_wave_barrier();  // keep the reads after the writes
      float v[16];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const float4 t = *(const float4*)(zw + (4 * (n >> 2) + j) * QP + 16 * hc + 4 * (n & 3));
        v[4 * j] = t.x; v[4 * j + 1] = t.y; v[4 * j + 2] = t.z; v[4 * j + 3] = t.w;
      }
      ZfpPrep zp;
      zfp_prepare(v, zp);
#pragma unroll
      for (int i = 0; i < KS * NP; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x002, 20, 0);
      }
      if (tile * kTok + 4 * (n >> 2) < a.T) {
        uint32_t wd[4];
        flags |= zfp_encode_planes<BITS>(zp, ztab, wd);
        const size_t blk = (cslice * size_t(a.T_cap / 4) + (a.t0 + tile * kTok) / 4 + (n >> 2)) * (kD / 4) +
                           8 * w + 4 * hc + (n & 3);
        zfp_store<BITS>(a.codes + blk * (2 * BITS), wd);
      }
    } else if constexpr (PASS) {
#pragma unroll
      for (int i = 0; i < KS * NP; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x002, 1, 0);
      }
      if (live) {
        float* dst = (float*)a.codes + crow * kD + 32 * w + 16 * hc;
#pragma unroll
        for (int q = 0; q < 4; ++q) *(float4*)(dst + 4 * q) = make_float4(z[4 * q], z[4 * q + 1], z[4 * q + 2], z[4 * q + 3]);
      }
    } else if constexpr (KEYS) {
      // z^T: lane (n, hc) holds tokens 8i + 4hc + j (e = 4i + j) of channel chA; the block is
      // the channel over the tile's 32 tokens (in-lane 16 + the other half-wave's 16)
      const bool bad = !(mn >= -3.0e38f && mx <= 3.0e38f);  // NaN or +-inf in the block
      const Side sd = make_side<true>(mn, mx, BITS);
      // the channel's LSB-first stream of 32 codes in token order (BITS words): this lane's
      // codes placed as if hc = 0 (token 8i + j at bit (8i + j) BITS), shifted by 4 BITS bits
      // for hc = 1, then the two half-wave patterns OR-ed together
      uint32_t words[BITS];
#pragma unroll
      for (int i = 0; i < BITS; ++i) words[i] = 0;
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const uint32_t q = code_u8(quantize_t(z[e], sd.mn, sd.inv));
        const int bit = (8 * (e >> 2) + (e & 3)) * BITS, wd = bit >> 5, off = bit & 31;
        words[wd] |= q << off;
        if (off + BITS > 32) words[wd + 1] |= q >> (32 - off);
      }
      if (hc) {
        constexpr int SH = 4 * BITS;  // <= 32
#pragma unroll
        for (int i = BITS - 1; i >= 0; --i) {
          const uint32_t lo = i > 0 ? words[i - 1] : 0u;
          words[i] = SH == 32 ? lo : ((words[i] << (SH & 31)) | (lo >> ((32 - SH) & 31)));
        }
      }
#pragma unroll
      for (int i = 0; i < BITS; ++i) words[i] |= __shfl_xor(words[i], 32);
#pragma unroll
      for (int i = 0; i < BITS; ++i) asm volatile("" ::"v"(words[i]));
      asm volatile("" ::"v"(sd.word));
#pragma unroll
      for (int i = 0; i < KS * NP; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x002, 6, 0);
      }
      if (hc == 0) {
        store_words<BITS>((uint32_t*)(cstage[P] + chA * 4 * BITS), words);
        sstage[P][chA] = sd.word;
      }
      flags |= sd.flags | (bad ? CG_FLAG_NONFINITE : 0);
    } else {
      if constexpr (TILE) {  // the other waves of the tile's channel block
#pragma unroll
        for (int o = 1; o < NB / 32; ++o) {
          const float2 v = red[P][w ^ o][n >> 4];
          mn = min_nan(mn, v.x);
          mx = max_nan(mx, v.y);
        }
      } else if constexpr (NB == 64) {
        const float2 o = red[P][w ^ 1][n];
        mn = min_nan(mn, o.x);
        mx = max_nan(mx, o.y);
      }
      const bool bad = !(mn >= -3.0e38f && mx <= 3.0e38f);  // NaN or +-inf in the block
      const Side sd = make_side<true>(mn, mx, BITS);
      float r[16];
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        // v_cvt_pk_u8_f32 below rounds to nearest even (packing bytes, or code_u8)
        r[e] = quantize_t(z[e], sd.mn, sd.inv);
      }
      constexpr int NW = (BITS & 1) ? BITS : BITS / 2;  // words this lane stores
      uint32_t words[NW];
      // v_cvt_pk_u8_f32 rounds to nearest even (the quantiser's rint) and saturates to
      // [0, 255] (codes are in [0, 2^b - 1] by construction of the side information); bytes
      // then go to b-bit fields of the LSB-first stream
      auto pk4 = [](float c0, float c1, float c2, float c3) {
        uint32_t v = __builtin_amdgcn_cvt_pk_u8_f32(c0, 0, 0u);
        v = __builtin_amdgcn_cvt_pk_u8_f32(c1, 1, v);
        v = __builtin_amdgcn_cvt_pk_u8_f32(c2, 2, v);
        return __builtin_amdgcn_cvt_pk_u8_f32(c3, 3, v);
      };
      if constexpr (BITS == 8) {
#pragma unroll
        for (int i = 0; i < 4; ++i) words[i] = pk4(r[4 * i], r[4 * i + 1], r[4 * i + 2], r[4 * i + 3]);
      } else if constexpr (BITS == 4) {
        // byte j of the word holds codes 2j (low nibble) and 2j+1 (high nibble)
#pragma unroll
        for (int i = 0; i < 2; ++i) {
          const float* c = r + 8 * i;
          words[i] = pk4(c[0], c[2], c[4], c[6]) | (pk4(c[1], c[3], c[5], c[7]) << 4);
        }
      } else if constexpr (BITS == 2) {
        // byte j holds codes 4j .. 4j+3 in 2-bit fields
        words[0] = pk4(r[0], r[4], r[8], r[12]) | (pk4(r[1], r[5], r[9], r[13]) << 2) |
                   (pk4(r[2], r[6], r[10], r[14]) << 4) | (pk4(r[3], r[7], r[11], r[15]) << 6);
      } else {
        uint32_t q[16];
#pragma unroll
        for (int e = 0; e < 16; ++e) q[e] = code_u8(r[e]);
        if constexpr (BITS == 6) {
          pack16<BITS>(q, words);
        } else {
          // 16 odd-width codes span 1.5 words: the lane pair of a token packs its 32 codes
          // (BITS words) together and the lower half stores them
          uint32_t hq[16];
#pragma unroll
          for (int e = 0; e < 16; ++e) hq[e] = __shfl_xor(q[e], 32);
#pragma unroll
          for (int i = 0; i < BITS; ++i) words[i] = 0;
#pragma unroll
          for (int e = 0; e < 32; ++e) {
            const uint32_t v = e < 16 ? q[e] : hq[e - 16];
            const int bit = e * BITS, wd = bit >> 5, off = bit & 31;
            words[wd] |= v << off;
            if (off + BITS > 32) words[wd + 1] |= v >> (32 - off);
          }
        }
      }
      // keep the epilogue in this block (not sunk into the store branch) so the scheduler can
      // interleave it with the matrix-core chain
#pragma unroll
      for (int i = 0; i < NW; ++i) asm volatile("" ::"v"(words[i]));
      asm volatile("" ::"v"(sd.word));
#pragma unroll
      for (int i = 0; i < KS * NP; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x002, 6, 0);
      }
      uint8_t* crowp = cstage[P] + n * RB;
      if constexpr ((BITS & 1) == 0) {
        store_words<NW>((uint32_t*)(crowp + (4 * w + 2 * hc) * BITS), words);
      } else if (hc == 0) {
        uint32_t* dst = (uint32_t*)(crowp + (4 * w) * BITS);
#pragma unroll
        for (int i = 0; i < BITS; ++i) dst[i] = words[i];
      }
      if (live) flags |= sd.flags | (bad ? CG_FLAG_NONFINITE : 0);
      if constexpr (TILE) {
        if (hc == 0 && (n & 15) == 0 && w % (NB / 32) == 0) sstage[P][(n >> 4) * NBK + w / (NB / 32)] = sd.word;
      } else if constexpr (NB == 16) {
        sstage[P][n * NBK + 2 * w + hc] = sd.word;
      } else if constexpr (NB == 32) {
        if (hc == 0) sstage[P][n * NBK + w] = sd.word;
      } else {
        if (hc == 0 && (w & 1) == 0) sstage[P][n * NBK + (w >> 1)] = sd.word;
      }
    }
  };
  for (int tile = tb; tile < te; tile += 2) {
    step(tile, std::integral_constant<int, 0>());
    if (tile + 1 < te) step(tile + 1, std::integral_constant<int, 1>());
  }
  if constexpr (QUANT) {
    // the last tile's staging: every wave's LDS writes done, then the final contiguous stores
    __builtin_amdgcn_s_waitcnt(waitcnt_imm(63));
    __builtin_amdgcn_s_barrier();
    if ((te - tb) & 1) flush(te - 1, std::integral_constant<int, 0>());
    else flush(te - 1, std::integral_constant<int, 1>());
  }
  ring_copy();
  if (flags && a.err) atomicOr(a.err, flags);
}

// ------------------------------------------------------------------------------------------
// decode
// ------------------------------------------------------------------------------------------
// KIVI decode: of a cache holding positions [0, held), [0, tq) are quantised and [tq, held)
// sit raw in the window ring, tq = floor((held - W) / kg) kg (0 below W).  Returns the view
// rows [0, Tq) that are quantised (view row r is position t0 + r), Tq <= Tv.
__device__ __forceinline__ int kivi_quantised_rows(const MfmaArgs& a, int held, int Tv) {
  const int tq = held < a.win ? 0 : ((held - a.win) / a.kg) * a.kg;
  return max(0, min(Tv, tq - a.t0));
}

// Positions row b holds under per-row lengths: pos[b] + pos_add.  A length outside
// [0, T_cap] sets CG_FLAG_POS_RANGE (once per slice) and the row is skipped.
__device__ __forceinline__ bool row_held(const MfmaArgs& a, int b, int chunk, int& held) {
  const int hb = a.pos[b] + a.pos_add;
  if (hb < 0 || hb > a.T_cap) {
    if (a.err && chunk == 0 && threadIdx.x == 0) atomicOr(a.err, CG_FLAG_POS_RANGE);
    return false;
  }
  held = hb;
  return true;
}

// View rows [r0, r1) copied from the window ring (bf16, slot = position mod ring_slots).
template <bool OUT_BF16>
__device__ void ring_rows(const MfmaArgs& a, size_t cslice, char* ys, int r0, int r1) {
  constexpr int YB = OUT_BF16 ? 2 : 4;
  for (int gi = r0 * 16 + int(threadIdx.x); gi < r1 * 16; gi += kThreads) {
    const int row = gi >> 4, j = gi & 15;
    const int slot = (a.t0 + row) % a.ring_slots;
    const u32x4_t v = *(const u32x4_t*)(a.ring + (cslice * a.ring_slots + slot) * kD + 8 * j);
    char* dst = ys + YB * (int64_t(row) * a.st + 8 * j);
    if constexpr (OUT_BF16) {
      *(u32x4_t*)dst = v;
    } else {
      float4 lo = make_float4(bf16_to_f32(v[0] & 0xffffu), bf16_to_f32(v[0] >> 16), bf16_to_f32(v[1] & 0xffffu), bf16_to_f32(v[1] >> 16));
      float4 hi = make_float4(bf16_to_f32(v[2] & 0xffffu), bf16_to_f32(v[2] >> 16), bf16_to_f32(v[3] & 0xffffu), bf16_to_f32(v[3] >> 16));
      *(float4*)dst = lo;
      *(float4*)(dst + 16) = hi;
    }
  }
}


// Sum over the 8-channel segments [j0, j1) of the gauge buffer's column sums of channel i
// (the two split planes of G^T over each segment's channels in i's group).
__device__ __forceinline__ float seg_colsum(const MfmaArgs& a, int l, int h, int i, int j0, int j1) {
  const float* cs = a.cs8 + ((size_t(l) * 2 + a.s) * a.Hg + h) * (kD / 8) * kD + i;
  float acc = 0.0f;
  for (int c = j0 / 8; c < j1 / 8; ++c) acc += cs[c * kD];
  return acc;
}

template <int NP, int KS, int BITS, int NB, bool OUT_BF16, int TB = 1>
__global__ __launch_bounds__(kThreads, 2) void dec_mfma(MfmaArgs a) {
  static_assert(TB == 1 || TB == 16, "token-channel tiles of 16 tokens");
  constexpr int NBK = kD / NB;                      // blocks per token row
  __shared__ __attribute__((aligned(16))) uint8_t qtile[2][kTok * kRowBytes];  // codes as bf16
  __shared__ uint32_t stile[2][kTok * NBK];         // side words
  __shared__ __attribute__((aligned(16))) float colsum[NBK][kD];
  __shared__ float mtile[2][kTok][kD / 8];         // per (token, group) centre grid points
  // decoded tile, staged so that it leaves as whole token rows (16-byte granules XOR-swizzled
  // within a row, like qtile)
  constexpr int YB = OUT_BF16 ? 2 : 4;              // output bytes per element
  constexpr int GPR = kD * YB / 16;                 // 16-byte granules per output row
  __shared__ __attribute__((aligned(16))) uint8_t ystage[2][kTok * kD * YB];

  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int n = lane & 31, hc = lane >> 5;
  const int logical = xcd_remap(blockIdx.x, gridDim.x);
  const int slice = logical / a.chunks, chunk = logical - slice * a.chunks;
  if (slice >= a.nslices) return;
  const int h = slice % a.H, b = (slice / a.H) % a.B, lv = slice / (a.H * a.B);
  const int l = lv + a.l0;
  int Tv = a.T;  // view tokens to write
  int held = a.kivi || TB > 1 ? a.len : INT_MAX;  // positions the cache holds
  if (a.pos) {
    if (!row_held(a, b, chunk, held)) return;
    Tv = min(Tv, held - a.t0);
  }
  const int ntiles = (Tv + kTok - 1) / kTok;
  const int tb = chunk * a.tiles_per_wg;
  const int te_all = min(ntiles, tb + a.tiles_per_wg);
  if (tb >= te_all) return;
  char* ys = a.x + (OUT_BF16 ? 2 : 4) * (size_t(lv) * a.sl + size_t(b) * a.sb + size_t(h) * a.sh);
  const size_t cslice = (size_t(l) * a.cB + b) * a.cH + h;
  // KIVI / tiles: the quantised view rows [0, Tq) go through the pipeline, the window or
  // staged rows after it
  const int Tq = a.kivi ? kivi_quantised_rows(a, held, Tv) : (TB > 1 ? max(0, min(Tv, held / TB * TB - a.t0)) : Tv);
  const int te = min(te_all, (Tq + kTok - 1) / kTok);
  if (tb >= te) {
    ring_rows<OUT_BF16>(a, cslice, ys, max(Tq, tb * kTok), min(Tv, te_all * kTok));
    return;
  }
  const int Tv_all = Tv;
  Tv = Tq;  // rows the pipeline writes

  const int kbase = a.g >= 32 ? (32 * w / a.g) * a.g : 32 * w;
  const int chA = 32 * w + 16 * ((n >> 2) & 1) + 4 * (n >> 3) + (n & 3);
  bf16x8_t A[NP][KS];
  load_a<NP, KS>(A, a, l, h, chA, kbase, hc);  // a.gp holds the G^T planes for decode

  // Centring.  Groups smaller than blocks (g <= 32, or g = 64 in 128-channel tiles): every
  // (token, group) is centred on the code of the group's first channel, so a group whose codes
  // are all equal decodes from the centre term alone.  Token-channel tiles with groups no
  // smaller than blocks: every (token, block) is centred on the token's first code of the block.
  // Either way the centre is a value of the token itself, so the centre term and the matrix-core
  // sums of the offsets q - c stay of the order of the token's own values; a tile's range is set
  // by 16 tokens, and centring its tokens on the tile's midpoint instead lets the two terms
  // cancel to far below their size for a token far from that midpoint.  Other blocks (one
  // token's channels) are centred on their grid midpoint (code 2^(b-1)).
  const bool gc = a.g < NB;
  const bool bc = TB > 1 && !gc;
  const int gsegs = a.g >> 4;      // 16-channel staging segments per group (g >= 16)
  constexpr int BSEGS = NB / 16;   // staging segments per block
  // column sums: per block (colsum[k][i] = sum_{j in block k} G[j][i]) or, when centring per
  // group, per group (colsum[0][i] = sum_{j in group(i)} G[j][i]), of the same split planes
  // the matrix core multiplies
  for (int idx = threadIdx.x; idx < NBK * kD; idx += kThreads) {
    const int k = idx / kD, i = idx - k * kD;
    const int r = i / a.g;
    if (!gc || k == 0)
      colsum[k][i] = seg_colsum(a, l, h, i, gc ? r * a.g : k * NB, gc ? (r + 1) * a.g : (k + 1) * NB);
  }

  // staging of a tile's code rows: thread owns token tid/8, channels 16*(tid%8) .. +16
  const int st_tok = threadIdx.x >> 3, st_seg = threadIdx.x & 7;
  const int st_blk = (16 * st_seg) / NB;           // block of the thread's channels
  constexpr int SEGW = (16 * BITS + 31) / 32 + 1;  // words covering one 16-code segment
  uint32_t cw[SEGW];
  uint32_t sw = 0, cfirst = 0;
  auto fetch = [&](int tile) {
    const int tok = min(tile * kTok + st_tok, Tv - 1);
    const size_t crow = cslice * a.T_cap + size_t(a.t0 + tok);
    const uint32_t* row = (const uint32_t*)(a.codes + crow * (kD * BITS / 8));
    const int bit0 = 16 * st_seg * BITS;
#pragma unroll
    for (int i = 0; i < SEGW; ++i) {
      const int wi = (bit0 >> 5) + i;
      cw[i] = wi < kD * BITS / 32 ? row[wi] : 0u;
    }
    // shift the segment down to bit 0 (odd widths start mid-word)
#pragma unroll
    for (int i = 0; i + 1 < SEGW; ++i) cw[i] = __builtin_amdgcn_alignbit(cw[i + 1], cw[i], bit0 & 31);
    sw = a.side[crow / TB * NBK + st_blk];  // the token's block, or its tile's
    // first code of a 32- or 64-channel group, or of a tile block, that starts in an earlier
    // segment (word aligned)
    if (gc && a.g >= 32 && st_seg % gsegs) cfirst = row[(a.g * (st_seg / gsegs) * BITS) >> 5] & ((1u << BITS) - 1u);
    if (bc && st_seg % BSEGS) cfirst = row[(NB * st_blk * BITS) >> 5] & ((1u << BITS) - 1u);
  };
  auto put = [&](int buf) {
    uint32_t q[16];
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const int bit = e * BITS, wd = bit >> 5, off = bit & 31;
      uint32_t v = cw[wd] >> off;
      if (off + BITS > 32) v |= cw[wd + 1] << (32 - off);
      q[e] = v & ((1u << BITS) - 1u);
    }
    // centre of the first and second half of the segment
    int c0 = 1 << (BITS - 1), c1 = c0;
    if (gc) {
      c0 = (a.g >= 32 && st_seg % gsegs) ? int(cfirst) : int(q[0]);
      c1 = a.g == 8 ? int(q[8]) : c0;
    } else if (bc) {
      c0 = st_seg % BSEGS ? int(cfirst) : int(q[0]);
      c1 = c0;
    }
    uint32_t v[8];
#pragma unroll
    for (int e = 0; e < 16; e += 2) {
      const int c = e < 8 ? c0 : c1;
      // bf16 of q - c: exact, |q - c| <= 255
      v[e >> 1] = (__float_as_uint(float(int(q[e]) - c)) >> 16) |
                  ((__float_as_uint(float(int(q[e + 1]) - c)) >> 16) << 16);
    }
    uint8_t* rowp = &qtile[buf][st_tok * kRowBytes];
    *(u32x4_t*)(rowp + 16 * swz(st_tok, 2 * st_seg)) = u32x4_t{v[0], v[1], v[2], v[3]};
    *(u32x4_t*)(rowp + 16 * swz(st_tok, 2 * st_seg + 1)) = u32x4_t{v[4], v[5], v[6], v[7]};
    if ((16 * st_seg) % NB == 0) stile[buf][st_tok * NBK + st_blk] = sw;
    if (gc) {
      // grid point of each group's centre code, written by the thread holding the group start
      const float mn = f16_bits_to_f32(sw & 0xffffu), sc = f16_bits_to_f32(sw >> 16);
      if (a.g == 8) {
        mtile[buf][st_tok][2 * st_seg] = mn + float(c0) * sc;
        mtile[buf][st_tok][2 * st_seg + 1] = mn + float(c1) * sc;
      } else if (a.g == 16) {
        mtile[buf][st_tok][st_seg] = mn + float(c0) * sc;
      } else if (st_seg % gsegs == 0) {
        mtile[buf][st_tok][st_seg / gsegs] = mn + float(c0) * sc;
      }
    } else if (bc && st_seg % BSEGS == 0) {
      mtile[buf][st_tok][st_blk] = f16_bits_to_f32(sw & 0xffffu) + float(c0) * f16_bits_to_f32(sw >> 16);
    }
  };

  // staged rows of `tile` -> the view: thread i moves granules i, i + 256, ... (row = granule /
  // GPR); rows past the written range are skipped
  auto flush = [&](int tile, int buf) {
    const int nlive = Tv - tile * kTok;
#pragma unroll
    for (int k = 0; k < kTok * GPR / kThreads; ++k) {
      const int gi = int(threadIdx.x) + k * kThreads;
      const int row = gi / GPR, j = gi % GPR;
      if (row < nlive) {
        const u32x4_t v = *(const u32x4_t*)(&ystage[buf][row * kD * YB + 16 * (j ^ (row & (GPR - 1)))]);
        store_stream(ys + YB * (size_t(tile * kTok + row) * a.st) + 16 * j, v);
      }
    }
  };

  fetch(tb);
  put(0);
  if (tb + 1 < te) fetch(tb + 1);
  __syncthreads();

  // K range split into block segments of KSS K-steps each
  constexpr int KR = KS * 16;
  constexpr int SEG = (KR < NB ? KR : NB) / 16;
  constexpr int NSEG = KS / SEG;
  for (int tile = tb; tile < te; ++tile) {
    const int buf = (tile - tb) & 1;
    if (tile + 1 < te) {
      put(buf ^ 1);
      if (tile + 2 < te) fetch(tile + 2);
    }
    if (tile > tb) flush(tile - 1, buf ^ 1);
    const uint8_t* rowp = &qtile[buf][n * kRowBytes];
    float y[16];
#pragma unroll
    for (int e = 0; e < 16; ++e) y[e] = 0.0f;
#pragma unroll
    for (int sgi = 0; sgi < NSEG; ++sgi) {
      f32x16_t acc0 = {}, acc1 = {};
#pragma unroll
      for (int u = 0; u < SEG; ++u) {
        const int kk = sgi * SEG + u;
        const int j = (kbase >> 3) + 2 * kk + hc;
        const bf16x8_t bv = as_bf16x8(*(const u32x4_t*)(rowp + 16 * swz(n, j)));
#pragma unroll
        for (int p = 0; p < NP; ++p) {
          if ((u * NP + p) & 1) acc1 = mfma(A[p][kk], bv, acc1);
          else acc0 = mfma(A[p][kk], bv, acc0);
        }
      }
      const int blk = (kbase + 16 * SEG * sgi) / NB;
      const uint32_t swd = stile[buf][n * NBK + blk];
      const float sc = f16_bits_to_f32(swd >> 16);
      if (gc || bc) {
#pragma unroll
        for (int e = 0; e < 16; ++e) y[e] = fmaf(sc, acc0[e] + acc1[e], y[e]);
      } else {
        const float mid = f16_bits_to_f32(swd & 0xffffu) + float(1 << (BITS - 1)) * sc;  // grid midpoint
        const float4* cs = (const float4*)&colsum[blk][32 * w + 16 * hc];
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) {
          const float4 c = cs[q4];
          const float cc[4] = {c.x, c.y, c.z, c.w};
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            const int e = 4 * q4 + u;
            y[e] = fmaf(sc, acc0[e] + acc1[e], fmaf(mid, cc[u], y[e]));
          }
        }
      }
    }
    if (gc) {
      // centre term of the row's group (one group per lane, two for g = 8)
      const int ch0 = 32 * w + 16 * hc;
      const float m0 = mtile[buf][n][ch0 / a.g];
      const float m1 = mtile[buf][n][(ch0 + 8) / a.g];
      const float4* cs = (const float4*)&colsum[0][ch0];
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        const float4 c = cs[q4];
        const float cc[4] = {c.x, c.y, c.z, c.w};
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int e = 4 * q4 + u;
          y[e] = fmaf(e < 8 ? m0 : m1, cc[u], y[e]);
        }
      }
    } else if (bc) {
      // centre terms of the row's blocks (column sums of blocks outside its group are zero)
      const int ch0 = 32 * w + 16 * hc;
#pragma unroll
      for (int k = 0; k < NBK; ++k) {
        const float mk = mtile[buf][n][k];
        const float4* cs = (const float4*)&colsum[k][ch0];
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) {
          const float4 c = cs[q4];
          const float cc[4] = {c.x, c.y, c.z, c.w};
#pragma unroll
          for (int u = 0; u < 4; ++u) y[4 * q4 + u] = fmaf(mk, cc[u], y[4 * q4 + u]);
        }
      }
    }
    // this lane's 16 channels 32w + 16hc .. +16 of token row n into the staging tile
    uint8_t* yrow = &ystage[buf][n * kD * YB];
    if constexpr (OUT_BF16) {
      uint32_t pk[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) pk[e] = f32_to_bf16_rne(y[2 * e]) | (f32_to_bf16_rne(y[2 * e + 1]) << 16);
      const int j0 = 4 * w + 2 * hc;
      *(u32x4_t*)(yrow + 16 * (j0 ^ (n & (GPR - 1)))) = u32x4_t{pk[0], pk[1], pk[2], pk[3]};
      *(u32x4_t*)(yrow + 16 * ((j0 + 1) ^ (n & (GPR - 1)))) = u32x4_t{pk[4], pk[5], pk[6], pk[7]};
    } else {
      const int j0 = 8 * w + 4 * hc;
#pragma unroll
      for (int q = 0; q < 4; ++q)
        *(float4*)(yrow + 16 * ((j0 + q) ^ (n & (GPR - 1)))) = make_float4(y[4 * q], y[4 * q + 1], y[4 * q + 2], y[4 * q + 3]);
    }
    __syncthreads();
  }
  flush(te - 1, (te - 1 - tb) & 1);
  ring_rows<OUT_BF16>(a, cslice, ys, max(Tq, tb * kTok), min(Tv_all, te_all * kTok));
}

// ------------------------------------------------------------------------------------------
// decode, blocks inside one gauge group (g >= n)
// ------------------------------------------------------------------------------------------
// The matrix core reads the codes without a float conversion: with b <= 7 the bf16 word
// 0x3F80 | (q << (7 - b)) is exactly 1 + q 2^-b, built from the packed stream with shifts and
// masks, so per block k
//   zhat_j = mn_k + q_j sc_k = (mn_k - 2^b sc_k) + 2^b sc_k B_j,   B_j = 1 + q_j 2^-b,
//   xhat_i = sum_k ( 2^b sc_k (G^T B)_{k,i} + (mn_k - 2^b sc_k) colsum_k(G^T)_i ).
// With b = 8 the operand is q itself (exact in bf16) and the offset term is mn_k colsum_k.
// B stays within [1, 2), so the block-local matrix-core sums stay of the order of the block's
// range.  This needs every block inside one gauge group (a block spanning two groups can mix
// a quiet group with another group's outlier, where the two terms cancel).
//
// A lane's B fragment for one K-step holds 8 codes of its token; which 8 channels (and in
// which order) is chosen so that the fragment is a handful of shifts of one packed word, and
// the A fragments (the rows of G^T, loaded once) are gathered in the same channel order.

// Channel order of the B fragments (and of the A fragments gathered to match): lane half hc
// owns the 8 SEG channels [16 SEG s + 8 SEG hc, +8 SEG) of block segment s of the wave's K
// range; K-step u of the segment takes, with b = 4, channels 8u + (0,4,1,5,2,6,3,7) of that
// region (nibble pairs of one packed word; the same order with b = 6, pairs 24 bits apart),
// with b = 2 channels 16 (u/2) + 4 (u%2) + (0,8,1,9,2,10,3,11) (2-bit pairs of one word; the
// same order with b = 3, pairs 24 bits apart), otherwise 8u + (0..7).
template <int NP, int KS, int BITS, int SEG>
__device__ void load_a_perm(bf16x8_t (&A)[NP][KS], const MfmaArgs& a, int l, int h, int ch, int kbase, int hc) {
  const int g = a.g, r = ch / g;
  const size_t blk = ((size_t(l) * 2 + a.s) * a.Hg + h) * a.R + r;
  // 8 consecutive entries of row ch from channel j (8-aligned, so inside one group), zero
  // outside the row's group
  auto load8 = [&](int p, int j) {
    u32x4_t v = {0u, 0u, 0u, 0u};
    if (j / g == r) v = *(const u32x4_t*)(a.gp[p] + blk * g * g + size_t(ch % g) * g + (j % g));
    return v;
  };
  // bf16 pair (lo half of x or hi half, lo half of y or hi half) -> one word
  auto pair_lo = [](uint32_t x, uint32_t y) { return __builtin_amdgcn_perm(y, x, 0x05040100u); };
  auto pair_hi = [](uint32_t x, uint32_t y) { return __builtin_amdgcn_perm(y, x, 0x07060302u); };
#pragma unroll
  for (int kk = 0; kk < KS; ++kk) {
    const int s = kk / SEG, u = kk % SEG;
    const int region = kbase + 16 * SEG * s + 8 * SEG * hc;
#pragma unroll
    for (int p = 0; p < NP; ++p) {
      u32x4_t f;
      if constexpr (BITS == 4 || BITS == 6) {
        // channels region + 8u + (0,4,1,5,2,6,3,7)
        const u32x4_t v = load8(p, region + 8 * u);
        f[0] = pair_lo(v[0], v[2]);
        f[1] = pair_hi(v[0], v[2]);
        f[2] = pair_lo(v[1], v[3]);
        f[3] = pair_hi(v[1], v[3]);
      } else if constexpr (BITS == 2 || BITS == 3) {
        // channels base + 4 (u & 1) + (0,8,1,9,2,10,3,11), base = region + 16 (u >> 1)
        const int base = region + 16 * (u >> 1);
        const u32x4_t lo = load8(p, base), hi = load8(p, base + 8);
        const int w0 = 2 * (u & 1);
        f[0] = pair_lo(lo[w0], hi[w0]);
        f[1] = pair_hi(lo[w0], hi[w0]);
        f[2] = pair_lo(lo[w0 + 1], hi[w0 + 1]);
        f[3] = pair_hi(lo[w0 + 1], hi[w0 + 1]);
      } else {
        f = load8(p, region + 8 * u);
      }
      A[p][kk] = as_bf16x8(f);
    }
  }
}

// Largest N in {0, 2, 4, 8, 12, 16, 20, 24, 32, 40} not above n: wait until at most N vector
// memory operations of the wave are outstanding (and all its LDS operations are done).
__device__ __forceinline__ void wait_vm_atmost(int n) {
  if (n >= 40) __builtin_amdgcn_s_waitcnt(waitcnt_imm(40));
  else if (n >= 32) __builtin_amdgcn_s_waitcnt(waitcnt_imm(32));
  else if (n >= 24) __builtin_amdgcn_s_waitcnt(waitcnt_imm(24));
  else if (n >= 20) __builtin_amdgcn_s_waitcnt(waitcnt_imm(20));
  else if (n >= 16) __builtin_amdgcn_s_waitcnt(waitcnt_imm(16));
  else if (n >= 12) __builtin_amdgcn_s_waitcnt(waitcnt_imm(12));
  else if (n >= 8) __builtin_amdgcn_s_waitcnt(waitcnt_imm(8));
  else if (n >= 4) __builtin_amdgcn_s_waitcnt(waitcnt_imm(4));
  else if (n >= 2) __builtin_amdgcn_s_waitcnt(waitcnt_imm(2));
  else __builtin_amdgcn_s_waitcnt(waitcnt_imm(0));
}

constexpr int kDStages = 8;  // decoder LDS ring of code and side tiles (fewer for 8-bit f32 out)

// One barrier per 32-token tile t:
//   wait for tile t's LDS-direct loads, barrier; write tile t-1's staged rows to the view;
//   issue the loads of tile t + kDStages - 1 into the slot tile t-1 used; read tile t's codes
//   and side words, build the B fragments, matrix-core chains per block segment, fold the
//   block terms, convert and stage the rows.
// Every wave issues exactly two loads per tile (codes, side words) and GPR stores per flush
// (lanes past the written range repeat a live granule), so the number of vector-memory
// operations younger than a tile's loads is known and waited for exactly.
template <int NP, int KS, int BITS, int NB, bool OUT_BF16>
__global__ __launch_bounds__(kThreads, NP == 2 ? 3 : 2) void dec_fast(MfmaArgs a) {
  constexpr int RB = kD * BITS / 8;                  // code bytes per token row
  constexpr int NBK = kD / NB;                       // side words per token row
  constexpr int SEG = (16 * KS < NB ? 16 * KS : NB) / 16;  // K-steps per block segment
  constexpr int NSEG = KS / SEG;
  constexpr int RW = SEG * BITS / 4;                 // packed words of a lane's region
  constexpr int YB = OUT_BF16 ? 2 : 4;
  constexpr int GPR = kD * YB / 16;                  // 16-byte granules per output row
  constexpr int F = kTok * GPR / kThreads;           // stores per thread per flush
  static_assert(SEG * BITS % 4 == 0 && NSEG <= 2, "unsupported block layout");
  constexpr int DS = (BITS == 8 && !OUT_BF16) ? 6 : kDStages;  // ring depth (LDS below 64 KB)
  __shared__ __attribute__((aligned(16))) uint8_t ctile[DS][kTok * RB];
  __shared__ __attribute__((aligned(16))) uint32_t stile[DS][kTok * NBK];
  __shared__ __attribute__((aligned(16))) float colsum[NBK][kD];
  __shared__ __attribute__((aligned(16))) uint8_t ystage[2][kTok * kD * YB];

  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int n = lane & 31, hc = lane >> 5;
  const int logical = xcd_remap(blockIdx.x, gridDim.x);
  const int slice = logical / a.chunks, chunk = logical - slice * a.chunks;
  if (slice >= a.nslices) return;
  const int h = slice % a.H, b = (slice / a.H) % a.B, lv = slice / (a.H * a.B);
  const int l = lv + a.l0;
  int Tv = a.T;
  int held = a.kivi ? a.len : INT_MAX;  // positions the cache holds
  if (a.pos) {
    if (!row_held(a, b, chunk, held)) return;
    Tv = min(Tv, held - a.t0);
  }
  const int ntiles = (Tv + kTok - 1) / kTok;
  const int tb = chunk * a.tiles_per_wg;
  const int te_all = min(ntiles, tb + a.tiles_per_wg);
  if (tb >= te_all) return;
  char* ys = a.x + YB * (size_t(lv) * a.sl + size_t(b) * a.sb + size_t(h) * a.sh);
  const size_t cslice = (size_t(l) * a.cB + b) * a.cH + h;
  const size_t crow0 = cslice * size_t(a.T_cap) + a.t0;
  // KIVI: the quantised view rows [0, Tq) go through the pipeline, the window after it
  const int Tq = a.kivi ? kivi_quantised_rows(a, held, Tv) : Tv;
  const int te = min(te_all, (Tq + kTok - 1) / kTok);
  if (tb >= te) {
    ring_rows<OUT_BF16>(a, cslice, ys, max(Tq, tb * kTok), min(Tv, te_all * kTok));
    return;
  }
  const int Tv_all = Tv;
  Tv = Tq;  // rows the pipeline writes

  const int kbase = a.g >= 32 ? (32 * w / a.g) * a.g : 32 * w;
  const int chA = 32 * w + 16 * ((n >> 2) & 1) + 4 * (n >> 3) + (n & 3);
  bf16x8_t A[NP][KS];
  load_a_perm<NP, KS, BITS, SEG>(A, a, l, h, chA, kbase, hc);  // a.gp holds the G^T planes

  // colsum[k][i] = sum over channels j of block k in the group of i of G[j][i], of the split
  // planes the matrix core multiplies (so the offset term cancels against the matrix-core
  // sums of the same matrix and the planes' truncation error stays proportional to zhat)
  for (int idx = threadIdx.x; idx < NBK * kD; idx += kThreads) {
    const int k = idx / kD, i = idx - k * kD;
    colsum[k][i] = seg_colsum(a, l, h, i, k * NB, (k + 1) * NB);
  }

  // LDS-direct loads: wave w fills code slots [8 BITS w, 8 BITS (w+1)) and side words
  // [8 NBK w, 8 NBK (w+1)) of the tile; rows past the view repeat its last row.  The code tile
  // is stored by 16-byte column: slot c 32 + r holds granule c of token row r, so the lanes
  // of a fragment read (one token row each) hit consecutive slots.
  const int cgi = 8 * BITS * w + lane, cgrow = cgi % kTok, cgpart = cgi / kTok;
  const int swi = 8 * NBK * w + lane, swrow = swi / NBK, swk = swi % NBK;
  auto issue = [&](int tile) {
    const int st = (tile - tb) % DS;
    const int last = Tv - 1 - tile * kTok;
    const size_t row0 = crow0 + size_t(tile) * kTok;
    if (lane < 8 * BITS)
      __builtin_amdgcn_global_load_lds(a.codes + (row0 + min(cgrow, last)) * RB + 16 * cgpart,
                                       (__attribute__((address_space(3))) void*)(ctile[st] + 16 * 8 * BITS * w), 16, 0, 0);
    if (lane < 8 * NBK) {
      __builtin_amdgcn_global_load_lds(a.side + (row0 + min(swrow, last)) * NBK + swk,
                                       (__attribute__((address_space(3))) void*)(stile[st] + 8 * NBK * w), 4, 0, 0);
    }
  };
  // staged rows of `tile` -> the view; lanes past the written rows repeat the last live row's
  // granules (same data, same address), so every thread issues F stores
  int64_t yoff[F];  // byte offset of the thread's granules from the tile's first row
  int ysrc[F];      // their staging offsets
#pragma unroll
  for (int k = 0; k < F; ++k) {
    const int gi = int(threadIdx.x) + k * kThreads, row = gi / GPR, j = gi % GPR;
    yoff[k] = int64_t(YB) * row * a.st + 16 * j;
    ysrc[k] = row * kD * YB + 16 * (j ^ (row & (GPR - 1)));
  }
  const int64_t ytile = int64_t(YB) * kTok * a.st;
  auto flush = [&](int tile, int buf) {
    const int nlive = min(kTok, Tv - tile * kTok);
    char* yt = ys + tile * ytile;
    if (nlive == kTok) {
#pragma unroll
      for (int k = 0; k < F; ++k) store_stream(yt + yoff[k], *(const u32x4_t*)(&ystage[buf][ysrc[k]]));
    } else {
#pragma unroll
      for (int k = 0; k < F; ++k) {
        int gi = int(threadIdx.x) + k * kThreads;
        if (gi >= nlive * GPR) gi = (nlive - 1) * GPR + (gi % GPR);
        const int row = gi / GPR, j = gi % GPR;
        const u32x4_t v = *(const u32x4_t*)(&ystage[buf][row * kD * YB + 16 * (j ^ (row & (GPR - 1)))]);
        store_stream(yt + int64_t(YB) * row * a.st + 16 * j, v);
      }
    }
  };
  // vector-memory operations of this wave issued after the loads of tile t, at the top of
  // iteration t: the prologue loads of later tiles, then per earlier iteration i its flush (F,
  // when i > tb) and its loads (2, when i + DS - 1 < te)
  auto younger = [&](int t) {
    if (t - (DS - 1) >= tb && t + DS - 2 < te) return (DS - 2) * (F + 2);  // steady state
    int c = 0;
    const int first = t - (DS - 1);  // iteration that issued tile t's loads (< tb: prologue)
    if (first < tb) c += 2 * (min(te, tb + DS - 1) - 1 - t);
    for (int i = max(first + 1, tb); i < t; ++i) c += (i > tb ? F : 0) + (i + DS - 1 < te ? 2 : 0);
    return c;  // (the flush of iteration `first` precedes its loads)
  };

  for (int t = tb; t < min(te, tb + DS - 1); ++t) issue(t);
  __syncthreads();  // colsum

  // sc / gamma per unit sc: codes enter as 1 + q 2^-b (6 bits: 1 + q 2^-7), 8-bit codes as q
  constexpr float kScale = BITS == 8 ? 1.0f : (BITS == 6 ? 128.0f : float(1 << BITS));
  // code_frag's constants, opaque to constant folding so that they stay in VGPRs
  uint32_t one = 0x3F803F80u,
           fmask = BITS == 2 ? 0x00600060u : (BITS == 3 ? 0x00700070u : (BITS == 6 ? 0x003F003Fu : 0x00780078u));
  asm volatile("" : "+v"(one), "+v"(fmask));
  for (int t = tb; t < te; ++t) {
    const int P = (t - tb) & 1;
    wait_vm_atmost(younger(t));
    __builtin_amdgcn_s_barrier();
    if (t > tb) flush(t - 1, P ^ 1);
    if (t + DS - 1 < te) issue(t + DS - 1);
    const int st = (t - tb) % DS;
    uint32_t sw[NBK];
#pragma unroll
    for (int k = 0; k < NBK; ++k) sw[k] = stile[st][n * NBK + k];
    float y[16];
#pragma unroll
    for (int sgi = 0; sgi < NSEG; ++sgi) {
      // region of this lane: channels kbase + 16 SEG sgi + 8 SEG hc .. + 8 SEG
      const int c0 = kbase + 16 * SEG * sgi + 8 * SEG * hc;
      uint32_t rw[RW];
      const int d0 = c0 * BITS / 32;  // first packed word of the region in the token row
      if constexpr (RW % 4 == 0) {
#pragma unroll
        for (int gq = 0; gq < RW / 4; ++gq) {
          const u32x4_t v = *(const u32x4_t*)(ctile[st] + ((d0 / 4 + gq) * kTok + n) * 16);
          rw[4 * gq] = v[0]; rw[4 * gq + 1] = v[1]; rw[4 * gq + 2] = v[2]; rw[4 * gq + 3] = v[3];
        }
      } else if constexpr (RW % 2 == 0) {
        // d0 is even here: word pairs (d, d+1) share a 16-byte column
#pragma unroll
        for (int i = 0; i < RW; i += 2) {
          const int d = d0 + i;
          const uint2 v = *(const uint2*)(ctile[st] + ((d >> 2) * kTok + n) * 16 + (d & 3) * 4);
          rw[i] = v.x; rw[i + 1] = v.y;
        }
      } else {
#pragma unroll
        for (int i = 0; i < RW; ++i) {
          const int d = d0 + i;
          rw[i] = *(const uint32_t*)(ctile[st] + ((d >> 2) * kTok + n) * 16 + (d & 3) * 4);
        }
      }
      f32x16_t acc = {};
#pragma unroll
      for (int u = 0; u < SEG; ++u) {
        const bf16x8_t bv = code_frag<BITS, RW>(rw, u, one, fmask);
#pragma unroll
        for (int p = 0; p < NP; ++p) acc = mfma(A[p][sgi * SEG + u], bv, acc);
      }
      const int blk = (kbase + 16 * SEG * sgi) / NB;
      const float mn = f16_bits_to_f32(sw[blk] & 0xffffu), sc = f16_bits_to_f32(sw[blk] >> 16);
      const float scg = sc * kScale;
      const float beta = BITS == 8 ? mn : mn - scg;
      const float4* cs = (const float4*)&colsum[blk][32 * w + 16 * hc];
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        const float4 c = cs[q4];
        const float cc[4] = {c.x, c.y, c.z, c.w};
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int e = 4 * q4 + u;
          const float base = sgi == 0 ? beta * cc[u] : fmaf(beta, cc[u], y[e]);
          y[e] = fmaf(scg, acc[e], base);
        }
      }
    }
    // this lane's channels 32w + 16hc .. +16 of token row n into the staging tile
    uint8_t* yrow = &ystage[P][n * kD * YB];
    if constexpr (OUT_BF16) {
      typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
      typedef float f32x2_t __attribute__((ext_vector_type(2)));
      uint32_t pk[8];
#pragma unroll
      for (int e = 0; e < 8; ++e)
        pk[e] = __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t{y[2 * e], y[2 * e + 1]}), bf16x2_t));
      const int j0 = 4 * w + 2 * hc;
      *(u32x4_t*)(yrow + 16 * (j0 ^ (n & (GPR - 1)))) = u32x4_t{pk[0], pk[1], pk[2], pk[3]};
      *(u32x4_t*)(yrow + 16 * ((j0 + 1) ^ (n & (GPR - 1)))) = u32x4_t{pk[4], pk[5], pk[6], pk[7]};
    } else {
      const int j0 = 8 * w + 4 * hc;
#pragma unroll
      for (int q = 0; q < 4; ++q)
        *(float4*)(yrow + 16 * ((j0 + q) ^ (n & (GPR - 1)))) = make_float4(y[4 * q], y[4 * q + 1], y[4 * q + 2], y[4 * q + 3]);
    }
  }
  __builtin_amdgcn_s_waitcnt(waitcnt_imm(63));
  __builtin_amdgcn_s_barrier();
  flush(te - 1, (te - 1 - tb) & 1);
  ring_rows<OUT_BF16>(a, cslice, ys, max(Tq, tb * kTok), min(Tv_all, te_all * kTok));
}

// ------------------------------------------------------------------------------------------
// decode centred per token, bf16 output: token-channel tiles (TB = 16: one range per 16 tokens x
// NB channels), and per-token blocks spanning gauge groups (TB = 1, g < n)
// ------------------------------------------------------------------------------------------
// Every token is centred on a code of its own (the per-token centring of dec_mfma): on its first
// code of each gauge group when groups are smaller than blocks (GC), else (tiles only) on its
// first code of each block.  The 32 code rows of a view tile are consecutive cache rows, so they
// stream into an LDS ring as one contiguous block by LDS-direct loads, with the side words beside
// them (per-token blocks: the rows' words, spread over the waves; tiles: each wave takes the words
// of the at most three 16-token tiles the rows touch into a slot of its own); the ring's waits are
// counted exactly as in dec_fast.  In the iteration before a tile's matrix-core step, thread (row
// r, segment s) converts the 16 codes of channels 16 s .. 16 s + 15 of row r to the bf16 offsets
// q - c (exact) in a double-buffered tile, and writes the centre value mn + c sc and the block's
// scale beside it.  The waves multiply the offsets by the two G^T planes; the fold adds sc times
// each block segment's sums and the centre terms through per-group or per-block column sums.
// Ring depth: code + side stages within what is left of 52 KB, so that three workgroups fit per
// CU (with two the tile decoder ran about 40% slower: it waits on its loads), at most kDStages.
constexpr int centred_stages(int bits, int nbk, int tb) {
  const int fixed = 2 * kTok * kRowBytes + 2 * kTok * kD * 2 + 2 * kD * 4 + 2 * kTok * (kD / 8) * 4 +
                    2 * kTok * nbk * 4;
  const int stage = kTok * kD * bits / 8 + (tb > 1 ? 4 * 3 * nbk : kTok * nbk) * 4;
  const int room = 52 * 1024 - fixed;
  return room / stage > kDStages ? kDStages : room / stage;
}

template <int NP, int KS, int BITS, int NB, int TB>
__global__ __launch_bounds__(kThreads, 3) void dec_centred(MfmaArgs a) {
  constexpr int RB = kD * BITS / 8;            // code bytes per row
  constexpr int NBK = kD / NB;                 // blocks per row
  // groups smaller than blocks: centred per group (per-token blocks take this kernel only then,
  // with groups of at most 32 channels)
  constexpr bool GC = TB > 1 ? 16 * KS < NB : true;
  constexpr int KR = 16 * KS;                  // K range of a wave (its gauge group, or groups)
  constexpr int SEG = (KR < NB ? KR : NB) / 16;  // K-steps per block segment of that range
  constexpr int NSEG = KS / SEG;
  constexpr int GPR = kD * 2 / 16;             // 16-byte granules per bf16 output row
  constexpr int F = kTok * GPR / kThreads;     // stores per thread per flush
  constexpr int DS = centred_stages(BITS, NBK, TB);
  constexpr int SW = TB > 1 ? 4 * 3 * NBK : kTok * NBK;  // side words of a stage
  static_assert(DS >= 3, "LDS ring too shallow");
  static_assert(TB == 16 ? (NB == 64 || NB == 128) : (TB == 1 && KS == 2 && NB <= 64), "tile or centred block shape");
  __shared__ __attribute__((aligned(16))) uint8_t ctile[DS][kTok * RB];   // code rows
  __shared__ __attribute__((aligned(16))) uint32_t stile[DS][SW];         // side words
  __shared__ __attribute__((aligned(16))) uint8_t qtile[2][kTok * kRowBytes];  // offsets q - c, bf16
  __shared__ float ctr[2][kTok][kD / 8];       // centre values per (row, group or block)
  __shared__ float scl[2][kTok][NBK];          // block scales per row
  __shared__ __attribute__((aligned(16))) float colsum[GC ? 1 : NBK][kD];
  __shared__ __attribute__((aligned(16))) uint8_t ystage[2][kTok * kD * 2];

  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int n = lane & 31, hc = lane >> 5;
  const int logical = xcd_remap(blockIdx.x, gridDim.x);
  const int slice = logical / a.chunks, chunk = logical - slice * a.chunks;
  if (slice >= a.nslices) return;
  const int h = slice % a.H, b = (slice / a.H) % a.B, lv = slice / (a.H * a.B);
  const int l = lv + a.l0;
  int Tv = a.T;
  int held = a.kivi || TB > 1 ? a.len : INT_MAX;  // positions the cache holds
  if (a.pos) {
    if (!row_held(a, b, chunk, held)) return;
    Tv = min(Tv, held - a.t0);
  }
  const int ntiles = (Tv + kTok - 1) / kTok;
  const int tb = chunk * a.tiles_per_wg;
  const int te_all = min(ntiles, tb + a.tiles_per_wg);
  if (tb >= te_all) return;
  char* ys = a.x + 2 * (size_t(lv) * a.sl + size_t(b) * a.sb + size_t(h) * a.sh);
  const size_t cslice = (size_t(l) * a.cB + b) * a.cH + h;
  const size_t crow0 = cslice * size_t(a.T_cap) + a.t0;
  // KIVI / tiles: the quantised view rows [0, Tq) go through the pipeline, the window or staged
  // rows after them are copied
  const int Tq = a.kivi ? kivi_quantised_rows(a, held, Tv) : (TB > 1 ? max(0, min(Tv, held / TB * TB - a.t0)) : Tv);
  const int te = min(te_all, (Tq + kTok - 1) / kTok);
  if (tb >= te) {
    ring_rows<true>(a, cslice, ys, max(Tq, tb * kTok), min(Tv, te_all * kTok));
    return;
  }
  const int Tv_all = Tv;
  Tv = Tq;

  const int kbase = a.g >= 32 ? (32 * w / a.g) * a.g : 32 * w;
  const int chA = 32 * w + 16 * ((n >> 2) & 1) + 4 * (n >> 3) + (n & 3);
  bf16x8_t A[NP][KS];
  load_a<NP, KS>(A, a, l, h, chA, kbase, hc);  // a.gp holds the G^T planes for decode
  // column sums of the planes the matrix core multiplies: per group (GC) or per block
  for (int idx = threadIdx.x; idx < (GC ? 1 : NBK) * kD; idx += kThreads) {
    const int k = idx / kD, i = idx - k * kD;
    const int r = i / a.g;
    colsum[k][i] = seg_colsum(a, l, h, i, GC ? r * a.g : k * NB, GC ? (r + 1) * a.g : (k + 1) * NB);
  }

  // LDS-direct loads: wave w moves granules [8 BITS w, 8 BITS (w + 1)) of the tile's code block
  // (row gi / BITS, part gi % BITS; rows past the view repeat its last row) and side words: per-token
  // blocks the words of rows 8 w .. 8 w + 7; tiles, into its own slot, the words of the (at most
  // three) 16-token tiles the rows touch (tiles past the quantised rows repeat the last one)
  const int cgi = 8 * BITS * w + lane, cgrow = cgi / BITS, cgpart = cgi % BITS;
  const int swi = 8 * NBK * w + lane, swrow = swi / NBK, swk = swi % NBK;
  auto issue = [&](int tile) {
    const int st = (tile - tb) % DS;
    const int last = Tv - 1 - tile * kTok;
    const size_t row0 = crow0 + size_t(tile) * kTok;
    if (lane < 8 * BITS)
      __builtin_amdgcn_global_load_lds(a.codes + (row0 + min(cgrow, last)) * RB + 16 * cgpart,
                                       (__attribute__((address_space(3))) void*)(ctile[st] + 16 * 8 * BITS * w), 16, 0, 0);
    if constexpr (TB > 1) {
      const size_t blk0 = row0 / TB, blast = (row0 + last) / TB;
      if (lane < 3 * NBK)
        __builtin_amdgcn_global_load_lds(a.side + min(blk0 + lane / NBK, blast) * NBK + lane % NBK,
                                         (__attribute__((address_space(3))) void*)(stile[st] + 3 * NBK * w), 4, 0, 0);
    } else if (lane < 8 * NBK) {
      __builtin_amdgcn_global_load_lds(a.side + (row0 + min(swrow, last)) * NBK + swk,
                                       (__attribute__((address_space(3))) void*)(stile[st] + 8 * NBK * w), 4, 0, 0);
    }
  };
  int64_t yoff[F];
  int ysrc[F];
#pragma unroll
  for (int k = 0; k < F; ++k) {
    const int gi = int(threadIdx.x) + k * kThreads, row = gi / GPR, j = gi % GPR;
    yoff[k] = int64_t(2) * row * a.st + 16 * j;
    ysrc[k] = row * kD * 2 + 16 * (j ^ (row & (GPR - 1)));
  }
  const int64_t ytile = int64_t(2) * kTok * a.st;
  auto flush = [&](int tile, int buf) {
    const int nlive = min(kTok, Tv - tile * kTok);
    char* yt = ys + tile * ytile;
    if (nlive == kTok) {
#pragma unroll
      for (int k = 0; k < F; ++k) store_stream(yt + yoff[k], *(const u32x4_t*)(&ystage[buf][ysrc[k]]));
    } else {
#pragma unroll
      for (int k = 0; k < F; ++k) {
        int gi = int(threadIdx.x) + k * kThreads;
        if (gi >= nlive * GPR) gi = (nlive - 1) * GPR + (gi % GPR);
        const int row = gi / GPR, j = gi % GPR;
        const u32x4_t v = *(const u32x4_t*)(&ystage[buf][row * kD * 2 + 16 * (j ^ (row & (GPR - 1)))]);
        store_stream(yt + int64_t(2) * row * a.st + 16 * j, v);
      }
    }
  };
  // vector-memory operations of this wave issued after the loads of tile X, at the wait of
  // iteration t (before its barrier): the prologue's later loads, then per iteration i < t its
  // flush (F stores, i > tb) and its loads (2, i + DS - 1 < te)
  const int pe = min(te, tb + DS - 1);
  auto younger = [&](int X, int t) {
    // steady state: X's loads came from iteration X - (DS - 1) >= tb, and every iteration since
    // flushed and issued
    if (X - (DS - 1) >= tb && t + DS - 2 < te) return (t - (X - (DS - 1)) - 1) * (F + 2);
    int c = 0, i = tb;
    if (X < pe) c = 2 * (pe - 1 - X);
    else i = X - (DS - 1) + 1;
    for (; i < t; ++i) c += (i > tb ? F : 0) + (i + DS - 1 < te ? 2 : 0);
    return c;
  };

  // conversion of a tile's codes: thread (row cr, segment cs)
  const int cr = threadIdx.x >> 3, cs = threadIdx.x & 7;
  const int cblk = (16 * cs) / NB;                 // block of the segment
  constexpr int SEGW = (16 * BITS + 31) / 32 + 1;  // words covering one 16-code segment
  constexpr uint32_t QM = (1u << BITS) - 1u;
  auto convert = [&](int tile, int buf) {
    const int st = (tile - tb) % DS;
    const int rr = min(cr, Tv - 1 - tile * kTok);  // rows past the view repeat the last one
    const uint32_t* row = reinterpret_cast<const uint32_t*>(ctile[st] + rr * RB);
    const int bit0 = 16 * cs * BITS;
    uint32_t cw[SEGW];
#pragma unroll
    for (int i = 0; i < SEGW; ++i) {
      const int wi = (bit0 >> 5) + i;
      cw[i] = wi < kD * BITS / 32 ? row[wi] : 0u;
    }
#pragma unroll
    for (int i = 0; i + 1 < SEGW; ++i) cw[i] = __builtin_amdgcn_alignbit(cw[i + 1], cw[i], bit0 & 31);
    uint32_t q[16];
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const int bit = e * BITS, wd = bit >> 5, off = bit & 31;
      uint32_t v = cw[wd] >> off;
      if (off + BITS > 32) v |= cw[wd + 1] << (32 - off);
      q[e] = v & QM;
    }
    // centres: the unit's first code (in this segment, or word-aligned at the unit's start)
    int c0, c1;
    if constexpr (GC) {
      const int gsegs = a.g >> 4;
      if (a.g == 8) {
        c0 = int(q[0]);
        c1 = int(q[8]);
      } else {
        c0 = (cs % gsegs) ? int(row[(a.g * (cs / gsegs) * BITS) >> 5] & QM) : int(q[0]);
        c1 = c0;
      }
    } else {
      constexpr int BSEGS = NB / 16;
      c0 = (cs % BSEGS) ? int(row[(NB * cblk * BITS) >> 5] & QM) : int(q[0]);
      c1 = c0;
    }
    uint32_t v[8];
#pragma unroll
    for (int e = 0; e < 16; e += 2) {
      const int c = e < 8 ? c0 : c1;
      v[e >> 1] = (__float_as_uint(float(int(q[e]) - c)) >> 16) | ((__float_as_uint(float(int(q[e + 1]) - c)) >> 16) << 16);
    }
    uint8_t* rowp = &qtile[buf][cr * kRowBytes];
    *(u32x4_t*)(rowp + 16 * swz(cr, 2 * cs)) = u32x4_t{v[0], v[1], v[2], v[3]};
    *(u32x4_t*)(rowp + 16 * swz(cr, 2 * cs + 1)) = u32x4_t{v[4], v[5], v[6], v[7]};
    // side word of the row's block (tiles: of its 16-token tile, in this wave's copy of the slot)
    uint32_t sw;
    if constexpr (TB > 1) {
      const size_t crow = crow0 + size_t(tile) * kTok + rr;
      const int bi = int(crow / TB - (crow0 + size_t(tile) * kTok) / TB);
      sw = stile[st][3 * NBK * w + bi * NBK + cblk];
    } else {
      sw = stile[st][rr * NBK + cblk];
    }
    const float mn = f16_bits_to_f32(sw & 0xffffu), sc = f16_bits_to_f32(sw >> 16);
    if ((16 * cs) % NB == 0) scl[buf][cr][cblk] = sc;
    if constexpr (GC) {
      const int gsegs = a.g >> 4;
      if (a.g == 8) {
        ctr[buf][cr][2 * cs] = mn + float(c0) * sc;
        ctr[buf][cr][2 * cs + 1] = mn + float(c1) * sc;
      } else if (cs % gsegs == 0) {
        ctr[buf][cr][cs / gsegs] = mn + float(c0) * sc;
      }
    } else if (cs % (NB / 16) == 0) {
      ctr[buf][cr][cblk] = mn + float(c0) * sc;
    }
  };

  for (int t = tb; t < pe; ++t) issue(t);
  wait_vm_atmost(younger(tb, tb));
  __syncthreads();  // tile tb's loads, colsum
  convert(tb, 0);
  for (int t = tb; t < te; ++t) {
    const int P = (t - tb) & 1;
    if (t + 1 < te) wait_vm_atmost(younger(t + 1, t));
    else __builtin_amdgcn_s_waitcnt(waitcnt_imm(63));
    __builtin_amdgcn_s_barrier();
    if (t > tb) flush(t - 1, P ^ 1);
    if (t + DS - 1 < te) issue(t + DS - 1);
    if (t + 1 < te) convert(t + 1, P ^ 1);
    const uint8_t* rowp = &qtile[P][n * kRowBytes];
    float y[16];
#pragma unroll
    for (int e = 0; e < 16; ++e) y[e] = 0.0f;
#pragma unroll
    for (int sgi = 0; sgi < NSEG; ++sgi) {
      f32x16_t acc0 = {}, acc1 = {};
#pragma unroll
      for (int u = 0; u < SEG; ++u) {
        const int kk = sgi * SEG + u;
        const int j = (kbase >> 3) + 2 * kk + hc;
        const bf16x8_t bv = as_bf16x8(*(const u32x4_t*)(rowp + 16 * swz(n, j)));
#pragma unroll
        for (int p = 0; p < NP; ++p) {
          if ((u * NP + p) & 1) acc1 = mfma(A[p][kk], bv, acc1);
          else acc0 = mfma(A[p][kk], bv, acc0);
        }
      }
      const float sc = scl[P][n][(kbase + 16 * SEG * sgi) / NB];
#pragma unroll
      for (int e = 0; e < 16; ++e) y[e] = fmaf(sc, acc0[e] + acc1[e], y[e]);
    }
    // centre terms (column sums of groups or blocks outside the output's group are zero)
    const int ch0 = 32 * w + 16 * hc;
    if constexpr (GC) {
      const float m0 = ctr[P][n][ch0 / a.g];
      const float m1 = ctr[P][n][(ch0 + 8) / a.g];
      const float4* csp = (const float4*)&colsum[0][ch0];
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        const float4 c = csp[q4];
        const float cc[4] = {c.x, c.y, c.z, c.w};
#pragma unroll
        for (int u = 0; u < 4; ++u) y[4 * q4 + u] = fmaf(4 * q4 + u < 8 ? m0 : m1, cc[u], y[4 * q4 + u]);
      }
    } else {
#pragma unroll
      for (int k = 0; k < NBK; ++k) {
        const float mk = ctr[P][n][k];
        const float4* csp = (const float4*)&colsum[k][ch0];
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) {
          const float4 c = csp[q4];
          const float cc[4] = {c.x, c.y, c.z, c.w};
#pragma unroll
          for (int u = 0; u < 4; ++u) y[4 * q4 + u] = fmaf(mk, cc[u], y[4 * q4 + u]);
        }
      }
    }
    uint8_t* yrow = &ystage[P][n * kD * 2];
    typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
    typedef float f32x2_t __attribute__((ext_vector_type(2)));
    uint32_t pk[8];
#pragma unroll
    for (int e = 0; e < 8; ++e)
      pk[e] = __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t{y[2 * e], y[2 * e + 1]}), bf16x2_t));
    const int j0 = 4 * w + 2 * hc;
    *(u32x4_t*)(yrow + 16 * (j0 ^ (n & (GPR - 1)))) = u32x4_t{pk[0], pk[1], pk[2], pk[3]};
    *(u32x4_t*)(yrow + 16 * ((j0 + 1) ^ (n & (GPR - 1)))) = u32x4_t{pk[4], pk[5], pk[6], pk[7]};
  }
  __builtin_amdgcn_s_waitcnt(waitcnt_imm(63));
  __builtin_amdgcn_s_barrier();
  flush(te - 1, (te - 1 - tb) & 1);
  ring_rows<true>(a, cslice, ys, max(Tq, tb * kTok), min(Tv_all, te_all * kTok));
}

// ------------------------------------------------------------------------------------------
// decode, KIVI keys (per-channel ranges over 32-token groups), groups of at most 32 channels
// ------------------------------------------------------------------------------------------
// LDS ring depth: code + side stages within what is left of 52 KB (three workgroups per CU)
// for bf16 output, of 64 KB for binary32 output, at most kDStages
constexpr int keys_stages(int bits, bool bf16) {
  const int fixed = 2 * kTok * kD * (bf16 ? 2 : 4);
  const int room = (bf16 ? 52 : 64) * 1024 - fixed, stage = kD * 4 * bits + kD * 4;
  return room / stage > kDStages ? kDStages : room / stage;
}

// One tile is one key group (cache positions 32k .. 32k + 31).  Wave w's contraction runs over
// the gauge group(s) of its 32 output channels: its own 32 channels for groups of at most 32
// (KS = 2), the 64 or 128 channels of its group otherwise (KS = 4, 8), each wave then
// dequantising every code it multiplies (the code block is in LDS; the waves of a 64- or
// 128-channel group repeat that work rather than exchange it behind a second barrier).  Lane
// (n, hc) rebuilds zhat = fl(mn + q sc) of token n for its K-channels in binary32 (the
// dequantised value itself), splits it into three bf16 planes (exact: a binary32 value holds
// 24 significant bits), and the matrix core multiplies them by the two G^T planes (plane
// products below 2^-24 of the leading term dropped).  The error is thus relative to the group
// norm of zhat, whatever the channels' offsets; with the identity gauge the result is zhat bit
// for bit.
template <int NP, int KS, int BITS, bool OUT_BF16>
__global__ __launch_bounds__(kThreads, OUT_BF16 ? 3 : 2) void dec_keys(MfmaArgs a) {
  static_assert((KS == 2 || KS == 4 || KS == 8) && NP == 2, "K-steps of a gauge group, two gauge planes");
  constexpr int CB = 4 * BITS;                       // bytes of one channel's 32 codes
  constexpr int YB = OUT_BF16 ? 2 : 4;
  constexpr int GPR = kD * YB / 16;
  constexpr int F = kTok * GPR / kThreads;
  constexpr int DS = keys_stages(BITS, OUT_BF16);
  static_assert(DS >= 3, "LDS ring too shallow");
  __shared__ __attribute__((aligned(16))) uint8_t ctile[DS][kD * CB];   // code block of a group
  __shared__ __attribute__((aligned(16))) uint32_t stile[DS][kD];       // side word per channel
  __shared__ __attribute__((aligned(16))) uint8_t ystage[2][kTok * kD * YB];

  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int n = lane & 31, hc = lane >> 5;
  const int logical = xcd_remap(blockIdx.x, gridDim.x);
  const int slice = logical / a.chunks, chunk = logical - slice * a.chunks;
  if (slice >= a.nslices) return;
  const int h = slice % a.H, b = (slice / a.H) % a.B, lv = slice / (a.H * a.B);
  const int l = lv + a.l0;
  int Tv = a.T;
  int held = a.len;
  if (a.pos) {
    if (!row_held(a, b, chunk, held)) return;
    Tv = min(Tv, held - a.t0);
  }
  if (Tv <= 0) return;
  char* ys = a.x + YB * (size_t(lv) * a.sl + size_t(b) * a.sb + size_t(h) * a.sh);
  const size_t cslice = (size_t(l) * a.cB + b) * a.cH + h;
  const int Tq = kivi_quantised_rows(a, held, Tv);  // quantised view rows [0, Tq)
  // tiles u = key groups g0 + u; tile u holds view rows 32 (g0 + u) - t0 + j, j < 32
  const int g0 = a.t0 / kTok;
  const int ntiles = (a.t0 + Tv + kTok - 1) / kTok - g0;
  const int tb = chunk * a.tiles_per_wg;
  const int te_all = min(ntiles, tb + a.tiles_per_wg);
  if (tb >= te_all) return;
  // key groups holding quantised view rows; none when Tq = 0 (a range that starts inside a group
  // and lies in the window would otherwise keep that group, and its flush would have no live row)
  const int te = Tq > 0 ? min(te_all, (a.t0 + Tq + kTok - 1) / kTok - g0) : 0;
  const int row_lo = max(0, kTok * (g0 + tb) - a.t0), row_hi = min(Tv, kTok * (g0 + te_all) - a.t0);
  if (tb >= te) {
    ring_rows<OUT_BF16>(a, cslice, ys, max(Tq, row_lo), row_hi);
    return;
  }

  const int kbase = (32 * w) & ~(16 * KS - 1);  // first channel of the wave's gauge group(s)
  const int chA = 32 * w + 16 * ((n >> 2) & 1) + 4 * (n >> 3) + (n & 3);
  bf16x8_t A[NP][KS];
  load_a<NP, KS>(A, a, l, h, chA, kbase, hc);  // rows chA of the G^T planes, natural K order

  // LDS-direct loads of a group: wave w moves code granules [8 BITS w, +8 BITS) and side words
  // [32 w, +32) of the group block (contiguous in the cache)
  const int wu = __builtin_amdgcn_readfirstlane(w);
  const size_t grp0 = cslice * size_t(a.T_cap / kTok) + g0;
  auto issue = [&](int tile) {
    const int st = (tile - tb) % DS;
    const size_t gi = grp0 + tile;
    if (lane < 8 * BITS)
      __builtin_amdgcn_global_load_lds(a.codes + gi * (kD * CB) + 16 * (8 * BITS * w + lane),
                                       (__attribute__((address_space(3))) void*)(ctile[st] + 16 * 8 * BITS * wu), 16, 0, 0);
    if (lane < 32)
      __builtin_amdgcn_global_load_lds(a.side + gi * kD + 32 * w + lane,
                                       (__attribute__((address_space(3))) void*)(stile[st] + 32 * wu), 4, 0, 0);
  };
  // staged rows -> the view: tile row j is view row 32 (g0 + tile) - t0 + j; rows outside the
  // quantised range repeat a live row's granule (same data, same address)
  int64_t yoff[F];
  int ysrc[F];
#pragma unroll
  for (int k = 0; k < F; ++k) {
    const int gi = int(threadIdx.x) + k * kThreads, row = gi / GPR, j = gi % GPR;
    yoff[k] = int64_t(YB) * row * a.st + 16 * j;
    ysrc[k] = row * kD * YB + 16 * (j ^ (row & (GPR - 1)));
  }
  auto flush = [&](int tile, const uint8_t* stage) {
    const int r0 = kTok * (g0 + tile) - a.t0;          // view row of tile row 0 (may be < 0)
    const int lo = max(0, -r0), hi = min(kTok, Tq - r0);  // live tile rows
    char* yt = ys + int64_t(YB) * r0 * a.st;
    if (lo == 0 && hi == kTok) {
#pragma unroll
      for (int k = 0; k < F; ++k) store_stream(yt + yoff[k], *(const u32x4_t*)(stage + ysrc[k]));
    } else {
#pragma unroll
      for (int k = 0; k < F; ++k) {
        const int gi = int(threadIdx.x) + k * kThreads, j = gi % GPR;
        int row = gi / GPR;
        row = row < lo ? lo : (row >= hi ? hi - 1 : row);
        const u32x4_t v = *(const u32x4_t*)(stage + row * kD * YB + 16 * (j ^ (row & (GPR - 1))));
        store_stream(yt + int64_t(YB) * row * a.st + 16 * j, v);
      }
    }
  };
  // vector-memory operations a wave has issued after tile X's two loads, at the wait of
  // iteration t: the prologue's later loads, then per iteration i the flush of tile i - 1 (F
  // stores) and the loads of tile i + DS - 1
  const int pe = min(te, tb + DS - 1);
  auto younger = [&](int X, int t) {
    if (X - (DS - 1) >= tb && t + DS - 2 < te) return (t - (X - (DS - 1)) - 1) * (F + 2);
    int c = 0, i = tb;
    if (X < pe) c = 2 * (pe - 1 - X);
    else i = X - (DS - 1) + 1;
    for (; i < t; ++i) c += (i > tb ? F : 0) + (i + DS - 1 < te ? 2 : 0);
    return c;
  };
  // this lane's code of token n in a channel stream: word wd, bit offset off
  constexpr uint32_t MASK = (1u << BITS) - 1u;
  const int cbit = n * BITS, cwd = cbit >> 5, coff = cbit & 31;

  for (int t = tb; t < pe; ++t) issue(t);
  for (int t = tb; t < te; ++t) {
    const int P = (t - tb) & 1;
    wait_vm_atmost(younger(t, t));
    __builtin_amdgcn_s_barrier();
    if (t > tb) flush(t - 1, ystage[P ^ 1]);
    if (t + DS - 1 < te) issue(t + DS - 1);
    const uint8_t* ct = ctile[(t - tb) % DS];
    const uint32_t* sw = stile[(t - tb) % DS];
    f32x16_t acc = {};
#pragma unroll
    for (int kk = 0; kk < KS; ++kk) {
      const int j0 = kbase + 16 * kk + 8 * hc;
      const u32x4_t s0 = *(const u32x4_t*)(sw + j0), s1 = *(const u32x4_t*)(sw + j0 + 4);
      const uint32_t swd[8] = {s0[0], s0[1], s0[2], s0[3], s1[0], s1[1], s1[2], s1[3]};
      float zh[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const uint32_t* cw = (const uint32_t*)(ct + (j0 + e) * CB);
        uint32_t v;
        if constexpr (32 % BITS == 0) {
          v = cw[cwd] >> coff;
        } else {  // the code may straddle two words (never past the stream's last word)
          const uint32_t lo = cw[cwd], hi = coff + BITS > 32 ? cw[cwd + 1] : 0u;
          v = uint32_t(((uint64_t(hi) << 32) | lo) >> coff);
        }
        const float mn = f16_bits_to_f32(swd[e] & 0xffffu), sc = f16_bits_to_f32(swd[e] >> 16);
        zh[e] = fmaf(float(v & MASK), sc, mn);  // q sc is exact: one rounding, as dequantised
      }
      // three bf16 planes of zhat by truncation (each residual exact in binary32)
      uint32_t bp[3][4];
#pragma unroll
      for (int e2 = 0; e2 < 4; ++e2) {
        uint32_t x0 = __float_as_uint(zh[2 * e2]), x1 = __float_as_uint(zh[2 * e2 + 1]);
#pragma unroll
        for (int p = 0; p < 3; ++p) {
          bp[p][e2] = __builtin_amdgcn_perm(x1, x0, 0x07060302u);
          if (p < 2) {
            x0 = __float_as_uint(__uint_as_float(x0) - __uint_as_float(x0 & 0xffff0000u));
            x1 = __float_as_uint(__uint_as_float(x1) - __uint_as_float(x1 & 0xffff0000u));
          }
        }
      }
      bf16x8_t B[3];
#pragma unroll
      for (int p = 0; p < 3; ++p) B[p] = as_bf16x8(u32x4_t{bp[p][0], bp[p][1], bp[p][2], bp[p][3]});
      // plane products, smallest first: (1,1) (0,2) (1,0) (0,1) (0,0)
      acc = mfma(A[1][kk], B[1], acc);
      acc = mfma(A[0][kk], B[2], acc);
      acc = mfma(A[1][kk], B[0], acc);
      acc = mfma(A[0][kk], B[1], acc);
      acc = mfma(A[0][kk], B[0], acc);
    }
    uint8_t* yrow = ystage[P] + n * kD * YB;
    if constexpr (OUT_BF16) {
      typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
      typedef float f32x2_t __attribute__((ext_vector_type(2)));
      uint32_t pk[8];
#pragma unroll
      for (int e = 0; e < 8; ++e)
        pk[e] = __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t{acc[2 * e], acc[2 * e + 1]}), bf16x2_t));
      const int j0 = 4 * w + 2 * hc;
      *(u32x4_t*)(yrow + 16 * (j0 ^ (n & (GPR - 1)))) = u32x4_t{pk[0], pk[1], pk[2], pk[3]};
      *(u32x4_t*)(yrow + 16 * ((j0 + 1) ^ (n & (GPR - 1)))) = u32x4_t{pk[4], pk[5], pk[6], pk[7]};
    } else {
      const int j0 = 8 * w + 4 * hc;
#pragma unroll
      for (int q = 0; q < 4; ++q)
        *(float4*)(yrow + 16 * ((j0 + q) ^ (n & (GPR - 1)))) = make_float4(acc[4 * q], acc[4 * q + 1], acc[4 * q + 2], acc[4 * q + 3]);
    }
  }
  __builtin_amdgcn_s_waitcnt(waitcnt_imm(63));
  __builtin_amdgcn_s_barrier();
  flush(te - 1, ystage[(te - 1 - tb) & 1]);
  ring_rows<OUT_BF16>(a, cslice, ys, max(Tq, row_lo), row_hi);
}

// ------------------------------------------------------------------------------------------
// dispatch
// ------------------------------------------------------------------------------------------
// Split planes of the gauge on the matrix core.  Decoding takes two (16 significant bits per
// entry: a few 1e-6 of the group norm).  Encoding takes two up to 4-bit codes and three
// above: a finer grid turns the same z error into more codes moved across a rounding
// boundary (with two planes about 3e-5 of 4-bit codes but 1.4e-4 of 6-bit codes move, against
// the 1e-4 budget).
// ------------------------------------------------------------------------------------------
// decode, zfp-style blocks (4 tokens x 4 channels of zhat, 16 RATE bits each)
// ------------------------------------------------------------------------------------------
// A workgroup owns a range of 32-token tiles of one slice.  Per tile, thread u * 32 + cb decodes
// block (tokens 4u .. 4u+3, channels 4cb .. 4cb+3) and splits each zhat into bf16 planes, written
// to an LDS tile per plane ([token][channel], 16-byte granules XOR-swizzled by token as in the
// encoder's ring); after a barrier wave w computes output channels 32w .. 32w+31 of the 32 tokens
// on the matrix cores, reading its B fragments straight from LDS: the plane products that matter
// against the two G^T planes accumulate in binary32 (as the KIVI key decoder does).  Splitting in
// the decoding thread does it once per value instead of once per wave.
//   binary32 output: three planes by truncation (each residual exact, so the planes sum to zhat),
//     five products;
//   bf16 output: the truncated high plane and the rounded-to-nearest residual, three products.
//     The dropped part is at most 2^-16 of each value, so with G orthogonal an output moves by at
//     most 2^-16 of the group's norm and typically by 2^-16 / sqrt(3 g) of it (independent
//     rounding errors), against the bf16 criterion of one ulp plus 1e-5 of the group's norm.
template <int KS, int RATE, bool OUT_BF16>
__global__ __launch_bounds__(kThreads, 2) void dec_zfp(MfmaArgs a) {
  constexpr int YB = OUT_BF16 ? 2 : 4;
  constexpr int NPL = OUT_BF16 ? 2 : 3;  // planes of zhat
  __shared__ __attribute__((aligned(16))) uint8_t zpl[NPL][kTok * kRowBytes];
  __shared__ ZfpTables ztab;

  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int n = lane & 31, hc = lane >> 5;
  const int logical = xcd_remap(blockIdx.x, gridDim.x);
  const int slice = logical / a.chunks, chunk = logical - slice * a.chunks;
  if (slice >= a.nslices) return;
  const int h = slice % a.H, b = (slice / a.H) % a.B, lv = slice / (a.H * a.B);
  const int l = lv + a.l0;
  const int ntiles = (a.T + kTok - 1) / kTok;
  const int tb = chunk * a.tiles_per_wg;
  const int te = min(ntiles, tb + a.tiles_per_wg);
  if (tb >= te) return;
  char* ys = a.x + YB * (size_t(lv) * a.sl + size_t(b) * a.sb + size_t(h) * a.sh);
  const size_t cslice = (size_t(l) * a.cB + b) * a.cH + h;

  const int kbase = a.g >= 32 ? (32 * w / a.g) * a.g : 32 * w;
  const int chA = 32 * w + 16 * ((n >> 2) & 1) + 4 * (n >> 3) + (n & 3);
  bf16x8_t A[2][KS];
  load_a<2, KS>(A, a, l, h, chA, kbase, hc);  // rows chA of the G^T planes
  int boff[KS];
#pragma unroll
  for (int kk = 0; kk < KS; ++kk) boff[kk] = n * kRowBytes + 16 * swz(n, (kbase >> 3) + 2 * kk + hc);

  const int tid = int(threadIdx.x), u = tid >> 5, cb = tid & 31;
  zfp_tables_init(ztab);
  __syncthreads();
  for (int t = tb; t < te; ++t) {
    // 1. blocks -> zhat planes (the view's token count and offset are multiples of 4)
    if (4 * u < a.T - t * kTok) {
      const size_t blk = (cslice * size_t(a.T_cap / 4) + (a.t0 + t * kTok) / 4 + u) * (kD / 4) + cb;
      uint32_t wd[4];
      zfp_load<RATE>(a.codes + blk * (2 * RATE), wd);
      float v[16];
      zfp_decode_block<RATE>(wd, ztab, v);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        uint32_t pw[NPL][2];
#pragma unroll
        for (int e2 = 0; e2 < 2; ++e2) {
          uint32_t x0 = __float_as_uint(v[4 * j + 2 * e2]), x1 = __float_as_uint(v[4 * j + 2 * e2 + 1]);
#pragma unroll
          for (int p = 0; p < NPL; ++p) {
            if (OUT_BF16 && p == NPL - 1) {
              typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
              typedef float f32x2_t __attribute__((ext_vector_type(2)));
              pw[p][e2] = __builtin_bit_cast(
                  uint32_t, __builtin_convertvector((f32x2_t{__uint_as_float(x0), __uint_as_float(x1)}), bf16x2_t));
            } else {
              pw[p][e2] = __builtin_amdgcn_perm(x1, x0, 0x07060302u);
            }
            if (p < NPL - 1) {
              x0 = __float_as_uint(__uint_as_float(x0) - __uint_as_float(x0 & 0xffff0000u));
              x1 = __float_as_uint(__uint_as_float(x1) - __uint_as_float(x1 & 0xffff0000u));
            }
          }
        }
        const int row = 4 * u + j;
        const int off = row * kRowBytes + 16 * swz(row, cb >> 1) + 8 * (cb & 1);
#pragma unroll
        for (int p = 0; p < NPL; ++p) *(uint2*)(zpl[p] + off) = make_uint2(pw[p][0], pw[p][1]);
      }
    }
    __syncthreads();
    // 2. xhat = G^T zhat for the lane's token n and channels 32w + 16hc + [0, 16)
    f32x16_t acc = {};
#pragma unroll
    for (int kk = 0; kk < KS; ++kk) {
      bf16x8_t B[NPL];
#pragma unroll
      for (int p = 0; p < NPL; ++p) B[p] = as_bf16x8(*(const u32x4_t*)(zpl[p] + boff[kk]));
      // plane products, smallest first: (1,1) (0,2) (1,0) (0,1) (0,0); with two planes of
      // zhat (1,0) (0,1) (0,0)
      if constexpr (NPL == 3) {
        acc = mfma(A[1][kk], B[1], acc);
        acc = mfma(A[0][kk], B[2], acc);
      }
      acc = mfma(A[1][kk], B[0], acc);
      acc = mfma(A[0][kk], B[1], acc);
      acc = mfma(A[0][kk], B[0], acc);
    }
    const int row = t * kTok + n;
    if (row < a.T) {
      char* yr = ys + int64_t(YB) * (int64_t(row) * a.st + 32 * w + 16 * hc);
      if constexpr (OUT_BF16) {
        typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
        typedef float f32x2_t __attribute__((ext_vector_type(2)));
        uint32_t pk[8];
#pragma unroll
        for (int e = 0; e < 8; ++e)
          pk[e] = __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t{acc[2 * e], acc[2 * e + 1]}), bf16x2_t));
        *(u32x4_t*)yr = u32x4_t{pk[0], pk[1], pk[2], pk[3]};
        *(u32x4_t*)(yr + 16) = u32x4_t{pk[4], pk[5], pk[6], pk[7]};
      } else {
#pragma unroll
        for (int q = 0; q < 4; ++q) *(float4*)(yr + 16 * q) = make_float4(acc[4 * q], acc[4 * q + 1], acc[4 * q + 2], acc[4 * q + 3]);
      }
    }
    __syncthreads();  // the planes are read before the next tile is decoded into them
  }
}

template <int KS, int RATE>
void* zfp_dec_kernel(bool bf16) {
  return bf16 ? (void*)dec_zfp<KS, RATE, true> : (void*)dec_zfp<KS, RATE, false>;
}

template <int KS>
void* zfp_dec_by_rate(int rate, bool bf16) {
  switch (rate) {
    case 2: return zfp_dec_kernel<KS, 2>(bf16);
    case 3: return zfp_dec_kernel<KS, 3>(bf16);
    case 4: return zfp_dec_kernel<KS, 4>(bf16);
    case 6: return zfp_dec_kernel<KS, 6>(bf16);
    case 8: return zfp_dec_kernel<KS, 8>(bf16);
  }
  return nullptr;
}

constexpr int kNP = kDecPlanes;
constexpr int enc_planes(int bits) { return bits >= 6 ? 3 : 2; }

int cu_count() {
  static int cus = 0;
  if (!cus) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
      cus = 256;
  }
  return cus;
}

// Split the (slice, tile) space into workgroups: as many as can be resident at once (the
// kernel's occupancy per CU times the CUs), each a contiguous tile range of one slice; the
// count is padded to a multiple of 8 (XCD remap).
//
// CG_TILES_PER_WG=k (read at every launch) fixes the tiles per workgroup instead, so that small
// inputs run the multi-tile pipeline (ring wrap, prefetch, overlapped flush, exact waits) that
// the resident grid only reaches on large ones; the tests compare both geometries.
int forced_tiles_per_wg() {
  const char* e = getenv("CG_TILES_PER_WG");
  if (!e || !*e) return 0;
  const long v = strtol(e, nullptr, 10);
  return v > 0 && v < (1 << 20) ? int(v) : 0;
}

void plan(MfmaArgs& m, int nslices, int T, const void* fn) {
  const int ntiles = (T + kTok - 1) / kTok;
  int occ = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&occ, fn, kThreads, 0) != hipSuccess || occ < 1) occ = 2;
  const int target = occ * cu_count();
  int chunks = (target + nslices - 1) / nslices;
  chunks = chunks < 1 ? 1 : (chunks > ntiles ? ntiles : chunks);
  m.tiles_per_wg = (ntiles + chunks - 1) / chunks;
  if (const int f = forced_tiles_per_wg()) m.tiles_per_wg = f < ntiles ? f : (ntiles > 0 ? ntiles : 1);
  m.chunks = (ntiles + m.tiles_per_wg - 1) / m.tiles_per_wg;
  m.nslices = nslices;
}

template <int KS, int BITS, int NB>
void* enc_kernel(int mode, int bt) {
  if (mode == kModePass) return (void*)enc_mfma<kNP, KS, 8, 64, kModePass>;
  if (mode == kModeZfp) return NB == 64 ? (void*)enc_mfma<kNP, KS, BITS, 64, kModeZfp> : nullptr;
  if (mode == kModeKeys) return (void*)enc_mfma<enc_planes(BITS), KS, BITS, 32, kModeKeys>;
  if constexpr (NB >= 64) {
    if (bt == 16) return (void*)enc_mfma<enc_planes(BITS), KS, BITS, NB, kModeBU, 16>;
  }
  if constexpr (NB <= 64) {
    if (bt == 1) return (void*)enc_mfma<enc_planes(BITS), KS, BITS, NB, kModeBU>;
  }
  return nullptr;
}

template <int KS, int BITS>
void* enc_by_nb(int nb, int mode, int bt) {
  switch (nb) {
    case 16: return enc_kernel<KS, BITS, 16>(mode, bt);
    case 32: return enc_kernel<KS, BITS, 32>(mode, bt);
    case 64: return enc_kernel<KS, BITS, 64>(mode, bt);
    case 128: return enc_kernel<KS, BITS, 128>(mode, bt);
  }
  return nullptr;
}

template <int KS>
void* enc_by_bits(int bits, int nb, int mode, int bt) {
  switch (bits) {
    case 2: return enc_by_nb<KS, 2>(nb, mode, bt);
    case 3: return enc_by_nb<KS, 3>(nb, mode, bt);
    case 4: return enc_by_nb<KS, 4>(nb, mode, bt);
    case 6: return enc_by_nb<KS, 6>(nb, mode, bt);
    case 8: return enc_by_nb<KS, 8>(nb, mode, bt);
  }
  return nullptr;
}

// (token-channel tiles: blocks of 64 or 128 channels, centred per (token, group) or per
// (token, block); per-token blocks spanning groups centred per (token, group); bf16 output on
// dec_centred's LDS ring)
template <int KS, int BITS, int NB>
void* dec_kernel(bool bf16, int bt, bool gsmall) {
  if constexpr (NB >= 64) {
    if (bt == 16) {
      if (bf16) return (void*)dec_centred<kNP, KS, BITS, NB, 16>;
      return (void*)dec_mfma<kNP, KS, BITS, NB, false, 16>;
    }
  }
  if constexpr (NB <= 64) {
    if (bt == 1) {
      if constexpr (KS == 2 && centred_stages(BITS, kD / NB, 1) >= 3) {
        if (bf16 && gsmall) return (void*)dec_centred<kNP, KS, BITS, NB, 1>;
      }
      if (bf16) return (void*)dec_mfma<kNP, KS, BITS, NB, true>;
      return (void*)dec_mfma<kNP, KS, BITS, NB, false>;
    }
  }
  return nullptr;
}

template <int KS, int BITS>
void* dec_by_nb(int nb, bool bf16, int bt, bool gsmall) {
  switch (nb) {
    case 16: return dec_kernel<KS, BITS, 16>(bf16, bt, gsmall);
    case 32: return dec_kernel<KS, BITS, 32>(bf16, bt, gsmall);
    case 64: return dec_kernel<KS, BITS, 64>(bf16, bt, gsmall);
    case 128: return dec_kernel<KS, BITS, 128>(bf16, bt, gsmall);
  }
  return nullptr;
}

template <int KS>
void* dec_by_bits(int bits, int nb, bool bf16, int bt, bool gsmall) {
  switch (bits) {
    case 2: return dec_by_nb<KS, 2>(nb, bf16, bt, gsmall);
    case 3: return dec_by_nb<KS, 3>(nb, bf16, bt, gsmall);
    case 4: return dec_by_nb<KS, 4>(nb, bf16, bt, gsmall);
    case 6: return dec_by_nb<KS, 6>(nb, bf16, bt, gsmall);
    case 8: return dec_by_nb<KS, 8>(nb, bf16, bt, gsmall);
  }
  return nullptr;
}

int ksteps(int g) { return g >= 128 ? 8 : (g == 64 ? 4 : 2); }

// dec_fast variants exist where a lane's code region is whole words and a wave's K range
// holds at most two blocks (one token's blocks; token-channel tiles take the centred decoder)
template <int KS, int BITS, int NB>
void* fast_kernel(bool bf16, int bt) {
  constexpr int SEG = (16 * KS < NB ? 16 * KS : NB) / 16;
  if constexpr (SEG * BITS % 4 == 0 && KS / SEG <= 2) {
    if constexpr (NB <= 64) {
      if (bt == 1) {
        if (bf16) return (void*)dec_fast<kNP, KS, BITS, NB, true>;
        return (void*)dec_fast<kNP, KS, BITS, NB, false>;
      }
    }
  }
  return nullptr;
}

template <int KS, int BITS>
void* fast_by_nb(int nb, bool bf16, int bt) {
  switch (nb) {
    case 16: return fast_kernel<KS, BITS, 16>(bf16, bt);
    case 32: return fast_kernel<KS, BITS, 32>(bf16, bt);
    case 64: return fast_kernel<KS, BITS, 64>(bf16, bt);
    case 128: return fast_kernel<KS, BITS, 128>(bf16, bt);
  }
  return nullptr;
}

template <int KS>
void* fast_by_bits(int bits, int nb, bool bf16, int bt) {
  switch (bits) {
    case 2: return fast_by_nb<KS, 2>(nb, bf16, bt);
    case 3: return fast_by_nb<KS, 3>(nb, bf16, bt);
    case 4: return fast_by_nb<KS, 4>(nb, bf16, bt);
    case 6: return fast_by_nb<KS, 6>(nb, bf16, bt);
    case 8: return fast_by_nb<KS, 8>(nb, bf16, bt);
  }
  return nullptr;
}

template <int KS, int BITS>
void* keys_kernel(bool bf16) {
  if (bf16) return (void*)dec_keys<kNP, KS, BITS, true>;
  return (void*)dec_keys<kNP, KS, BITS, false>;
}

template <int KS>
void* keys_by_bits(int bits, bool bf16) {
  switch (bits) {
    case 2: return keys_kernel<KS, 2>(bf16);
    case 3: return keys_kernel<KS, 3>(bf16);
    case 4: return keys_kernel<KS, 4>(bf16);
    case 6: return keys_kernel<KS, 6>(bf16);
    case 8: return keys_kernel<KS, 8>(bf16);
  }
  return nullptr;
}

bool group_ok(int g) { return g == 8 || g == 16 || g == 32 || g == 64 || g == 128; }

bool bits_ok(int b) { return b == 2 || b == 3 || b == 4 || b == 6 || b == 8; }

}  // namespace

bool mfma_encode_supported(const ViewDev& X, const GaugeDev& G, const CodecDev& c) {
  if (!X.bf16 || X.d != kD || !group_ok(G.g)) return false;
  if (c.backend == CG_BACKEND_PASSTHROUGH) return true;
  if (c.backend == CG_BACKEND_ZFP) return bits_ok(c.bits);
  if (c.backend == CG_BACKEND_KIVI)
    return bits_ok(c.bits) && c.kg == kTok && (c.kvc == 16 || c.kvc == 32 || c.kvc == 64) && c.win % kTok == 0;
  if (c.backend != CG_BACKEND_BLOCK_UNIFORM || !bits_ok(c.bits)) return false;
  if (c.bt == 16) return c.n == 64 || c.n == 128;  // token-channel tiles
  return c.bt == 1 && (c.n == 16 || c.n == 32 || c.n == 64);
}

bool mfma_decode_supported(int s, const ViewDev& Y, const GaugeDev& G, const CodecDev& c) {
  if (Y.d != kD || !group_ok(G.g) || !bits_ok(c.bits)) return false;
  if (c.backend == CG_BACKEND_ZFP) return true;
  if (c.backend == CG_BACKEND_BLOCK_UNIFORM && c.bt != 1)  // tiles: blocks inside a group, or centred groups
    return c.bt == 16 && (c.n == 64 || c.n == 128);
  if (c.backend == CG_BACKEND_KIVI) {
    if (c.win % kTok) return false;
    if (s == 0) return c.kg == kTok;  // one tile per key group
    return c.kvc == 16 || c.kvc == 32 || c.kvc == 64;  // values: block-uniform rows
  }
  return c.backend == CG_BACKEND_BLOCK_UNIFORM && (c.n == 16 || c.n == 32 || c.n == 64);
}

hipError_t launch_encode_mfma(int s, const ViewDev& X, int l0, const GaugeDev& G, const CodecDev& c,
                              const CacheDev& k, int t0, int tq, int* err, hipStream_t st) {
  if (X.T == 0) return hipSuccess;
  MfmaArgs m{};
  m.x = (char*)X.ptr;
  m.sl = X.sl; m.sb = X.sb; m.sh = X.sh; m.st = X.st;
  m.L = X.L; m.B = X.B; m.H = X.H; m.T = X.T;
  m.l0 = l0; m.s = s; m.t0 = t0;
  for (int p = 0; p < 3; ++p) m.gp[p] = G.hi[p];
  m.g32 = G.f32; m.g = G.g; m.R = G.R; m.Hg = G.H;
  m.codes = k.codes; m.side = k.side; m.T_cap = k.T_cap; m.cB = k.B; m.cH = k.H;
  m.err = err;
  const bool pass = c.backend == CG_BACKEND_PASSTHROUGH, kivi = c.backend == CG_BACKEND_KIVI;
  const bool zfp = c.backend == CG_BACKEND_ZFP;
  const bool tiles = c.backend == CG_BACKEND_BLOCK_UNIFORM && c.bt > 1;
  m.tq = kivi || tiles ? tq : X.T;
  m.ring = k.ring;
  m.ring_slots = kivi ? c.win + c.kg : (tiles ? c.bt : 0);
  const int mode = pass ? kModePass : (zfp ? kModeZfp : (kivi && s == 0 ? kModeKeys : kModeBU));
  const int nb = pass || zfp ? 64 : (kivi ? c.kvc : c.n), bits = pass ? 8 : c.bits, bt = tiles ? c.bt : 1;
  void* fn = nullptr;
  switch (ksteps(G.g)) {
    case 2: fn = enc_by_bits<2>(bits, nb, mode, bt); break;
    case 4: fn = enc_by_bits<4>(bits, nb, mode, bt); break;
    case 8: fn = enc_by_bits<8>(bits, nb, mode, bt); break;
  }
  if (!fn) return hipErrorInvalidValue;
  plan(m, X.L * X.B * X.H, X.T, fn);
  const int nwg = ((m.nslices * m.chunks + 7) / 8) * 8;
  void* args[] = {&m};
  return hipLaunchKernel(fn, dim3(nwg), dim3(kThreads), args, 0, st);
}

hipError_t launch_decode_mfma(int s, const CacheDev& k, int l0, const GaugeDev& G, const CodecDev& c, int t0,
                              int len, const int* pos, int pos_add, const ViewDev& Y, int* err, hipStream_t st) {
  if (Y.T == 0) return hipSuccess;
  MfmaArgs m{};
  m.x = (char*)Y.ptr;
  m.sl = Y.sl; m.sb = Y.sb; m.sh = Y.sh; m.st = Y.st;
  m.L = Y.L; m.B = Y.B; m.H = Y.H; m.T = Y.T;
  m.l0 = l0; m.s = s; m.t0 = t0;
  for (int p = 0; p < 3; ++p) m.gp[p] = G.tr[p];
  m.g32 = G.f32; m.cs8 = G.cs8; m.g = G.g; m.R = G.R; m.Hg = G.H;
  m.codes = k.codes; m.side = k.side; m.T_cap = k.T_cap; m.cB = k.B; m.cH = k.H;
  m.pos = pos;
  m.pos_add = pos_add;
  m.err = err;
  m.kivi = c.backend == CG_BACKEND_KIVI;
  m.win = c.win;
  m.kg = c.kg;
  m.len = len;
  m.ring = k.ring;
  const int bt = c.backend == CG_BACKEND_BLOCK_UNIFORM ? c.bt : 1;
  m.ring_slots = bt > 1 ? bt : c.win + c.kg;
  if (m.kivi && s == 0) {
    // one tile per 32-position key group: the first may start before t0
    void* fn = nullptr;
    switch (ksteps(G.g)) {
      case 2: fn = keys_by_bits<2>(c.bits, Y.bf16); break;
      case 4: fn = keys_by_bits<4>(c.bits, Y.bf16); break;
      case 8: fn = keys_by_bits<8>(c.bits, Y.bf16); break;
    }
    if (!fn) return hipErrorInvalidValue;
    plan(m, Y.L * Y.B * Y.H, t0 % kTok + Y.T, fn);
    const int nwg = ((m.nslices * m.chunks + 7) / 8) * 8;
    void* args[] = {&m};
    return hipLaunchKernel(fn, dim3(nwg), dim3(kThreads), args, 0, st);
  }
  if (c.backend == CG_BACKEND_ZFP) {
    void* fn = nullptr;
    switch (ksteps(G.g)) {
      case 2: fn = zfp_dec_by_rate<2>(c.bits, Y.bf16); break;
      case 4: fn = zfp_dec_by_rate<4>(c.bits, Y.bf16); break;
      case 8: fn = zfp_dec_by_rate<8>(c.bits, Y.bf16); break;
    }
    if (!fn) return hipErrorInvalidValue;
    plan(m, Y.L * Y.B * Y.H, Y.T, fn);
    const int nwg = ((m.nslices * m.chunks + 7) / 8) * 8;
    void* args[] = {&m};
    return hipLaunchKernel(fn, dim3(nwg), dim3(kThreads), args, 0, st);
  }
  const int nb = m.kivi ? c.kvc : c.n;
  void* fn = nullptr;
  if (G.g >= nb && bt == 1) {
    // blocks (of one token) inside one group: codes feed the matrix core without conversion
    switch (ksteps(G.g)) {
      case 2: fn = fast_by_bits<2>(c.bits, nb, Y.bf16, bt); break;
      case 4: fn = fast_by_bits<4>(c.bits, nb, Y.bf16, bt); break;
      case 8: fn = fast_by_bits<8>(c.bits, nb, Y.bf16, bt); break;
    }
  }
  if (!fn) {
    switch (ksteps(G.g)) {
      case 2: fn = dec_by_bits<2>(c.bits, nb, Y.bf16, bt, G.g < nb); break;
      case 4: fn = dec_by_bits<4>(c.bits, nb, Y.bf16, bt, G.g < nb); break;
      case 8: fn = dec_by_bits<8>(c.bits, nb, Y.bf16, bt, G.g < nb); break;
    }
  }
  if (!fn) return hipErrorInvalidValue;
  plan(m, Y.L * Y.B * Y.H, Y.T, fn);
  const int nwg = ((m.nslices * m.chunks + 7) / 8) * 8;
  void* args[] = {&m};
  return hipLaunchKernel(fn, dim3(nwg), dim3(kThreads), args, 0, st);
}

}  // namespace cg
