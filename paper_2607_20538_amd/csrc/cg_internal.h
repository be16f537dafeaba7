// Internal declarations shared by the host entry points and the kernel translation units of
// the gauge-coded KV codec library.  Not part of the C ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "codec_gauge.h"

namespace cg {

// Split planes of G^T the matrix-core decoders multiply (G^T ~= tr[0] + tr[1]).
constexpr int kDecPlanes = 2;

// Device gauge buffer (filled by gauge_make):
//   f32  : G            [nblk][g][g] binary32, nblk = L*2*H*R, block ((l*2+s)*H+h)*R+r
//   hi[p]: split planes of G,   bf16 [nblk][g][g], G ~= hi[0] + hi[1] + hi[2]
//   tr[p]: split planes of G^T, bf16 [nblk][g][g] (block transposed)
//   cs8  : decoder column sums, binary32 [L*2*H][d/8][d]: entry (head, c, i) is the sum over
//          the 8 channels j of segment c that share i's group of tr[0][i][j] + tr[1][i][j]
//          (summed exactly, rounded once), head = (l*2+s)*H+h
// Every section starts on a 256-byte boundary.
struct GaugeLayout {
  int64_t nblk = 0, nhead = 0;
  int g = 0, d = 0;
  size_t off_f32 = 0, off_hi[3] = {0, 0, 0}, off_tr[3] = {0, 0, 0}, off_cs8 = 0, total = 0;
};

inline size_t align256(size_t v) { return (v + 255) & ~size_t(255); }

inline GaugeLayout gauge_layout(const cg_gauge_shape& s) {
  GaugeLayout gl;
  if (s.L <= 0 || s.H <= 0 || s.d <= 0 || s.g <= 0 || s.d % s.g) return gl;
  gl.g = s.g;
  gl.nblk = int64_t(s.L) * 2 * s.H * (s.d / s.g);
  size_t gg = size_t(s.g) * s.g;
  size_t off = 0;
  gl.off_f32 = off;
  off = align256(off + gl.nblk * gg * 4);
  for (int p = 0; p < 3; ++p) {
    gl.off_hi[p] = off;
    off = align256(off + gl.nblk * gg * 2);
  }
  for (int p = 0; p < 3; ++p) {
    gl.off_tr[p] = off;
    off = align256(off + gl.nblk * gg * 2);
  }
  gl.d = s.d;
  gl.nhead = int64_t(s.L) * 2 * s.H;
  gl.off_cs8 = off;
  off = align256(off + size_t(gl.nhead) * (s.d / 8) * s.d * 4);
  gl.total = off;
  return gl;
}

// Kernel-side description of the gauge buffer.
struct GaugeDev {
  const float* f32;
  const uint16_t* hi[3];
  const uint16_t* tr[3];
  const float* cs8;
  int g, R, H;
};

// Codec parameters as the kernels see them.
struct CodecDev {
  int backend, bits, n, kg, kvc, win;
  int bt;  // block-uniform tile tokens (1: one token per block); 1 for the other backends
};

// A strided KV tensor view [L][B][H][T][d] (element strides, channel stride 1).
struct ViewDev {
  void* ptr;
  int64_t sl, sb, sh, st;
  int L, B, H, T, d;
  int bf16;
};

// A compressed cache of one type s.
struct CacheDev {
  uint8_t* codes;
  uint32_t* side;      // one 32-bit word (min | scale << 16) per block
  uint16_t* ring;      // KIVI window, or the staging window of block-uniform tiles
  int L, B, H, T_cap, d;
};

// Paged caches: batch row b's position t lives in cache row (page, t mod page_size) with
// page = pages[b * max_pages + t / page_size] (the cache's batch dimension is the page pool);
// pages == nullptr: row b is cache batch row b.
struct PageDev {
  const int* pages = nullptr;
  int max_pages = 0, page_size = 0;
};

// Generic (VALU) kernels: every supported configuration.
hipError_t launch_encode_generic(int s, const ViewDev& X, int l0, const GaugeDev& G, const CodecDev& c,
                                 const CacheDev& k, int t0, int tq, int* err, hipStream_t st,
                                 const PageDev& pt = PageDev());
hipError_t launch_decode_generic(int s, const CacheDev& k, int l0, const GaugeDev& G, const CodecDev& c, int t0,
                                 int len, const int* pos, int pos_add, const ViewDev& Y, int* err, hipStream_t st);

// Matrix-core kernels: bf16, head dimension 128, block-uniform (n in {16, 32, 64}) or passthrough.
bool mfma_encode_supported(const ViewDev& X, const GaugeDev& G, const CodecDev& c);
bool mfma_decode_supported(int s, const ViewDev& Y, const GaugeDev& G, const CodecDev& c);
hipError_t launch_encode_mfma(int s, const ViewDev& X, int l0, const GaugeDev& G, const CodecDev& c,
                              const CacheDev& k, int t0, int tq, int* err, hipStream_t st);
hipError_t launch_decode_mfma(int s, const CacheDev& k, int l0, const GaugeDev& G, const CodecDev& c, int t0,
                              int len, const int* pos, int pos_add, const ViewDev& Y, int* err, hipStream_t st);

// Spectral statistics (section 4.2): workspace sections (bytes from the start, 256-aligned):
// energy sums binary64 [L][Tb][d], log sums binary64 [L], DCT-II rows binary64 [d][d], and for
// d = 128 the two bf16 planes of M = C_d G, [L][H][d][d] each.
struct SpecLayout {
  size_t off_acc = 0, off_lsum = 0, off_cd = 0, off_m[2] = {0, 0}, total = 0;
};
SpecLayout spec_layout(const cg_gauge_shape& s, int Tb);
hipError_t launch_spectral(int s, const ViewDev& X, const GaugeDev& G, int Tb, float tau, void* ws, double* stats,
                           double* energy, bool force_generic, hipStream_t st);

// Gradient of the training objective with respect to the gauge generators: workspace layout
// (the spectral statistics' own workspace first) and launch.
struct GradLayout {
  size_t off_m = 0, off_part = 0, off_dm = 0, off_work = 0, total = 0;
  int chunks = 1, blocks_per_wg = 1;
};
GradLayout grad_layout(const cg_gauge_shape& s, int B, int T, int Tb);
hipError_t launch_gauge_grad(int s, const ViewDev& X, const GaugeDev& G, const float* A, int Tb, float tau, float lam_f,
                             float lam_r, void* ws, double* stats, double* grad, bool force_generic, hipStream_t st);

// Decode-phase attention over the compressed caches (inverse gauge folded into the query and
// the output).  Query heads j = h * grp + jj of KV head h read that head's K / V caches.
struct AttendDev {
  ViewDev q, o;          // [nl][B][Hq][1][d]
  CacheDev kc, vc;
  int l0, Hq, grp;       // cache layer of view layer 0, query heads, query heads per KV head
  const int* lens;       // device [B] positions per batch row, or nullptr: every row holds `len`
  int len;
  float scale;
  int nsplit, chunk;     // token splits per row and tokens per split (a multiple of 64)
  int nqc;               // query chunks of at most 8 heads per workgroup
  float* part;           // partial results [nl][B][Hq][nsplit][2 + 2d] when nsplit > 1
  int* err;
  PageDev pt;            // paged caches (block-uniform per-token blocks or passthrough)
  int cap;               // positions a row can hold: T_cap, or max_pages * page_size
  int win;               // KIVI window (set by the launch for the matrix-core kernel)
};
struct AttendPlan {
  int nsplit = 1, chunk = 64, nqc = 1;
  size_t ws_bytes = 0;
};
// Split plan of a call covering `span` positions per row (the same rule sizes the workspace
// from the capacity, so a plan for span <= T_cap never needs more than that workspace).
AttendPlan attend_plan(int nl, int B, int H, int Hq, int d, int span);
hipError_t launch_attend(const AttendDev& a, const GaugeDev& G, const CodecDev& c, bool force_generic,
                         hipStream_t st);
// Library-owned scratch of kv_attend_noalloc: its size, and its device address on the current
// device (looked up once per device; the address, never the array's host-side name, goes to
// kernels).
size_t attend_scratch_bytes();
hipError_t attend_scratch(void** ptr);

// HBM streaming probe (read_bytes a multiple of 8 KB, write_bytes of 16 bytes).
hipError_t launch_stream_probe(const void* src, int64_t read_bytes, void* dst, int64_t write_bytes, hipStream_t st);

// Device self-test of the quantiser's division-free steps (which: 0 reciprocal, 1 division).
hipError_t launch_selftest(int which, unsigned long long* bad, hipStream_t st);

// Dispatching launchers (hip stream passed through).  All validate nothing: the host entry points do.
// Encode tokens [0, X.T) of view X into cache positions [t0, t0 + X.T); layer l of the view is
// cache layer l + l0.  tq: KIVI / tile tokens to quantise (others go to the window).
hipError_t launch_encode(int s, const ViewDev& X, int l0, const GaugeDev& G, const CodecDev& c, const CacheDev& k,
                         int t0, int tq, int* err, hipStream_t st);
// Decode cache positions [t0, t0 + Y.T) into view Y (layer l of Y is cache layer l + l0).
// If pos is non-NULL, batch row b holds pos[b] + pos_add tokens (a rolling step passes its
// positions with pos_add = 1, kv_decode its per-row lengths with pos_add = 0) and only the
// positions it holds are written (a count outside [0, T_cap] flags CG_FLAG_POS_RANGE and skips
// the row); otherwise every row holds `len` tokens (KIVI window and tile staging split).
hipError_t launch_decode(int s, const CacheDev& k, int l0, const GaugeDev& G, const CodecDev& c, int t0, int len,
                         const int* pos, int pos_add, const ViewDev& Y, int* err, hipStream_t st);
// Rolling append of one token per (layer, b, h) at pos[b] (layer l of Xn is cache layer l + l0).
hipError_t launch_append(int s, const ViewDev& Xn, int l0, const int* pos, const GaugeDev& G, const CodecDev& c,
                         const CacheDev& k, int* err, hipStream_t st, const PageDev& pt = PageDev());

}  // namespace cg
