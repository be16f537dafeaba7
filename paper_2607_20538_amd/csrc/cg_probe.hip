// HBM streaming probe: the memory pattern of the codec kernels without their arithmetic.
//
// Each workgroup streams a contiguous range of 8 KB source tiles global -> LDS with
// LDS-direct loads (a ring of five tiles, four in flight, one barrier per tile, as in the
// encoder) and, after each tile, writes its share of a contiguous destination range with
// 16-byte stores of data read back from the tile.  Its rate is the ceiling a kernel that reads
// `read_bytes` and writes `write_bytes` in one pass can reach on the device: HBM read and write
// streams interleaved in one kernel run slower than either stream alone.  The larger of the two
// streams carries the non-temporal policy, as in the codec kernels.
#include "cg_internal.h"
#include "cg_mfma_util.h"

namespace cg {
namespace {

constexpr int kProbeTile = 8192;  // bytes per tile: four waves x two 1 KB LDS-direct loads
constexpr int kProbeStages = 5;

template <bool NT_LOADS>
__global__ __launch_bounds__(kThreads, 3) void stream_probe(const char* __restrict__ src, int64_t ntiles,
                                                             char* __restrict__ dst, int64_t ngran) {
  __shared__ __attribute__((aligned(16))) uint8_t ring[kProbeStages][kProbeTile];
  const int lane = threadIdx.x & 63;
  const int wu = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int64_t nwg = gridDim.x, wg = blockIdx.x;
  const int64_t t0 = ntiles * wg / nwg, t1 = ntiles * (wg + 1) / nwg;
  const int64_t g0 = ngran * wg / nwg, g1 = ngran * (wg + 1) / nwg;
  const int nt = int(t1 - t0);
  if (nt <= 0) return;
  auto issue = [&](int t) {
    uint8_t* d = ring[t % kProbeStages] + 2048 * wu;
    const char* s = src + (t0 + t) * kProbeTile + 2048 * wu + 16 * lane;
#pragma unroll
    for (int q = 0; q < 2; ++q)
      __builtin_amdgcn_global_load_lds(s + 1024 * q, (__attribute__((address_space(3))) void*)(d + 1024 * q), 16, 0,
                                       NT_LOADS ? kLoadStreamPolicy : 0);
  };
  for (int t = 0; t < min(nt, kProbeStages - 1); ++t) issue(t);
  for (int t = 0; t < nt; ++t) {
    // tile t's loads landed (the loads of up to three later tiles may stay in flight; the
    // stores issued after them only make the count stricter)
    switch (min(nt - 1 - t, kProbeStages - 2)) {
      case 0: __builtin_amdgcn_s_waitcnt(waitcnt_imm(0)); break;
      case 1: __builtin_amdgcn_s_waitcnt(waitcnt_imm(2)); break;
      case 2: __builtin_amdgcn_s_waitcnt(waitcnt_imm(4)); break;
      default: __builtin_amdgcn_s_waitcnt(waitcnt_imm(6)); break;
    }
    __builtin_amdgcn_s_barrier();
    if (t + kProbeStages - 1 < nt) issue(t + kProbeStages - 1);
    // this tile's share of the destination granules
    const int64_t a = g0 + (g1 - g0) * t / nt, b = g0 + (g1 - g0) * (t + 1) / nt;
    const uint8_t* tile = ring[t % kProbeStages];
    for (int64_t gi = a + threadIdx.x; gi < b; gi += kThreads) {
      const u32x4_t v = *(const u32x4_t*)(tile + 16 * ((gi - a) & (kProbeTile / 16 - 1)));
      if constexpr (NT_LOADS) *(u32x4_t*)(dst + 16 * gi) = v;
      else store_stream(dst + 16 * gi, v);
    }
  }
}

}  // namespace

hipError_t launch_stream_probe(const void* src, int64_t read_bytes, void* dst, int64_t write_bytes, hipStream_t st) {
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess || hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
    cus = 256;
  const int64_t ntiles = read_bytes / kProbeTile;
  int64_t nwg = int64_t(3) * cus;
  if (nwg > ntiles) nwg = ntiles > 0 ? ntiles : 1;
  hipLaunchKernelGGL(read_bytes >= write_bytes ? stream_probe<true> : stream_probe<false>, dim3(unsigned(nwg)), dim3(kThreads), 0, st, static_cast<const char*>(src), ntiles,
                     static_cast<char*>(dst), write_bytes / 16);
  return hipGetLastError();
}

}  // namespace cg
