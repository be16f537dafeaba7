// Exhaustive device self-test of the binary32 steps of the quantiser that replace a division:
// the block range divided by 2^b - 1 and the reciprocal of a binary16 scale must equal
// correctly rounded division bit for bit (the CPU oracle divides with IEEE binary32 division);
// and of the binary16 directed roundings done by the hardware conversion under a rounding mode.
#include "cg_internal.h"
#include "cg_device.h"

namespace cg {
namespace {

// every positive finite binary16 value s: rcp_of_f16(s) == RN(1 / s)
__global__ void selftest_rcp(unsigned long long* bad) {
  const uint32_t h = blockIdx.x * blockDim.x + threadIdx.x + 1;
  if (h > 0x7bffu) return;
  const float s = f16_bits_to_f32(h);
  const float a = rcp_of_f16(s), b = __fdiv_rn(1.0f, s);
  if (__float_as_uint(a) != __float_as_uint(b)) atomicAdd(bad, 1ull);
}

// Binary32 division by a constant depends only on the dividend's significand while all
// intermediates stay normal, so one full binade proves every binade of normal results; the
// lowest binades (subnormal results) and the top ones (overflow) are checked in full too.
// A mismatch counts when the binary16 scale the quantiser derives (rounded up) differs.
__global__ void selftest_div(unsigned long long* bad, int bits, uint32_t exp_lo, uint32_t exp_hi) {
  const float d = float((1 << bits) - 1);
  const uint64_t n = uint64_t(exp_hi - exp_lo) << 23;
  for (uint64_t i = uint64_t(blockIdx.x) * blockDim.x + threadIdx.x; i < n; i += uint64_t(gridDim.x) * blockDim.x) {
    const uint32_t u = (exp_lo << 23) + uint32_t(i);
    const float a = __uint_as_float(u);
    const float x = div_by_qmax(a, bits), y = __fdiv_rn(a, d);
    if (f16_bits_up(x) != f16_bits_up(y)) atomicAdd(bad, 1ull);
  }
}

// binary16 rounding toward -inf / +inf by the hardware conversion under a directed mode
// against the software rounding, for every binary32 value of both signs whose exponent field
// lies in [exp_lo, exp_hi)
__global__ void selftest_f16_directed(unsigned long long* bad, uint32_t exp_lo, uint32_t exp_hi) {
  const uint64_t n = uint64_t(exp_hi - exp_lo) << 24;
  for (uint64_t i = uint64_t(blockIdx.x) * blockDim.x + threadIdx.x; i < n; i += uint64_t(gridDim.x) * blockDim.x) {
    const uint32_t u = ((exp_lo << 23) + uint32_t(i >> 1)) | (uint32_t(i & 1) << 31);
    const float v = __uint_as_float(u);
    if (f16_bits_down_hw(v) != f16_bits_down(v) || f16_bits_up_hw(v) != f16_bits_up(v)) atomicAdd(bad, 1ull);
  }
}

}  // namespace

hipError_t launch_selftest(int which, unsigned long long* bad, hipStream_t st) {
  if (which == 0) {
    hipLaunchKernelGGL(selftest_rcp, dim3((0x7bff + 255) / 256), dim3(256), 0, st, bad);
    return hipGetLastError();
  }
  if (which == 2) {
    // every binary32 value of both signs with exponent field 0 .. 255: zeros, subnormals,
    // normals, the infinities and the NaNs (a NaN converts to a NaN both ways)
    hipLaunchKernelGGL(selftest_f16_directed, dim3(8192), dim3(256), 0, st, bad, 0u, 256u);
    return hipGetLastError();
  }
  const int widths[5] = {2, 3, 4, 6, 8};
  const uint32_t ranges[4][2] = {{0, 4}, {100, 104}, {127, 128}, {250, 255}};
  for (int b : widths)
    for (const auto& r : ranges) {
      hipLaunchKernelGGL(selftest_div, dim3(2048), dim3(256), 0, st, bad, b, r[0], r[1]);
      hipError_t e = hipGetLastError();
      if (e != hipSuccess) return e;
    }
  return hipSuccess;
}

}  // namespace cg
