// Definitions shared by the matrix-core kernels (one copy per translation unit).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace cg {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

constexpr int kD = 128;          // head dimension handled here
constexpr int kTok = 32;         // tokens per tile (MFMA N)
constexpr int kThreads = 256;    // four waves
constexpr int kRowBytes = kD * 2;
// s_waitcnt immediate (gfx9 encoding: vmcnt[3:0] and [15:14], expcnt[6:4], lgkmcnt[11:8])
// waiting until at most `vm` vector-memory operations are outstanding, with lgkmcnt = 0 (all
// LDS operations of the wave done) and no wait on expcnt
constexpr int waitcnt_imm(int vm) { return (vm & 15) | ((vm >> 4) << 14) | (7 << 4) | (0 << 8); }

__device__ __forceinline__ int xcd_remap(int bid, int nwg) {
  // workgroups are dealt round-robin to the 8 XCDs; give each XCD a contiguous range of
  // logical workgroups so that the ranges of one slice share an L2
  const int per = nwg >> 3;
  return (bid & 7) * per + (bid >> 3);
}

// physical 16-byte granule of logical granule j in token row n
__device__ __forceinline__ int swz(int n, int j) { return j ^ (n & 15); }

__device__ __forceinline__ f32x16_t mfma(const bf16x8_t& a, const bf16x8_t& b, const f32x16_t& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ bf16x8_t as_bf16x8(const u32x4_t& v) { return __builtin_bit_cast(bf16x8_t, v); }

// a lane's value moved through DPP (all rows and banks enabled)
template <int CTRL>
__device__ __forceinline__ float dpp_mov(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
}
template <int CTRL>
__device__ __forceinline__ int dpp_mov_i(int v) {
  return __builtin_amdgcn_update_dpp(0, v, CTRL, 0xF, 0xF, false);
}

}  // namespace
}  // namespace cg
