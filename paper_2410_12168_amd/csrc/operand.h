// operand.h -- device helpers shared by the W4Ax GEMM kernels (gfx950).
//
// Packed codes are sign-magnitude.  A 4-bit dword holds 8 codes laid out so
// that (w & 0x87878787) and (rotr(w, 4) & 0x87878787) are OCP FP8-E4M3
// subnormal bytes equal to code * 2^-9 (codes 0..3 and 4..7 of the dword).
// An 8-bit byte (sign, 7-bit magnitude m) splits into two such bytes,
// hi = m >> 3 (0..15) and lo = m & 7, with code = 8 * hi + lo (a 4-bit hi is
// exact too: with its top bit in the exponent field the byte is the first
// normal binade, (8 + (hi & 7)) * 2^-9).
// v_mfma_f32_16x16x128_f8f6f4 multiplies these exactly: products are integers
// times 2^-18 and a K-block's sum stays below 2^24 units, so the fp32 result
// is the exact integer block sum scaled by 2^-18.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace comet {
namespace {

typedef int i32x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr uint32_t kSignMag = 0x87878787u;
constexpr float kUnit = 262144.0f;  // 2^18: (2^-9)^2 of the FP8 code encoding

__device__ __forceinline__ uint32_t rotr4(uint32_t w) { return __builtin_amdgcn_alignbit(w, w, 4); }

// 16 bytes of 4-bit codes (32 channels) -> 32 FP8 bytes, natural channel order.
__device__ __forceinline__ void unpack4(u32x4 v, u32x4& lo, u32x4& hi) {
  lo = u32x4{v[0] & kSignMag, rotr4(v[0]) & kSignMag, v[1] & kSignMag, rotr4(v[1]) & kSignMag};
  hi = u32x4{v[2] & kSignMag, rotr4(v[2]) & kSignMag, v[3] & kSignMag, rotr4(v[3]) & kSignMag};
}

// 8-bit codes -> FP8 of the high part (|code| >> 3, signed) and low part (|code| & 7, signed).
__device__ __forceinline__ uint32_t hi8(uint32_t w) { return ((w >> 3) & 0x0F0F0F0Fu) | (w & 0x80808080u); }
__device__ __forceinline__ uint32_t lo8(uint32_t w) { return w & kSignMag; }

__device__ __forceinline__ f32x4 mfma_fp8(const i32x8& a, const i32x8& b, f32x4 c) {
  // cbsz = blgp = 0: both operands OCP FP8-E4M3; zero scale operands select
  // the unscaled instruction.
  return __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a, b, c, 0, 0, 0, 0, 0, 0);
}

// The same with A's products scaled by 2^3 through the instruction's E8M0
// block scales (130 for A on every lane, 127 = 2^0 for B): chained after the
// low part's MFMA it adds 8 * hi * w for the high parts of 8-bit codes into
// the same accumulator, exactly, with no vector instruction.
__device__ __forceinline__ f32x4 mfma_fp8_x8(const i32x8& a, const i32x8& b, f32x4 c) {
  return __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a, b, c, 0, 0, 0, (int)0x82828282u, 0,
                                                          0x7F7F7F7F);
}

__device__ __forceinline__ f32x4 scale_products(float sa, float sw) {
  // v_mfma_f32_4x4x1_16b_f32: lane l receives sa(lane 4*(l/4) + i) * sw(lane l)
  // for i = 0..3.  With lane j holding the activation scale of row
  // 4*(j/16) + (j & 3) and lane l the weight scale of column l & 15, that is the
  // 16x16 accumulator layout (row 4*(l/16) + i, column l & 15).  K = 1 and
  // both factors have 11-bit significands, so every product is exact in fp32.
  return __builtin_amdgcn_mfma_f32_4x4x1f32(sa, sw, f32x4{0.f, 0.f, 0.f, 0.f}, 0, 0, 0);
}

}  // namespace
}  // namespace comet
