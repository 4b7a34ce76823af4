// swiglu.h -- SwiGLU of the gate/up GEMM output, h = SiLU(gate) * up, in the
// fp32 steps the library's definition fixes (so that every kernel producing
// h gives the same bits):
//   exp(x): x clamped to [-87, 88]; k = rint(x * log2 e); r = x - k * ln2 in
//           two fmas with ln2 split into a 16-bit-exact high part and a low
//           part (Cody-Waite); p = Taylor series of e^r to degree 7 in Horner
//           form (fmas); result ldexp(p, k);
//   SiLU(x) = x * (1 / (1 + exp(-x)));
//   h = fp16(SiLU(g) * u) for fp16 g and u.
// Gate and up columns come in 2G-wide groups (gate of channels jG .. jG+G-1,
// then up of the same channels), so one 256-column GEMM tile holds both halves
// of G = 128 channels: one input block of the next (down) projection.
#pragma once

#include <hip/hip_runtime.h>
#include <hip/hip_fp16.h>
#include <stdint.h>

namespace comet {

__device__ __forceinline__ float exp_f32(float x) {
  x = fminf(fmaxf(x, -87.0f), 88.0f);
  const float log2e = 1.44269504088896341f;
  const float ln2_hi = 0.693145751953125f;
  const float ln2_lo = 1.42860682030941723e-6f;
  const float k = rintf(x * log2e);
  float r = fmaf(-k, ln2_hi, x);
  r = fmaf(-k, ln2_lo, r);
  float p = 1.98412698412698413e-4f;  // 1/7!
  p = fmaf(p, r, 1.38888888888888889e-3f);
  p = fmaf(p, r, 8.33333333333333333e-3f);
  p = fmaf(p, r, 4.16666666666666667e-2f);
  p = fmaf(p, r, 1.66666666666666667e-1f);
  p = fmaf(p, r, 0.5f);
  p = fmaf(p, r, 1.0f);
  p = fmaf(p, r, 1.0f);
  return ldexpf(p, (int)k);
}

__device__ __forceinline__ float silu_f32(float x) { return x * (1.0f / (1.0f + exp_f32(-x))); }

// h for fp16 bit patterns g and u, as fp16 bits.
__device__ __forceinline__ uint16_t swiglu_f16(uint16_t g, uint16_t u) {
  const float gf = __half2float(__ushort_as_half(g));
  const float uf = __half2float(__ushort_as_half(u));
  return __half_as_ushort(__float2half_rn(silu_f32(gf) * uf));
}

}  // namespace comet
