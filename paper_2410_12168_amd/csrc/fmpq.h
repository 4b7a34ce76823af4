// fmpq.h -- device helpers of the FMPQ block quantizer (paper Sec. 3.2),
// shared by the quantization kernels and the GEMM epilogue that quantizes its
// output for the next layer.
//
// A lane holds 8 consecutive channels of one (row, block) pair and 16 lanes
// hold the block.  Scale and codes follow the block quantizer exactly:
// s = fp16_rne(RN(amax / qmax)), then per element
// q = clamp(rint(RN(x / s)), -qmax, qmax), packed sign-magnitude; every
// division is the correctly rounded quotient, computed as below.
//
// Division.  The codes need RN(x / s) exactly (IEEE fp32 division), which as
// a library division costs about ten vector instructions per element and made
// these kernels ALU-bound.  Instead each lane takes one reciprocal r within
// one ulp of 1/s (RN(1/s), or the hardware reciprocal) and per element
//     q0 = RN(x r),  rem = x - q0 s  (one fma, exact),  q = RN(q0 + rem r),
// Markstein's correction step.  Why q = RN(x / s) here: s is a binary16
// value, so its significand has at most 11 bits.  q0 is within 2 ulps of x/s,
// so rem is a multiple of ulp(q0) * 2^e(s) of at most 13 bits: exact.  The
// fma then sees x/s perturbed by at most |rem| |r - 1/s| <= 2^-45 ulp-units
// of the result, while x/s, when it is not a midpoint between binary32
// neighbours, lies at least 2^-35 units from one (x has 24 bits, s 11 bits),
// and it is never exactly a midpoint (a midpoint needs 25 significant bits
// times s's odd part).  So rounding the perturbed value gives RN(x / s).  The
// identity is also checked exhaustively on the CPU, over every binary16
// operand pair and with r = RN(1/s) and both of its neighbours.  s == 0 takes
// r = 0, which yields q = 0 as the quantizer requires.
//
#pragma once

#include <hip/hip_runtime.h>
#include <hip/hip_fp16.h>
#include <stdint.h>

#include "kernels.h"

namespace comet {
namespace {

struct Codes {
  uint32_t sign[8];
  uint32_t mag[8];
};

// RN(a / s) from r = RN(1/s) for a binary16 s (see above).
__device__ inline float div_rn(float a, float s, float r) {
  const float q0 = a * r;
  const float rem = fmaf(-q0, s, a);
  return fmaf(rem, r, q0);
}

// Magnitudes and signs follow q = clamp(rint(x / s), -qmax, qmax) with the
// sign taken from x (rint and the division are symmetric); a zero code has a
// clear sign bit.  Both divisions go through div_rn: the scale RN(amax / qmax)
// with the constant RN(1/qmax), the codes with r from the hardware
// reciprocal.  div_rn needs r within one ulp of 1/s, not correctly rounded
// (the margin argument above has room to spare); v_rcp_f32 is within one ulp,
// and both neighbours of RN(1/s) are checked exhaustively on the CPU, as is
// every amax / qmax.
__device__ inline uint16_t quantize8(const float (&x)[8], float amax, float qmax, Codes& c) {
  const float rq = qmax == 127.0f ? 1.0f / 127.0f : 1.0f / 7.0f;  // folded: RN(1/qmax)
  float s32 = div_rn(amax, qmax, rq);
  __half h = __float2half_rn(s32);
  float s = __half2float(h);
  const float r = s != 0.0f ? __builtin_amdgcn_rcpf(s) : 0.0f;
  #pragma unroll
  for (int i = 0; i < 8; ++i) {
    const float m = fminf(rintf(div_rn(fabsf(x[i]), s, r)), qmax);
    c.mag[i] = (uint32_t)m;
    c.sign[i] = (__float_as_uint(x[i]) >> 31) & (m != 0.0f ? 1u : 0u);
  }
  return __half_as_ushort(h);
}

// Sign-magnitude 4-bit codes of channels 0..7 into one dword.  Byte k:
//   bit 7 = sign(k), bits 6..4 = |code 4+k|, bit 3 = sign(4+((k+3)&3)), bits 2..0 = |code k|,
// so that (w & 0x87878787) and (rotr(w, 4) & 0x87878787) are FP8-E4M3 subnormals.
__device__ inline uint32_t pack4(const Codes& c) {
  uint32_t w = 0;
  #pragma unroll
  for (int k = 0; k < 4; ++k) {
    uint32_t b = (c.sign[k] << 7) | (c.mag[4 + k] << 4) | (c.sign[4 + ((k + 3) & 3)] << 3) | c.mag[k];
    w |= b << (8 * k);
  }
  return w;
}

__device__ inline uint2 pack8(const Codes& c) {
  uint32_t w0 = 0, w1 = 0;
  #pragma unroll
  for (int k = 0; k < 4; ++k) {
    w0 |= ((c.sign[k] << 7) | c.mag[k]) << (8 * k);
    w1 |= ((c.sign[4 + k] << 7) | c.mag[4 + k]) << (8 * k);
  }
  return make_uint2(w0, w1);
}

__device__ inline void load8(const uint16_t* p, float (&x)[8]) {
  uint4 v = *reinterpret_cast<const uint4*>(p);
  uint32_t w[4] = {v.x, v.y, v.z, v.w};
  #pragma unroll
  for (int i = 0; i < 4; ++i) {
    x[2 * i] = __half2float(__ushort_as_half((unsigned short)(w[i] & 0xFFFF)));
    x[2 * i + 1] = __half2float(__ushort_as_half((unsigned short)(w[i] >> 16)));
  }
}

// v from the lane that the DPP control selects within its 16-lane row
#define COMET_DPP_F32(v, ctrl) \
  __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), ctrl, 0xF, 0xF, false))

__device__ inline float max16(float v) {
  // max over the 16 lanes of one (row, block) pair, within the DPP row: the
  // quad butterflies (quad_perm [1,0,3,2] and [2,3,0,1]) give every lane its
  // quad's max, rotating the row by 4 and then 8 lanes combines the four quads
  v = fmaxf(v, COMET_DPP_F32(v, 0xB1));
  v = fmaxf(v, COMET_DPP_F32(v, 0x4E));
  v = fmaxf(v, COMET_DPP_F32(v, 0x124));
  v = fmaxf(v, COMET_DPP_F32(v, 0x128));
  return v;
}

__device__ inline int n8_before(const BlockMap& map, int g) {
  int n = 0;
  for (int w = 0; w < (g >> 6); ++w) n += __popcll(map.bits[w]);
  if (g & 63) n += __popcll(map.bits[g >> 6] & ((1ull << (g & 63)) - 1));
  return n;
}

}  // namespace
}  // namespace comet
