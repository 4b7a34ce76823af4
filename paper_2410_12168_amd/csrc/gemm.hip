// gemm.hip -- W4Ax mixed-precision GEMM for gfx950 (paper Sec. 4).
//
// Operand path.  Both operands arrive as sign-magnitude codes.  A 4-bit chunk
// becomes FP8-E4M3 subnormal bytes (code * 2^-9) with two masks and one
// rotate per 8 codes; an 8-bit activation byte (sign, 7-bit magnitude m)
// becomes two such FP8 bytes, hi = m >> 3 (0..15) and lo = m & 7, so that
// code = 8 * hi + lo.  Each 16x16 output block of one K-block is one
// v_mfma_f32_16x16x128_f8f6f4 (K = 128 = one block) for W4A4 and two for
// W4A8.  Products of such codes are integers times 2^-18 and their sums stay
// below 2^24 units, so the fp32 MFMA result is the exact block sum (the
// paper's integer tile result, Sec. 4.1) and needs no int->float convert.
// Dequantization (Sec. 4.3, scale divided by the zero-extension factor):
//     C += Y * (sa * 2^18) * sw      in fp32, once per output and K-block.
#include <hip/hip_runtime.h>
#include <hip/hip_fp16.h>
#include <stdint.h>

#include "kernels.h"

namespace comet {

namespace {

typedef int i32x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr uint32_t kSignMag = 0x87878787u;
constexpr float kUnit = 262144.0f;  // 2^18: (2^-9)^2 of the FP8 code encoding

__device__ inline uint32_t rotr4(uint32_t w) { return __builtin_amdgcn_alignbit(w, w, 4); }

// 16 bytes of 4-bit codes (32 channels) -> 8 dwords of FP8 operand bytes.
__device__ inline i32x8 unpack4(uint4 v) {
  i32x8 r;
  r[0] = (int)(v.x & kSignMag);
  r[1] = (int)(rotr4(v.x) & kSignMag);
  r[2] = (int)(v.y & kSignMag);
  r[3] = (int)(rotr4(v.y) & kSignMag);
  r[4] = (int)(v.z & kSignMag);
  r[5] = (int)(rotr4(v.z) & kSignMag);
  r[6] = (int)(v.w & kSignMag);
  r[7] = (int)(rotr4(v.w) & kSignMag);
  return r;
}

// 32 bytes of 8-bit codes -> hi (|code| >> 3 with sign) and lo (|code| & 7 with sign).
__device__ inline void unpack8(uint4 a, uint4 b, i32x8& hi, i32x8& lo) {
  uint32_t w[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
  #pragma unroll
  for (int i = 0; i < 8; ++i) {
    lo[i] = (int)(w[i] & kSignMag);
    hi[i] = (int)(((w[i] >> 3) & 0x0F0F0F0Fu) | (w[i] & 0x80808080u));
  }
}

__device__ inline f32x4 mfma_fp8(i32x8 a, i32x8 b, f32x4 c) {
  // cbsz = blgp = 0: both operands OCP FP8-E4M3; zero scale operands select
  // the unscaled instruction.
  return __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a, b, c, 0, 0, 0, 0, 0, 0);
}

__device__ inline float h2f(uint16_t h) { return __half2float(__ushort_as_half(h)); }

// Data-parallel kernel: one 128x128 output tile per workgroup of 4 waves, each
// wave a 64x64 quadrant (4x4 blocks of 16x16).  Operands are read straight
// from global memory into registers.  All loads clamp their row/column into
// range, so edge tiles never read out of bounds; stores are masked.
template <bool DIAG>
__global__ __launch_bounds__(256) void gemm_simple_kernel(GemmArgs a) {
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int r16 = lane & 15;
  const int q4 = lane >> 4;
  const int tile = blockIdx.x;
  const int tm = tile / a.tiles_n;
  const int tn = tile % a.tiles_n;
  const int row0 = tm * kTileM + (wave >> 1) * 64;
  const int col0 = tn * kTileN + (wave & 1) * 64;
  const int M = a.M, N = a.N, K = a.K;
  const int NG = K / kG;
  const size_t wrow = (size_t)(K / 2);

  f32x4 C[4][4];
  #pragma unroll
  for (int i = 0; i < 4; ++i)
    #pragma unroll
    for (int j = 0; j < 4; ++j) C[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  int n8 = 0;  // 8-bit blocks before g (for the block-major A offset)
  for (int g = 0; g < NG; ++g) {
    const bool b8 = (a.map.bits[g >> 6] >> (g & 63)) & 1;
    const size_t abase = (size_t)M * 64 * (size_t)(g + n8);
    n8 += b8 ? 1 : 0;

    i32x8 wf[4];
    float swf[4];
    #pragma unroll
    for (int cb = 0; cb < 4; ++cb) {
      const int col = min(col0 + cb * 16 + r16, N - 1);
      uint4 v = *reinterpret_cast<const uint4*>(a.W + (size_t)col * wrow + (size_t)g * 64 + q4 * 16);
      wf[cb] = unpack4(v);
      swf[cb] = h2f(a.sw[(size_t)g * N + col]);
    }
    float saf[4][4];
    #pragma unroll
    for (int rb = 0; rb < 4; ++rb)
      #pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int row = min(row0 + rb * 16 + 4 * q4 + i, M - 1);
        saf[rb][i] = h2f(a.sa[(size_t)g * M + row]) * kUnit;
      }

    #pragma unroll
    for (int rb = 0; rb < 4; ++rb) {
      const int arow = min(row0 + rb * 16 + r16, M - 1);
      i32x8 af, ahi;
      if (b8) {
        const uint8_t* p = a.A + abase + (size_t)arow * 128 + q4 * 32;
        uint4 v0 = *reinterpret_cast<const uint4*>(p);
        uint4 v1 = *reinterpret_cast<const uint4*>(p + 16);
        unpack8(v0, v1, ahi, af);
      } else {
        uint4 v = *reinterpret_cast<const uint4*>(a.A + abase + (size_t)arow * 64 + q4 * 16);
        af = unpack4(v);
      }
      #pragma unroll
      for (int cb = 0; cb < 4; ++cb) {
        f32x4 y = mfma_fp8(af, wf[cb], f32x4{0.f, 0.f, 0.f, 0.f});
        if (b8) {
          f32x4 yh = mfma_fp8(ahi, wf[cb], f32x4{0.f, 0.f, 0.f, 0.f});
          #pragma unroll
          for (int i = 0; i < 4; ++i) y[i] = __builtin_fmaf(yh[i], 8.0f, y[i]);  // exact
        }
        if (DIAG) {
          const int col = col0 + cb * 16 + r16;
          #pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int row = row0 + rb * 16 + 4 * q4 + i;
            if (row >= a.win_m0 && row < a.win_m1 && col >= a.win_n0 && col < a.win_n1) {
              const size_t idx = ((size_t)(row - a.win_m0) * (a.win_n1 - a.win_n0) +
                                  (col - a.win_n0)) * NG + g;
              a.acc[idx] = (int32_t)(y[i] * kUnit);
            }
          }
        } else {
          #pragma unroll
          for (int i = 0; i < 4; ++i)
            C[rb][cb][i] = __builtin_fmaf(y[i], saf[rb][i] * swf[cb], C[rb][cb][i]);
        }
      }
    }
  }
  if (DIAG) return;
  #pragma unroll
  for (int rb = 0; rb < 4; ++rb)
    #pragma unroll
    for (int cb = 0; cb < 4; ++cb) {
      const int col = col0 + cb * 16 + r16;
      #pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int row = row0 + rb * 16 + 4 * q4 + i;
        if (row < M && col < N)
          a.out[(size_t)row * N + col] = __half_as_ushort(__float2half_rn(C[rb][cb][i]));
      }
    }
}

}  // namespace

hipError_t launch_gemm_simple(const GemmArgs& a, bool diag, hipStream_t stream) {
  const int tiles_m = (a.M + kTileM - 1) / kTileM;
  const int tiles = tiles_m * a.tiles_n;
  if (diag)
    hipLaunchKernelGGL(gemm_simple_kernel<true>, dim3(tiles), dim3(256), 0, stream, a);
  else
    hipLaunchKernelGGL(gemm_simple_kernel<false>, dim3(tiles), dim3(256), 0, stream, a);
  return hipGetLastError();
}

}  // namespace comet
