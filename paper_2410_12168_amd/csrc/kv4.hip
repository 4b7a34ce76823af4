// kv4.hip -- 4-bit asymmetric group quantization of the KV cache for gfx950.
//
// The KV cache feeds the memory-bound attention operator, so it is stored in
// 4 bits regardless of compute granularity (Sec. 3.2), with channel-wise
// asymmetric INT4 groups (Sec. 6 setup).  A group is G consecutive channels of
// one token's K or V row; per group
//   mn = min x, mx = max x (zero extremes as +0),  s = fp16(fp32(mx - mn) / 15),
//   q  = clamp(rint(fp32(fp32(x - mn) / s)), 0, 15)   (0 when s == 0),
// and the reconstruction is fp16(fp32(q * s) + mn).
//
// Layout: codes [T][C/2] bytes (channel 2j in the low nibble of byte j),
// params fp16 [T][C/G][2] = {s, mn}.
//
// The division (x - mn) / s uses one correctly rounded reciprocal per lane and
// Markstein's correction step (two fmas per element), exact for a binary16 s;
// fmpq.h gives the argument.
//
// Work decomposition: a lane owns 8 consecutive channels (one 16-byte load);
// G/8 lanes share a group and reduce min/max with xor shuffles.  Groups are
// numbered row-major, so a wave reads 1 KB of contiguous fp16 and writes
// 256 B of contiguous codes.  HBM-bound: 2 bytes in, 0.5 byte out per channel
// plus 4 bytes per group.
#include <hip/hip_runtime.h>
#include <hip/hip_fp16.h>
#include <stdint.h>

#include "kernels.h"

namespace comet {

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

template <int L>
__device__ inline float group_min(float v) {
  #pragma unroll
  for (int o = 1; o < L; o <<= 1) v = fminf(v, __shfl_xor(v, o, L));
  return v;
}

template <int L>
__device__ inline float group_max(float v) {
  #pragma unroll
  for (int o = 1; o < L; o <<= 1) v = fmaxf(v, __shfl_xor(v, o, L));
  return v;
}

// L = G / 8 lanes per group; element offset of a lane = 8 * (global lane id).
template <int L>
__global__ __launch_bounds__(256) void kv4_quantize_kernel(const uint16_t* __restrict__ X,
                                                           uint8_t* __restrict__ codes,
                                                           uint16_t* __restrict__ params,
                                                           long long nlanes) {
  const long long t = (long long)blockIdx.x * 256 + threadIdx.x;
  const bool valid = t < nlanes;
  const long long tc = valid ? t : nlanes - 1;
  // read once: nontemporal, so the rows do not displace cached data
  const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(X + 8 * tc));
  uint32_t w[4] = {v.x, v.y, v.z, v.w};
  float x[8];
  #pragma unroll
  for (int i = 0; i < 4; ++i) {
    x[2 * i] = __half2float(__ushort_as_half((unsigned short)(w[i] & 0xFFFF)));
    x[2 * i + 1] = __half2float(__ushort_as_half((unsigned short)(w[i] >> 16)));
  }
  float mn = x[0], mx = x[0];
  #pragma unroll
  for (int i = 1; i < 8; ++i) {
    mn = fminf(mn, x[i]);
    mx = fmaxf(mx, x[i]);
  }
  mn = group_min<L>(mn);
  mx = group_max<L>(mx);
  // zero extremes as +0: fminf / fmaxf may keep either zero of a +0 / -0 tie
  if (mn == 0.0f) mn = 0.0f;
  if (mx == 0.0f) mx = 0.0f;
  const float range = mx - mn;
  const __half h = __float2half_rn(range / 15.0f);
  const float s = __half2float(h);
  const float r = s != 0.0f ? 1.0f / s : 0.0f;  // s == 0 gives q = 0
  uint32_t packed = 0;
  #pragma unroll
  for (int i = 0; i < 8; ++i) {
    const float a = x[i] - mn;
    const float q0 = a * r;
    const float q = fmaf(fmaf(-q0, s, a), r, q0);  // RN(a / s)
    packed |= (uint32_t)fminf(rintf(q), 15.0f) << (4 * i);
  }
  if (!valid) return;
  // the cache is read back much later: keep the codes out of the caches too
  __builtin_nontemporal_store(packed, reinterpret_cast<uint32_t*>(codes + 4 * tc));
  if ((threadIdx.x & (L - 1)) == 0) {
    const uint32_t p = (uint32_t)__half_as_ushort(h) |
                       ((uint32_t)__half_as_ushort(__float2half_rn(mn)) << 16);
    *reinterpret_cast<uint32_t*>(params + 2 * (tc / L)) = p;
  }
}

template <int L>
__global__ __launch_bounds__(256) void kv4_dequantize_kernel(const uint8_t* __restrict__ codes,
                                                             const uint16_t* __restrict__ params,
                                                             uint16_t* __restrict__ out,
                                                             long long nlanes) {
  const long long t = (long long)blockIdx.x * 256 + threadIdx.x;
  if (t >= nlanes) return;
  const uint32_t q = *reinterpret_cast<const uint32_t*>(codes + 4 * t);
  const uint32_t p = *reinterpret_cast<const uint32_t*>(params + 2 * (t / L));
  const float s = __half2float(__ushort_as_half((unsigned short)(p & 0xFFFF)));
  const float mn = __half2float(__ushort_as_half((unsigned short)(p >> 16)));
  uint32_t o[4];
  #pragma unroll
  for (int i = 0; i < 4; ++i) {
    const float p0 = (float)((q >> (8 * i)) & 15u) * s;
    const float p1 = (float)((q >> (8 * i + 4)) & 15u) * s;
    const uint32_t lo = __half_as_ushort(__float2half_rn(p0 + mn));
    const uint32_t hi = __half_as_ushort(__float2half_rn(p1 + mn));
    o[i] = lo | (hi << 16);
  }
  *reinterpret_cast<uint4*>(out + 8 * t) = make_uint4(o[0], o[1], o[2], o[3]);
}


}  // namespace

hipError_t launch_kv4_quantize(const uint16_t* X, uint8_t* codes, uint16_t* params, int T, int C,
                               int G, hipStream_t stream) {
  const long long nlanes = (long long)T * C / 8;
  const unsigned blocks = (unsigned)((nlanes + 255) / 256);
  switch (G) {
    case 32:
      hipLaunchKernelGGL(kv4_quantize_kernel<4>, dim3(blocks), dim3(256), 0, stream, X, codes,
                         params, nlanes);
      break;
    case 64:
      hipLaunchKernelGGL(kv4_quantize_kernel<8>, dim3(blocks), dim3(256), 0, stream, X, codes,
                         params, nlanes);
      break;
    case 128:
      hipLaunchKernelGGL(kv4_quantize_kernel<16>, dim3(blocks), dim3(256), 0, stream, X, codes,
                         params, nlanes);
      break;
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_kv4_dequantize(const uint8_t* codes, const uint16_t* params, uint16_t* out,
                                 int T, int C, int G, hipStream_t stream) {
  const long long nlanes = (long long)T * C / 8;
  const unsigned blocks = (unsigned)((nlanes + 255) / 256);
  switch (G) {
    case 32:
      hipLaunchKernelGGL(kv4_dequantize_kernel<4>, dim3(blocks), dim3(256), 0, stream, codes,
                         params, out, nlanes);
      break;
    case 64:
      hipLaunchKernelGGL(kv4_dequantize_kernel<8>, dim3(blocks), dim3(256), 0, stream, codes,
                         params, out, nlanes);
      break;
    case 128:
      hipLaunchKernelGGL(kv4_dequantize_kernel<16>, dim3(blocks), dim3(256), 0, stream, codes,
                         params, out, nlanes);
      break;
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace comet
