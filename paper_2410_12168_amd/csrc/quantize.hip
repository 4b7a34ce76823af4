// quantize.hip -- fused block quantize + pack kernels for gfx950.
//
// FMPQ (paper Sec. 3.2): every token's activations are split into blocks of
// G = 128 channels; each block is quantized symmetrically to 4 or 8 bits with
// one fp16 scale.  The same block quantizer packs the 4-bit weights offline.
//
// Work decomposition: 16 lanes own one (row, block) pair, 8 channels per lane
// (one 128-bit load of fp16).  The 16-lane max reduction stays inside a DPP
// row.  Each lane then emits one packed dword (4-bit) or two (8-bit), so a
// wave writes 256 B (4-bit) or 512 B (8-bit) of contiguous packed output.
// The activation grid is 2-D (block, row group): no 64-bit index division.
// 2 bytes in per channel, 0.5 or 1 byte out.
//
// Division: see fmpq.h.
//
// Channel permutation (Sec. 3.2): with a permutation the lane reads its 8
// channels X[m][perm[c]]: one vector load where the permutation leaves the
// chunk in place, one load per channel elsewhere.  The indices are the same
// for every row: a lane reads them once for all its rows.  An index outside
// [0, K) (compared unsigned, so negative ones too) reads channel K-1: no read
// leaves the row.
#include <hip/hip_runtime.h>
#include <hip/hip_fp16.h>
#include <stdint.h>

#include <algorithm>

#include "fmpq.h"
#include "kernels.h"
#include "swiglu.h"

namespace comet {

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// 16 bytes of fp16 that are read exactly once: nontemporal, so they do not
// displace cached data.
__device__ inline void load8_nt(const uint16_t* p, float (&x)[8]) {
  const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
  const uint32_t w[4] = {v.x, v.y, v.z, v.w};
  #pragma unroll
  for (int i = 0; i < 4; ++i) {
    x[2 * i] = __half2float(__ushort_as_half((unsigned short)(w[i] & 0xFFFF)));
    x[2 * i + 1] = __half2float(__ushort_as_half((unsigned short)(w[i] >> 16)));
  }
}

// The permutation indices perm[c0 .. c0+8), and whether they leave the chunk
// in place (perm[c0 + i] = c0 + i, true of most chunks of a calibrated plan).
__device__ inline bool perm_chunk(const int32_t* perm, int c0, uint32_t (&idx)[8]) {
  const uint4 i0 = *reinterpret_cast<const uint4*>(perm + c0);
  const uint4 i1 = *reinterpret_cast<const uint4*>(perm + c0 + 4);
  idx[0] = i0.x; idx[1] = i0.y; idx[2] = i0.z; idx[3] = i0.w;
  idx[4] = i1.x; idx[5] = i1.y; idx[6] = i1.z; idx[7] = i1.w;
  bool same = true;
  #pragma unroll
  for (int i = 0; i < 8; ++i) same = same && idx[i] == (uint32_t)(c0 + i);
  return same;
}

// One channel at a time; an index outside [0, K) reads channel K-1.
__device__ inline void gather8(const uint16_t* row, const uint32_t (&idx)[8], int K,
                               float (&x)[8]) {
  const uint32_t last = (uint32_t)(K - 1);
  #pragma unroll
  for (int i = 0; i < 8; ++i) x[i] = __half2float(__ushort_as_half(row[min(idx[i], last)]));
}

// Activations.  A workgroup owns one block g and 16 * R consecutive rows;
// 16-lane group q takes rows r0 + q + 16 j, j < R, whose 16-byte loads are all
// issued before any arithmetic.  Without a permutation (R = 2) the workgroups
// run block-fastest, so the chip streams whole rows of X at a time, and the
// loads are nontemporal.  With one (R = 4) they run row-fastest: the rows share
// the block's permutation indices, read once per lane, and a chunk that the
// permutation moves is gathered channel by channel.
template <bool kPerm, int R>
__global__ __launch_bounds__(256) void quantize_act_kernel(const uint16_t* __restrict__ X,
                                                           const int32_t* __restrict__ perm,
                                                           uint8_t* __restrict__ A,
                                                           uint16_t* __restrict__ sa, int M,
                                                           int K, BlockMap map) {
  const int lane16 = threadIdx.x & 15;
  const int g = kPerm ? blockIdx.y : blockIdx.x;
  const int rows0 = (kPerm ? blockIdx.x : blockIdx.y) * 16 * R + (threadIdx.x >> 4);
  const int c0 = g * kG + 8 * lane16;
  const bool b8 = (map.bits[g >> 6] >> (g & 63)) & 1;
  float x[R][8];
  #pragma unroll
  for (int j = 0; j < R; ++j) {
    const int m = min(rows0 + 16 * j, M - 1);
    if (kPerm)
      load8(X + (size_t)m * K + c0, x[j]);
    else
      load8_nt(X + (size_t)m * K + c0, x[j]);
  }
  bool same = true;
  uint32_t idx[8];
  if (kPerm) same = perm_chunk(perm, c0, idx);
  const size_t base = (size_t)M * 64 * (size_t)(g + n8_before(map, g));
  #pragma unroll
  for (int j = 0; j < R; ++j) {
    const int m = rows0 + 16 * j;
    if (kPerm && !same) gather8(X + (size_t)min(m, M - 1) * K, idx, K, x[j]);
    float a = 0.0f;
    #pragma unroll
    for (int i = 0; i < 8; ++i) a = fmaxf(a, fabsf(x[j][i]));
    a = max16(a);
    Codes c;
    const uint16_t s16 = quantize8(x[j], a, b8 ? 127.0f : 7.0f, c);
    if (m >= M) continue;
    if (b8) {
      *reinterpret_cast<uint2*>(A + base + (size_t)m * 128 + 8 * lane16) = pack8(c);
    } else {
      *reinterpret_cast<uint32_t*>(A + base + (size_t)m * 64 + 4 * lane16) = pack4(c);
    }
    if (lane16 == 0) sa[(size_t)g * M + m] = s16;
  }
}

// Weights: pair p -> (row n = p / NG, block g = p % NG).  W_packed is stored
// in 16-row panels: row n's block g at ((n / 16 * NG + g) * 16 + n % 16) * 64,
// so every GEMM reads a panel's K-block as one contiguous kilobyte.
template <bool kPerm>
__global__ __launch_bounds__(256) void pack_w4_kernel(const uint16_t* __restrict__ W,
                                                      const int32_t* __restrict__ perm,
                                                      uint8_t* __restrict__ Wp,
                                                      uint16_t* __restrict__ sw, int N, int K,
                                                      long long npairs) {
  const int lane16 = threadIdx.x & 15;
  const long long p = (long long)blockIdx.x * 16 + (threadIdx.x >> 4);
  const bool valid = p < npairs;
  const long long pc = valid ? p : npairs - 1;
  const int NG = K / kG;
  const int n = (int)(pc / NG);
  const int g = (int)(pc % NG);
  float x[8];
  const int c0 = g * kG + 8 * lane16;
  load8(W + (size_t)n * K + c0, x);
  if (kPerm) {
    uint32_t idx[8];
    if (!perm_chunk(perm, c0, idx)) gather8(W + (size_t)n * K, idx, K, x);
  }
  float a = 0.0f;
  #pragma unroll
  for (int i = 0; i < 8; ++i) a = fmaxf(a, fabsf(x[i]));
  a = max16(a);
  Codes c;
  uint16_t s16 = quantize8(x, a, 7.0f, c);
  if (!valid) return;
  const size_t chunk = ((size_t)(n / 16) * NG + g) * 16 + (size_t)(n % 16);
  *reinterpret_cast<uint32_t*>(Wp + chunk * 64 + 4 * lane16) = pack4(c);
  if (lane16 == 0) sw[(size_t)g * N + n] = s16;
}

// Per-channel running maximum of |X| over rows (the sampling step of the
// calibration, Sec. 3.2).  A lane owns 8 channels (one 16-byte load per row),
// a wave 512 channels; the 4 waves of a workgroup take every 4th row of the
// workgroup's row range, combine through LDS, and one lane per channel merges
// into absmax with an unsigned atomic max (non-negative fp32 values order like
// their bit patterns).  Bit-exact for any split: max is order-free.
__global__ __launch_bounds__(256) void channel_absmax_kernel(const uint16_t* __restrict__ X,
                                                             float* __restrict__ absmax, int M,
                                                             int K, int rows_per_wg) {
  __shared__ float red[4][64][9];
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int c0 = (blockIdx.x * 64 + lane) * 8;
  const int r0 = blockIdx.y * rows_per_wg;
  const int r1 = min(M, r0 + rows_per_wg);
  float a[8];
  #pragma unroll
  for (int i = 0; i < 8; ++i) a[i] = 0.0f;
  if (c0 < K) {
    for (int r = r0 + wave; r < r1; r += 4) {
      float x[8];
      load8(X + (size_t)r * K + c0, x);
      #pragma unroll
      for (int i = 0; i < 8; ++i) a[i] = fmaxf(a[i], fabsf(x[i]));
    }
  }
  #pragma unroll
  for (int i = 0; i < 8; ++i) red[wave][lane][i] = a[i];
  __syncthreads();
  // thread t merges channel c0(t / 8 lane) + t % 8 over the four waves
  const int l = threadIdx.x >> 3, i = threadIdx.x & 7;
  for (int h = 0; h < 2; ++h) {
    const int ll = l + 32 * h;
    const int c = (blockIdx.x * 64 + ll) * 8 + i;
    if (c < K) {
      float v = fmaxf(fmaxf(red[0][ll][i], red[1][ll][i]), fmaxf(red[2][ll][i], red[3][ll][i]));
      atomicMax(reinterpret_cast<unsigned int*>(absmax + c), __float_as_uint(v));
    }
  }
}

// SwiGLU + next-layer quantization of an fp16 gate/up output: workgroup
// (x, y) = (block j, 32 rows from 32 y); 16 lanes own one (row, block) pair
// and read 8 gate and 8 up values (two 16-byte loads), form h and quantize it
// as the activation quantizer does.
__global__ __launch_bounds__(256) void swiglu_quantize_kernel(const uint16_t* __restrict__ GU,
                                                              uint8_t* __restrict__ A,
                                                              uint16_t* __restrict__ sa, int M,
                                                              int I, BlockMap map) {
  const int lane16 = threadIdx.x & 15;
  const int j = blockIdx.x;
  const bool b8 = (map.bits[j >> 6] >> (j & 63)) & 1;
  const size_t base = (size_t)M * 64 * (size_t)(j + n8_before(map, j));
  #pragma unroll
  for (int t = 0; t < 2; ++t) {
    const int m = blockIdx.y * 32 + 16 * t + (threadIdx.x >> 4);
    const uint16_t* row = GU + (size_t)min(m, M - 1) * 2 * I + (size_t)j * 2 * kG + 8 * lane16;
    const uint4 gv = *reinterpret_cast<const uint4*>(row);
    const uint4 uv = *reinterpret_cast<const uint4*>(row + kG);
    const uint32_t gw[4] = {gv.x, gv.y, gv.z, gv.w}, uw[4] = {uv.x, uv.y, uv.z, uv.w};
    float x[8];
    #pragma unroll
    for (int i = 0; i < 8; ++i) {
      const uint16_t g = (uint16_t)(gw[i >> 1] >> (16 * (i & 1)));
      const uint16_t u = (uint16_t)(uw[i >> 1] >> (16 * (i & 1)));
      x[i] = __half2float(__ushort_as_half(swiglu_f16(g, u)));
    }
    float a = 0.0f;
    #pragma unroll
    for (int i = 0; i < 8; ++i) a = fmaxf(a, fabsf(x[i]));
    a = max16(a);
    Codes c;
    const uint16_t s16 = quantize8(x, a, b8 ? 127.0f : 7.0f, c);
    if (m >= M) continue;
    if (b8)
      *reinterpret_cast<uint2*>(A + base + (size_t)m * 128 + 8 * lane16) = pack8(c);
    else
      *reinterpret_cast<uint32_t*>(A + base + (size_t)m * 64 + 4 * lane16) = pack4(c);
    if (lane16 == 0) sa[(size_t)j * M + m] = s16;
  }
}

}  // namespace

hipError_t launch_swiglu_quantize(const uint16_t* GU, uint8_t* A, uint16_t* sa, int M, int I,
                                  const BlockMap& map, hipStream_t stream) {
  hipLaunchKernelGGL(swiglu_quantize_kernel, dim3((unsigned)(I / kG), (unsigned)((M + 31) / 32)),
                     dim3(256), 0, stream, GU, A, sa, M, I, map);
  return hipGetLastError();
}

hipError_t launch_quantize_act(const uint16_t* X, const int32_t* perm, uint8_t* A, uint16_t* sa,
                               int M, int K, const BlockMap& map, hipStream_t stream) {
  const unsigned NG = (unsigned)(K / kG);
  if (perm)
    hipLaunchKernelGGL((quantize_act_kernel<true, 4>), dim3((unsigned)((M + 63) / 64), NG),
                       dim3(256), 0, stream, X, perm, A, sa, M, K, map);
  else
    hipLaunchKernelGGL((quantize_act_kernel<false, 2>), dim3(NG, (unsigned)((M + 31) / 32)),
                       dim3(256), 0, stream, X, perm, A, sa, M, K, map);
  return hipGetLastError();
}

hipError_t launch_pack_w4(const uint16_t* W, const int32_t* perm, uint8_t* Wp, uint16_t* sw,
                          int N, int K, hipStream_t stream) {
  long long npairs = (long long)N * (K / kG);
  long long blocks = (npairs + 15) / 16;
  if (perm)
    hipLaunchKernelGGL(pack_w4_kernel<true>, dim3((unsigned)blocks), dim3(256), 0, stream, W,
                       perm, Wp, sw, N, K, npairs);
  else
    hipLaunchKernelGGL(pack_w4_kernel<false>, dim3((unsigned)blocks), dim3(256), 0, stream, W,
                       perm, Wp, sw, N, K, npairs);
  return hipGetLastError();
}

hipError_t launch_channel_absmax(const uint16_t* X, float* absmax, int M, int K,
                                 hipStream_t stream) {
  const int gx = (K + 511) / 512;
  // enough row slices to fill the chip, at least 16 rows per workgroup
  int gy = std::max(1, std::min((M + 15) / 16, std::max(1, 2048 / gx)));
  const int rows = (M + gy - 1) / gy;
  gy = (M + rows - 1) / rows;
  hipLaunchKernelGGL(channel_absmax_kernel, dim3(gx, gy), dim3(256), 0, stream, X, absmax, M, K,
                     rows);
  return hipGetLastError();
}

}  // namespace comet
