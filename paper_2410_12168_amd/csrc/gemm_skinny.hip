// gemm_skinny.hip -- W4Ax GEMM for few tokens (decode, M <= 64) on gfx950.
//
// With a handful of tokens the GEMM is a weight stream: every 4-bit weight is
// read from HBM once and used by at most 64 activation rows, so the bound is
// HBM bandwidth, not the matrix cores.  Each wave owns 16 output columns and
// a contiguous range of the K-block schedule (split-K slot), loads its weight
// fragments straight from HBM into registers (no LDS, no sharing), four
// K-blocks per batch with the next batch in flight while the current one
// computes, and reads the tiny activation operand through L2.  The operand
// path is the prefill kernel's: FP8-E4M3 subnormal codes, one
// v_mfma_f32_16x16x128_f8f6f4 per 16x16 block and K-block (two for 8-bit
// activation blocks), exact scale products from v_mfma_f32_4x4x1_16b_f32,
// fp32 FMA dequantization.  Split-K slots of one column block live in one
// workgroup and are added in slot order through LDS.
#include <hip/hip_runtime.h>
#include <hip/hip_fp16.h>
#include <stdint.h>

#include "kernels.h"
#include "operand.h"

namespace comet {

namespace {

constexpr int kD = 2;      // K-blocks per load batch (more waves fit than with deeper batches)
constexpr int kWaves = 4;  // waves per workgroup; the split-K slot count divides it

template <int R, bool B8>
struct Batch {
  u32x4 w[kD];
  u32x4 a[kD][R][B8 ? 2 : 1];
  uint32_t sa[kD][R];  // raw fp16 bits, converted when used (no wait at load time)
  uint32_t sw[kD];
};

// K-block order entry at schedule position `pos` (wave-uniform).  The order
// array is written once when the plan is built and only read by kernels, so
// it is read through the constant address space: scalar loads that the
// issue_point() barriers below do not force back to vector loads (a vector
// load here would queue behind the weight loads and wait for them).
typedef const int __attribute__((address_space(4)))* ConstIntPtr;
__device__ __forceinline__ int order_entry(const GemmArgs& p, int pos) {
  return ((ConstIntPtr)p.order)[pos];
}

// Loads schedule positions [pos, pos + kD), unconditionally.  Positions past
// the end of the wave's range read whatever valid block the order holds there
// (the order array is padded by kOrderPad >= 2 * kD - 1 entries) and are
// masked in compute_batch.  Unconditional loads keep every wait a partial
// one: a load under a branch makes the compiler's wait-count merge fall back
// to waiting for all loads, which serialises the double buffering.
template <int R, bool B8>
__device__ __forceinline__ void load_batch(const GemmArgs& p, int pos, int col, Batch<R, B8>& b) {
  static_assert(kOrderPad >= 2 * kD - 1, "order padding too short for the prefetch depth");
  const int lane = threadIdx.x & 63;
  const int r16 = lane & 15, q4 = lane >> 4;
  #pragma unroll
  for (int d = 0; d < kD; ++d) {
    const int e = order_entry(p, pos + d);
    const int g = e & 1023, aoff = e >> 11;
    b.w[d] = *reinterpret_cast<const u32x4*>(p.W + (size_t)col * (p.K / 2) + (size_t)g * 64 + q4 * 16);
    const uint8_t* A = p.A + (size_t)p.M * 64 * (size_t)aoff;
    #pragma unroll
    for (int r = 0; r < R; ++r) {
      const int row = min(16 * r + r16, p.M - 1);
      if constexpr (B8) {
        b.a[d][r][0] = *reinterpret_cast<const u32x4*>(A + (size_t)row * 128 + q4 * 32);
        b.a[d][r][1] = *reinterpret_cast<const u32x4*>(A + (size_t)row * 128 + q4 * 32 + 16);
      } else {
        b.a[d][r][0] = *reinterpret_cast<const u32x4*>(A + (size_t)row * 64 + q4 * 16);
      }
      // 4x4x1 operand: activation scale of row 16r + 4*q4 + (lane & 3)
      const int srow = min(16 * r + 4 * q4 + (lane & 3), p.M - 1);
      b.sa[d][r] = p.sa[(size_t)g * p.M + srow];
    }
    b.sw[d] = p.sw[(size_t)g * p.N + col];
  }
}

template <int R, bool B8, bool DIAG>
__device__ __forceinline__ void compute_batch(const GemmArgs& p, int pos, int end, int n0,
                                              const Batch<R, B8>& b, f32x4 (&C)[R]) {
  const int lane = threadIdx.x & 63;
  const int r16 = lane & 15, q4 = lane >> 4;
  const int NG = p.K / kG;
  #pragma unroll
  for (int d = 0; d < kD; ++d) {
    const bool valid = pos + d < end;  // a block past the range contributes zero
    {
      u32x4 lo, hi;
      unpack4(b.w[d], lo, hi);
      const i32x8 wf = {(int)lo[0], (int)lo[1], (int)lo[2], (int)lo[3],
                        (int)hi[0], (int)hi[1], (int)hi[2], (int)hi[3]};
      #pragma unroll
      for (int r = 0; r < R; ++r) {
        f32x4 y;
        if constexpr (B8) {
          i32x8 al, ah;
          #pragma unroll
          for (int i = 0; i < 4; ++i) {
            al[i] = (int)lo8(b.a[d][r][0][i]);
            al[4 + i] = (int)lo8(b.a[d][r][1][i]);
            ah[i] = (int)hi8(b.a[d][r][0][i]);
            ah[4 + i] = (int)hi8(b.a[d][r][1][i]);
          }
          const f32x4 yh = mfma_fp8(ah, wf, f32x4{0.f, 0.f, 0.f, 0.f});
          y = mfma_fp8(al, wf, yh * 8.0f);  // exact: integers below 2^24 units
        } else {
          u32x4 alo, ahi;
          unpack4(b.a[d][r][0], alo, ahi);
          const i32x8 af = {(int)alo[0], (int)alo[1], (int)alo[2], (int)alo[3],
                            (int)ahi[0], (int)ahi[1], (int)ahi[2], (int)ahi[3]};
          y = mfma_fp8(af, wf, f32x4{0.f, 0.f, 0.f, 0.f});
        }
        if constexpr (DIAG) {
          if (!valid) continue;
          const int g = order_entry(p, pos + d) & 1023;
          const int col = n0 + r16;
          #pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int row = 16 * r + 4 * q4 + i;
            if (row >= p.win_m0 && row < p.win_m1 && col >= p.win_n0 && col < p.win_n1) {
              const size_t idx = ((size_t)(row - p.win_m0) * (p.win_n1 - p.win_n0) +
                                  (col - p.win_n0)) * NG + g;
              p.acc[idx] = (int32_t)(y[i] * kUnit);
            }
          }
        } else {
          const float sa = __half2float(__ushort_as_half((unsigned short)b.sa[d][r])) * kUnit;
          const float sw = valid ? __half2float(__ushort_as_half((unsigned short)b.sw[d])) : 0.0f;
          const f32x4 P = scale_products(sa, sw);
          #pragma unroll
          for (int i = 0; i < 4; ++i) C[r][i] = __builtin_fmaf(y[i], P[i], C[r][i]);
        }
      }
    }
  }
}

// Compiler barrier: loads issued before it stay before it, and no
// instruction of the following compute is scheduled above it.  Without it the
// compiler sinks each batch's loads down to their first use, which turns the
// double buffering back into load-then-wait.  It orders only the issue; no
// wait for the loaded values is implied.
__device__ __forceinline__ void issue_point() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_sched_barrier(0);
}

// Schedule positions [pos, end), all of precision B8, in double-buffered
// batches: the loads of one batch are in flight while the other computes.
// Loads run at most 2 * kD - 1 positions past `end`.
template <int R, bool B8, bool DIAG>
__device__ __forceinline__ void stream(const GemmArgs& p, int pos, int end, int col, int n0,
                                       f32x4 (&C)[R]) {
  if (pos >= end) return;
  Batch<R, B8> x, y;
  load_batch<R, B8>(p, pos, col, x);
  for (;;) {
    load_batch<R, B8>(p, pos + kD, col, y);
    issue_point();
    compute_batch<R, B8, DIAG>(p, pos, end, n0, x, C);
    if (pos + kD >= end) break;
    load_batch<R, B8>(p, pos + 2 * kD, col, x);
    issue_point();
    compute_batch<R, B8, DIAG>(p, pos + kD, end, n0, y, C);
    pos += 2 * kD;
    if (pos >= end) break;
  }
}

// One wave = one (16-column block, split-K slot) unit; a workgroup of
// kWaves waves holds kWaves / S column blocks with all S slots of each, so
// the split-K partial sums are added inside the workgroup, through LDS, in
// slot order.  (A cross-workgroup reduction would need device-scope fences,
// and on this multi-XCD part each one writes back and invalidates the XCD's
// L2: measured ~12x slower for a 70B-sized weight stream.)
template <int R, bool DIAG>
__global__ __launch_bounds__(kWaves * 64) void skinny_kernel(GemmArgs p) {
  __shared__ f32x4 red[kWaves][R][64];
  const int lane = threadIdx.x & 63;
  const int r16 = lane & 15, q4 = lane >> 4;
  const int S = p.splits;
  // wave-uniform indices (readfirstlane keeps the schedule walk in scalar
  // registers)
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int cb = blockIdx.x * (kWaves / S) + wave / S, slot = wave % S;
  const bool active = cb < p.N / 16;  // the last workgroup may be partly idle
  const int n0 = cb * 16;
  const int col = n0 + r16;
  const int NG = p.K / kG;
  // this slot's share of the schedule positions
  const int g0 = NG * slot / S, g1 = NG * (slot + 1) / S;
  const int split = min(max(p.n4, g0), g1);

  f32x4 C[R];
  #pragma unroll
  for (int r = 0; r < R; ++r) C[r] = f32x4{0.f, 0.f, 0.f, 0.f};
  if (active) {
    stream<R, false, DIAG>(p, g0, split, col, n0, C);
    stream<R, true, DIAG>(p, split, g1, col, n0, C);
  }
  if constexpr (DIAG) return;

  if (S > 1) {
    #pragma unroll
    for (int r = 0; r < R; ++r) red[wave][r][lane] = C[r];
    __syncthreads();
    if (slot != 0) return;
    #pragma unroll
    for (int r = 0; r < R; ++r) {
      C[r] = red[wave][r][lane];
      for (int s = 1; s < S; ++s) C[r] += red[wave + s][r][lane];
    }
  }
  if (!active) return;
  #pragma unroll
  for (int r = 0; r < R; ++r)
    #pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row = 16 * r + 4 * q4 + i;
      if (row < p.M) p.out[(size_t)row * p.N + col] = __half_as_ushort(__float2half_rn(C[r][i]));
    }
}

template <int R>
hipError_t launch_r(const GemmArgs& a, bool diag, hipStream_t stream) {
  const int per_wg = kWaves / a.splits;
  const int blocks = (a.N / 16 + per_wg - 1) / per_wg;
  if (diag)
    hipLaunchKernelGGL((skinny_kernel<R, true>), dim3(blocks), dim3(kWaves * 64), 0, stream, a);
  else
    hipLaunchKernelGGL((skinny_kernel<R, false>), dim3(blocks), dim3(kWaves * 64), 0, stream, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_gemm_skinny(const GemmArgs& a, bool diag, hipStream_t stream) {
  if (a.splits < 1 || kWaves % a.splits != 0) return hipErrorInvalidValue;
  switch ((a.M + 15) / 16) {
    case 1: return launch_r<1>(a, diag, stream);
    case 2: return launch_r<2>(a, diag, stream);
    case 3: return launch_r<3>(a, diag, stream);
    case 4: return launch_r<4>(a, diag, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace comet
