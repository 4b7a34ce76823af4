// gemm_skinny.hip -- W4Ax GEMM for few tokens (decode, M <= 48) on gfx950.
//
// With a handful of tokens the GEMM is a weight stream: every 4-bit weight is
// read from HBM once and used by at most 48 activation rows, so the bound is
// HBM bandwidth, not the matrix cores.  Each wave owns 16 output columns and
// a contiguous K-block range (split-K slot), walked in natural block order in
// batches of four K-blocks.  The wave's 16 weight rows are one panel of
// W_packed, where each K-block is one contiguous kilobyte: one nontemporal
// 128-bit load per lane and K-block reads it whole, and lane r + 16 q lands
// exactly on its MFMA fragment (row r, codes 32 q .. 32 q + 31), so the
// weights go from HBM to the matrix core with no LDS round trip.  The next
// batch is in flight while the current one computes.  The tiny activation
// operand and the scales are read through L2, one K-block ahead.  For
// 8 < M <= 32 a second kernel shares the activation operand among the
// workgroup's waves through LDS (below).
//
// The operand path is the prefill kernel's: FP8-E4M3 subnormal codes, one
// v_mfma_f32_16x16x128_f8f6f4 per 16x16 block and K-block (two for 8-bit
// activation blocks), exact scale products from v_mfma_f32_4x4x1_16b_f32,
// fp32 FMA dequantization.  Split-K slots of one column block live in one
// workgroup and are added in slot order through LDS.
#include <hip/hip_runtime.h>
#include <hip/hip_fp16.h>
#include <stdint.h>

#include <type_traits>

#include "kernels.h"
#include "operand.h"

namespace comet {

namespace {

constexpr int kD = 4;      // K-blocks per weight batch (256 bytes of each weight row)
constexpr int kWaves = 4;  // waves per workgroup; the split-K slot count divides it

// One K-block's activation fragments and scales, loaded one step ahead.  Both
// 16-byte halves are always loaded (for a 4-bit block the second repeats the
// first), so every step issues the same loads and the compiler's waits stay
// partial.  With at most 8 rows one load per lane suffices (load_a's HALF
// form, which leaves a[r][1] unused).
template <int R>
struct AStep {
  u32x4 a[R][2];
};

// Scales of one batch, one load per row block (activations) and one for the
// weights: lane l holds the activation scale of row 16 r + l % 16 and the
// weight scale of column n0 + l % 16, both of K-block gb + l / 16.  A step
// takes its values from the lanes of its K-block (cross-lane reads).
template <int R>
struct SBatch {
  uint32_t sa[R];
  uint32_t sw;
};

// Precision bit of K-block g.
__device__ __forceinline__ bool is8(const GemmArgs& p, int g) {
  return (p.map.bits[g >> 6] >> (g & 63)) & 1;
}

// Offset of K-block g in A_packed, in units of M * 64 bytes: g plus the
// 8-bit blocks before it.
__device__ __forceinline__ int aoff_of(const GemmArgs& p, int g) {
  int n = 0;
  for (int w = 0; w < (g >> 6); ++w) n += __popcll(p.map.bits[w]);
  if (g & 63) n += __popcll(p.map.bits[g >> 6] & ((1ull << (g & 63)) - 1));
  return g + n;
}

// Activation fragments (rows 16 r + lane % 16, 32 codes of quarter lane / 16)
// and scales of K-block g, whose block starts at aoff * M * 64 bytes.
template <int R, bool HALF = false>
__device__ __forceinline__ void load_a(const GemmArgs& p, int g, int aoff, int col, AStep<R>& s) {
  const int lane = threadIdx.x & 63;
  const int r16 = lane & 15, q4 = lane >> 4;
  const uint32_t b8 = is8(p, g) ? 1u : 0u;
  const uint8_t* A = p.A + (size_t)p.M * 64 * (size_t)aoff;
  if constexpr (HALF) {
    // M <= 8: rows 8..15 of the fragment are padding.  Lane r of each
    // 16-lane row loads row r & 7: its (first) 16 bytes for r < 8, and for an
    // 8-bit block the second 16 bytes of the same 32-byte chunk for r >= 8.
    // compute_step moves the second halves down by eight lanes.
    const uint32_t row = (uint32_t)min(r16 & 7, p.M - 1);
    const uint32_t second = ((uint32_t)r16 >> 3) & b8;
    s.a[0][0] = *reinterpret_cast<const u32x4*>(A + (row << (6 + b8)) + ((uint32_t)q4 << (4 + b8)) +
                                               (second << 4));
    (void)col;
    return;
  }
  #pragma unroll
  for (int r = 0; r < R; ++r) {
    const uint32_t row = (uint32_t)min(16 * r + r16, p.M - 1);
    const uint8_t* base = A + (row << (6 + b8)) + ((uint32_t)q4 << (4 + b8));
    s.a[r][0] = *reinterpret_cast<const u32x4*>(base);
    s.a[r][1] = *reinterpret_cast<const u32x4*>(base + (b8 << 4));
  }
  (void)col;
}

template <int R>
__device__ __forceinline__ void load_scales(const GemmArgs& p, int gb, int n0, SBatch<R>& s) {
  const int lane = threadIdx.x & 63;
  const int g = min(gb + (lane >> 4), p.K / kG - 1);
  #pragma unroll
  for (int r = 0; r < R; ++r)
    s.sa[r] = p.sa[(size_t)g * p.M + min(16 * r + (lane & 15), p.M - 1)];
  s.sw = p.sw[(size_t)g * p.N + n0 + (lane & 15)];
}

// Weight fragments of the batch starting at K-block gb for the wave's panel
// (rows n0 .. n0 + 15): load i is K-block gb + i, lane r + 16 q reading row
// r's 16-byte chunk q.  K-blocks past glast (the slot's last block) repeat it:
// they are never computed, and the repeat is a cache hit, where reading on
// into the next slot's blocks would fetch them from HBM a second time.
__device__ __forceinline__ void load_w(const GemmArgs& p, int gb, int glast, int n0,
                                       u32x4 (&w)[4]) {
  const int lane = threadIdx.x & 63;
  const int NG = p.K / kG;
  const uint8_t* panel = p.W + (size_t)(n0 / 16) * NG * 1024 + (lane & 15) * 64 + (lane >> 4) * 16;
  #pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int g = min(gb + i, glast);
    w[i] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(panel + (size_t)g * 1024));
  }
}

template <int R, bool DIAG, bool HALF = false>
__device__ __forceinline__ void compute_step(const GemmArgs& p, const u32x4& wraw, int i, int g,
                                             bool b8, int n0, const AStep<R>& s,
                                             const SBatch<R>& sc, f32x4 (&C)[R]) {
  const int lane = threadIdx.x & 63;
  const int r16 = lane & 15, q4 = lane >> 4;
  const int NG = p.K / kG;
  u32x4 wlo, whi;
  unpack4(wraw, wlo, whi);
  const i32x8 wf = {(int)wlo[0], (int)wlo[1], (int)wlo[2], (int)wlo[3],
                    (int)whi[0], (int)whi[1], (int)whi[2], (int)whi[3]};
  #pragma unroll
  for (int r = 0; r < R; ++r) {
    f32x4 y;
    if (b8) {
      i32x8 al, ah;
      u32x4 x1 = s.a[r][1];
      if constexpr (HALF) {
        // second 16 bytes from the lane eight above, in the same 16-lane row
        #pragma unroll
        for (int k = 0; k < 4; ++k)
          x1[k] = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)s.a[r][0][k], 0x128, 0xF, 0xF, false);
      }
      #pragma unroll
      for (int k = 0; k < 4; ++k) {
        al[k] = (int)lo8(s.a[r][0][k]);
        al[4 + k] = (int)lo8(x1[k]);
        ah[k] = (int)hi8(s.a[r][0][k]);
        ah[4 + k] = (int)hi8(x1[k]);
      }
      const f32x4 yh = mfma_fp8(ah, wf, f32x4{0.f, 0.f, 0.f, 0.f});
      y = mfma_fp8(al, wf, yh * 8.0f);  // exact: integers below 2^24 units
    } else {
      u32x4 alo, ahi;
      unpack4(s.a[r][0], alo, ahi);
      const i32x8 af = {(int)alo[0], (int)alo[1], (int)alo[2], (int)alo[3],
                        (int)ahi[0], (int)ahi[1], (int)ahi[2], (int)ahi[3]};
      y = mfma_fp8(af, wf, f32x4{0.f, 0.f, 0.f, 0.f});
    }
    if constexpr (DIAG) {
      const int col = n0 + r16;
      #pragma unroll
      for (int k = 0; k < 4; ++k) {
        const int row = 16 * r + 4 * q4 + k;
        if (row >= p.win_m0 && row < p.win_m1 && col >= p.win_n0 && col < p.win_n1) {
          const size_t idx = ((size_t)(row - p.win_m0) * (p.win_n1 - p.win_n0) +
                              (col - p.win_n0)) * NG + g;
          p.acc[idx] = (int32_t)(y[k] * kUnit);
        }
      }
    } else {
      // 4x4x1 operands: activation scale of row 16 r + 4 q4 + (lane & 3),
      // weight scale of column n0 + lane % 16
      const uint32_t sab = (uint32_t)__shfl((int)sc.sa[r], 16 * i + 4 * q4 + (lane & 3));
      const uint32_t swb = (uint32_t)__shfl((int)sc.sw, 16 * i + r16);
      const float sa = __half2float(__ushort_as_half((unsigned short)sab)) * kUnit;
      const float sw = __half2float(__ushort_as_half((unsigned short)swb));
      const f32x4 P = scale_products(sa, sw);
      #pragma unroll
      for (int k = 0; k < 4; ++k) C[r][k] = __builtin_fmaf(y[k], P[k], C[r][k]);
    }
  }
}

// Compiler barrier: loads issued before it stay before it, and no
// instruction of the following compute is scheduled above it.  Without it the
// compiler sinks loads down to their first use, which turns the prefetching
// back into load-then-wait.  It orders only the issue; no wait for the loaded
// values is implied.
__device__ __forceinline__ void issue_point() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_sched_barrier(0);
}

// One batch: K-blocks gb .. gb + 3 (those below g1 are computed) from weights
// `wc`, while the next batch's weights load into `wn`.  The activation step
// of K-block gb is in `x` on entry; `x` and `y` alternate, and the step of
// K-block gb + 4 is in `x` on exit.
template <int R, bool DIAG, bool HALF>
__device__ __forceinline__ void batch(const GemmArgs& p, int gb, int g1, int n0, int col,
                                      int& aoff, const u32x4 (&wc)[4], u32x4 (&wn)[4],
                                      const SBatch<R>& sc, SBatch<R>& sn, AStep<R>& x,
                                      AStep<R>& y, f32x4 (&C)[R]) {
  const int NG = p.K / kG;
  load_w(p, gb + kD, g1 - 1, n0, wn);
  load_scales<R>(p, gb + kD, n0, sn);
  #pragma unroll
  for (int i = 0; i < kD; ++i) {
    const int g = gb + i;
    const bool b8 = is8(p, min(g, NG - 1));
    // next step's activations: K-block g + 1 (clamped into range)
    const int gn = min(g + 1, NG - 1);
    const int an = g + 1 < NG ? aoff + 1 + (b8 ? 1 : 0) : aoff;
    AStep<R>& cur = (i & 1) ? y : x;
    AStep<R>& nxt = (i & 1) ? x : y;
    load_a<R, HALF>(p, gn, an, col, nxt);
    issue_point();
    if (g < g1) compute_step<R, DIAG, HALF>(p, wc[i], i, g, b8, n0, cur, sc, C);
    aoff = an;
  }
}

// One wave = one (16-column block, split-K slot) unit; a workgroup of
// kWaves waves holds kWaves / S column blocks with all S slots of each, so
// the split-K partial sums are added inside the workgroup, through LDS, in
// slot order.  (A cross-workgroup reduction would need device-scope fences,
// and on this multi-XCD part each one writes back and invalidates the XCD's
// L2: measured ~12x slower for a 70B-sized weight stream.)
template <int R, bool DIAG, bool HALF>
__global__ __launch_bounds__(kWaves * 64) void skinny_kernel(GemmArgs p) {
  __shared__ f32x4 red[kWaves][R][64];
  const int lane = threadIdx.x & 63;
  const int r16 = lane & 15, q4 = lane >> 4;
  const int S = p.splits;
  // wave-uniform indices (readfirstlane keeps the walk in scalar registers)
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int cb = blockIdx.x * (kWaves / S) + wave / S, slot = wave % S;
  const bool active = cb < p.N / 16;  // the last workgroup may be partly idle
  const int n0 = active ? cb * 16 : 0;
  const int col = n0 + r16;
  const int NG = p.K / kG;
  // this slot's K-blocks, in natural order
  const int g0 = NG * slot / S, g1 = NG * (slot + 1) / S;

  f32x4 C[R];
  #pragma unroll
  for (int r = 0; r < R; ++r) C[r] = f32x4{0.f, 0.f, 0.f, 0.f};
  if (active && g0 < g1) {
    u32x4 wa[4], wb[4];
    SBatch<R> sa_, sb_;
    AStep<R> x, y;
    int aoff = aoff_of(p, g0);
    load_w(p, g0, g1 - 1, n0, wa);
    load_scales<R>(p, g0, n0, sa_);
    load_a<R, HALF>(p, g0, aoff, col, x);
    for (int gb = g0;;) {
      batch<R, DIAG, HALF>(p, gb, g1, n0, col, aoff, wa, wb, sa_, sb_, x, y, C);
      gb += kD;
      if (gb >= g1) break;
      batch<R, DIAG, HALF>(p, gb, g1, n0, col, aoff, wb, wa, sb_, sa_, x, y, C);
      gb += kD;
      if (gb >= g1) break;
    }
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
  const bool half = R == 1 && a.M <= 8;
  if (diag) {
    if (half)
      hipLaunchKernelGGL((skinny_kernel<1, true, true>), dim3(blocks), dim3(kWaves * 64), 0, stream, a);
    else
      hipLaunchKernelGGL((skinny_kernel<R, true, false>), dim3(blocks), dim3(kWaves * 64), 0, stream, a);
  } else {
    if (half)
      hipLaunchKernelGGL((skinny_kernel<1, false, true>), dim3(blocks), dim3(kWaves * 64), 0, stream, a);
    else
      hipLaunchKernelGGL((skinny_kernel<R, false, false>), dim3(blocks), dim3(kWaves * 64), 0, stream, a);
  }
  return hipGetLastError();
}


// ---------------------------------------------------------------------------
// Few-token kernel with the activation operand shared through LDS (8 < M <=
// 32, at most two split-K slots).  A workgroup holds four column blocks and all S
// slots of each (4 S waves).  The per-wave kernel above reads the whole
// activation operand of every K-block in every wave, which costs the memory
// pipeline more than the weight stream once M reaches 8.  Here the four waves
// of a slot load one batch of four K-blocks together, one K-block each,
// unpack 4-bit codes once, and leave every MFMA fragment in a double-buffered
// LDS area at [batch buffer][slot][K-block][row block][lane] (32 bytes each);
// one barrier per batch publishes it.  Weights, scales and dequantization are
// those of the per-wave kernel.
constexpr int kCBW = 4;  // column blocks per workgroup

template <int R, int S>
struct SharedA {
  static constexpr int Bytes = 2 * S * kD * R * 2048;
};

// This wave's share of batch gb's activation fragments: K-block gb + (wave %
// 4), every row block, all 64 lanes' 32-byte fragments.  Both 16-byte halves
// are always loaded (for a 4-bit block the second repeats the first), so the
// loads are the same every batch.
template <int R>
struct AChunk {
  u32x4 v[R][2];
  bool b8;
};
template <int R>
__device__ __forceinline__ void chunk_load(const GemmArgs& p, int g, AChunk<R>& c) {
  const int lane = threadIdx.x & 63;
  const int r16 = lane & 15, q4 = lane >> 4;
  c.b8 = is8(p, g);
  const uint32_t b8 = c.b8 ? 1u : 0u;
  const uint8_t* A = p.A + (size_t)p.M * 64 * (size_t)aoff_of(p, g);
  #pragma unroll
  for (int r = 0; r < R; ++r) {
    const uint32_t row = (uint32_t)min(16 * r + r16, p.M - 1);
    const uint8_t* base = A + (row << (6 + b8)) + ((uint32_t)q4 << (4 + b8));
    c.v[r][0] = *reinterpret_cast<const u32x4*>(base);
    c.v[r][1] = *reinterpret_cast<const u32x4*>(base + (b8 << 4));
  }
}
// FP8 bytes of a 4-bit block (unpacked here, once per workgroup), raw codes of
// an 8-bit block (split into hi and lo at use).
template <int R>
__device__ __forceinline__ void chunk_store(const AChunk<R>& c, uint8_t* dst) {
  const int lane = threadIdx.x & 63;
  #pragma unroll
  for (int r = 0; r < R; ++r) {
    u32x4 lo = c.v[r][0], hi = c.v[r][1];
    if (!c.b8) unpack4(c.v[r][0], lo, hi);
    *reinterpret_cast<u32x4*>(dst + r * 2048 + lane * 32) = lo;
    *reinterpret_cast<u32x4*>(dst + r * 2048 + lane * 32 + 16) = hi;
  }
}

// `live` is false for steps past the slot's last K-block: they run anyway
// (their operands are valid clamped data) and add y * 0 = 0, which keeps the
// loop free of branches that would make the compiler's load waits
// conservative.
template <int R, bool DIAG>
__device__ __forceinline__ void compute_shared(const GemmArgs& p, const u32x4& wraw, int i, int g,
                                               bool b8, bool live, int n0, const uint8_t* frag,
                                               const SBatch<R>& sc, f32x4 (&C)[R]) {
  const int lane = threadIdx.x & 63;
  const int r16 = lane & 15, q4 = lane >> 4;
  const int NG = p.K / kG;
  u32x4 wlo, whi;
  unpack4(wraw, wlo, whi);
  const i32x8 wf = {(int)wlo[0], (int)wlo[1], (int)wlo[2], (int)wlo[3],
                    (int)whi[0], (int)whi[1], (int)whi[2], (int)whi[3]};
  #pragma unroll
  for (int r = 0; r < R; ++r) {
    const u32x4 x0 = *reinterpret_cast<const u32x4*>(frag + r * 2048 + lane * 32);
    const u32x4 x1 = *reinterpret_cast<const u32x4*>(frag + r * 2048 + lane * 32 + 16);
    f32x4 y;
    if (b8) {
      i32x8 al, ah;
      #pragma unroll
      for (int k = 0; k < 4; ++k) {
        al[k] = (int)lo8(x0[k]);
        al[4 + k] = (int)lo8(x1[k]);
        ah[k] = (int)hi8(x0[k]);
        ah[4 + k] = (int)hi8(x1[k]);
      }
      const f32x4 yh = mfma_fp8(ah, wf, f32x4{0.f, 0.f, 0.f, 0.f});
      y = mfma_fp8(al, wf, yh * 8.0f);  // exact: integers below 2^24 units
    } else {
      const i32x8 af = {(int)x0[0], (int)x0[1], (int)x0[2], (int)x0[3],
                        (int)x1[0], (int)x1[1], (int)x1[2], (int)x1[3]};
      y = mfma_fp8(af, wf, f32x4{0.f, 0.f, 0.f, 0.f});
    }
    if constexpr (DIAG) {
      const int col = n0 + r16;
      #pragma unroll
      for (int k = 0; k < 4; ++k) {
        const int row = 16 * r + 4 * q4 + k;
        if (live && row >= p.win_m0 && row < p.win_m1 && col >= p.win_n0 && col < p.win_n1) {
          const size_t idx = ((size_t)(row - p.win_m0) * (p.win_n1 - p.win_n0) +
                              (col - p.win_n0)) * NG + g;
          p.acc[idx] = (int32_t)(y[k] * kUnit);
        }
      }
    } else {
      const uint32_t sab = (uint32_t)__shfl((int)sc.sa[r], 16 * i + 4 * q4 + (lane & 3));
      const uint32_t swb = (uint32_t)__shfl((int)sc.sw, 16 * i + r16);
      const float sa = __half2float(__ushort_as_half((unsigned short)sab)) * kUnit;
      const float sw = live ? __half2float(__ushort_as_half((unsigned short)swb)) : 0.0f;
      const f32x4 P = scale_products(sa, sw);
      #pragma unroll
      for (int k = 0; k < 4; ++k) C[r][k] = __builtin_fmaf(y[k], P[k], C[r][k]);
    }
  }
}

// Every wave runs the same number of batches and barriers: the longest slot's
// count.  Waves whose column block lies past N, or whose slot has fewer
// K-blocks, still load their share of the activations and meet every barrier.
template <int R, int S, bool DIAG>
__global__ __launch_bounds__(kCBW * S * 64) void skinny_shared_kernel(GemmArgs p) {
  __shared__ __attribute__((aligned(16))) uint8_t sA[SharedA<R, S>::Bytes];
  __shared__ f32x4 red[S > 1 ? kCBW * S : 1][R][64];
  const int lane = threadIdx.x & 63;
  const int r16 = lane & 15, q4 = lane >> 4;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int slot = wave / kCBW, wi = wave % kCBW;
  const int cb = blockIdx.x * kCBW + wi;
  const bool active = cb < p.N / 16;
  const int n0 = active ? cb * 16 : 0;
  const int col = n0 + r16;
  const int NG = p.K / kG;
  const int g0 = NG * slot / S, g1 = NG * (slot + 1) / S;
  const int nb = ((NG + S - 1) / S + kD - 1) / kD;  // batches of the longest slot
  auto area = [&](int buf, int i) { return sA + (((buf * S + slot) * kD + i) * R) * 2048; };

  f32x4 C[R];
  #pragma unroll
  for (int r = 0; r < R; ++r) C[r] = f32x4{0.f, 0.f, 0.f, 0.f};
  u32x4 wa[kD], wb[kD];
  SBatch<R> sa_, sb_;
  AChunk<R> ch;
  // Waves past N load and compute from column block 0 and store nothing.
  // prologue: batch 0's activations stored, its weights and scales in flight
  chunk_load<R>(p, min(g0 + wi, NG - 1), ch);
  load_scales<R>(p, g0, n0, sa_);
  load_w(p, g0, g1 - 1, n0, wa);
  chunk_store<R>(ch, area(0, wi));
  __syncthreads();
  // One batch b from weights wc and scales sc.  With NEXT, the next batch's
  // activation chunk and scales are loaded first and its weights last, so
  // that the wait for the chunk before the barrier leaves the weight loads in
  // flight (loads complete in order).
  auto batch_shared = [&](auto next, int b, const u32x4 (&wc)[kD], u32x4 (&wn)[kD],
                          const SBatch<R>& sc, SBatch<R>& sn) {
    constexpr bool NEXT = decltype(next)::value;
    const int gb = g0 + kD * b;
    if constexpr (NEXT) {
      chunk_load<R>(p, min(gb + kD + wi, NG - 1), ch);
      load_scales<R>(p, gb + kD, n0, sn);
      load_w(p, gb + kD, g1 - 1, n0, wn);
    }
    issue_point();
    #pragma unroll
    for (int i = 0; i < kD; ++i) {
      const int g = min(gb + i, NG - 1);
      compute_shared<R, DIAG>(p, wc[i], i, g, is8(p, g), gb + i < g1, n0, area(b & 1, i), sc, C);
      __builtin_amdgcn_sched_barrier(0);  // keep steps apart: fewer live registers
    }
    if constexpr (NEXT) chunk_store<R>(ch, area((b + 1) & 1, wi));
    __syncthreads();
  };
  using Next = std::true_type;
  using Last = std::false_type;
  int b = 0;
  for (; b + 2 < nb; b += 2) {
    batch_shared(Next(), b, wa, wb, sa_, sb_);
    batch_shared(Next(), b + 1, wb, wa, sb_, sa_);
  }
  if (nb - b == 2) {
    batch_shared(Next(), b, wa, wb, sa_, sb_);
    batch_shared(Last(), b + 1, wb, wa, sb_, sa_);
  } else {
    batch_shared(Last(), b, wa, wb, sa_, sb_);
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
      for (int s = 1; s < S; ++s) C[r] += red[wave + s * kCBW][r][lane];
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

template <int R, int S>
hipError_t launch_shared(const GemmArgs& a, bool diag, hipStream_t stream) {
  const int blocks = (a.N / 16 + kCBW - 1) / kCBW;
  const dim3 grid(blocks), block(kCBW * S * 64);
  if (diag)
    hipLaunchKernelGGL((skinny_shared_kernel<R, S, true>), grid, block, 0, stream, a);
  else
    hipLaunchKernelGGL((skinny_shared_kernel<R, S, false>), grid, block, 0, stream, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_gemm_skinny(const GemmArgs& a, bool diag, hipStream_t stream) {
  if (a.splits < 1 || kWaves % a.splits != 0) return hipErrorInvalidValue;
  // 8 < M <= 32: the shared-activation kernel.  At M <= 8 the per-wave kernel
  // is faster: it needs fewer registers (four waves per SIMD against three),
  // and with so few rows its activation reads cost little.
  const int R = (a.M + 15) / 16;
  if (skinny_shared(a.M, a.splits)) {
    if (R == 1)
      return a.splits == 1 ? launch_shared<1, 1>(a, diag, stream) : launch_shared<1, 2>(a, diag, stream);
    return a.splits == 1 ? launch_shared<2, 1>(a, diag, stream) : launch_shared<2, 2>(a, diag, stream);
  }
  switch (R) {
    case 1: return launch_r<1>(a, diag, stream);
    case 2: return launch_r<2>(a, diag, stream);
    case 3: return launch_r<3>(a, diag, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace comet
