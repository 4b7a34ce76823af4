// gemm_skinny.hip -- W4Ax GEMM for few tokens (decode) on gfx950.
//
// With a few tokens the GEMM is a weight stream: every 4-bit weight is read
// from HBM once and used by few activation rows, so the bound is HBM
// bandwidth, not the matrix cores.  Three designs live here:
//   * the per-wave and shared-activation kernels (M <= 48, any N), first
//     below;
//   * the stream kernels (M <= 64, when the 16-column weight panels divide
//     evenly over the CUs): each workgroup owns whole panels and streams them
//     as contiguous runs, at the end of the file.
// In the per-wave kernel each wave owns 16 output columns and
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
      // exact: integers below 2^24 units
      y = mfma_fp8_x8(ah, wf, mfma_fp8(al, wf, f32x4{0.f, 0.f, 0.f, 0.f}));
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
// LDS area at [batch buffer][slot][K-block][row block] (2 KB each: all lanes'
// first 16 bytes, then all lanes' second 16 bytes, so that both fragment
// reads are linear and free of bank conflicts; 32 bytes per lane in a row
// read at ~60% of the rate); one barrier per batch publishes it.  Weights, scales and dequantization are
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
    *reinterpret_cast<u32x4*>(dst + r * 2048 + lane * 16) = lo;
    *reinterpret_cast<u32x4*>(dst + r * 2048 + 1024 + lane * 16) = hi;
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
    const u32x4 x0 = *reinterpret_cast<const u32x4*>(frag + r * 2048 + lane * 16);
    const u32x4 x1 = *reinterpret_cast<const u32x4*>(frag + r * 2048 + 1024 + lane * 16);
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
      // exact: integers below 2^24 units
      y = mfma_fp8_x8(ah, wf, mfma_fp8(al, wf, f32x4{0.f, 0.f, 0.f, 0.f}));
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


// ---------------------------------------------------------------------------
// Few-token stream kernel (M <= 8).  W_packed's 16-row panels make the whole
// weight matrix one contiguous run of 1 KB items, item p * NG + g being panel
// p's K-block g.  Each workgroup owns kp whole panels and its 16 waves split
// the workgroup's kp * NG items into contiguous ranges, so every wave streams
// one long run of W_packed (56 KB for the LLaMA-3-70B gate_up), four items
// per batch with the next batch in flight, and the grid is exactly one wave
// of workgroups (no tail round).  A wave accumulates one panel at a time: a
// panel it covers whole is stored at once; the partial first and last panels
// of its range stay in registers until the end, go through LDS, and the wave
// that holds a panel's first item adds the partials of the following waves
// in wave order (no cross-workgroup traffic; deterministic).
//
// Per workgroup, LDS holds the activation scales and a table of every
// block's offset in A_packed and precision, read once per batch.  With LDSA
// the activation operand itself is unpacked to FP8 into LDS once per
// workgroup (1 KB per 4-bit block, the hi and lo parts of an 8-bit block),
// so an item's fragment is two LDS reads with no unpacking; otherwise each
// item reads its fragment from L2 and unpacks it.
constexpr int kStreamWaves = 16;
constexpr int kSB = 4;  // items per batch

struct StreamLayout {
  int a_bytes;     // unpacked activation operand (LDSA), else 0
  int sa_off;      // activation scales, fp16 [NG][8]
  int info_off;    // block table, int [NG + kSB]
  int bytes;       // total, at least the partials' [waves][2][64] f32x4
};

__host__ __device__ inline StreamLayout stream_layout(int NG, int n8, bool ldsa) {
  StreamLayout l;
  l.a_bytes = ldsa ? (NG + n8) * 1024 : 0;
  l.sa_off = l.a_bytes;
  l.info_off = l.sa_off + NG * 16;
  const int end = l.info_off + (NG + kSB) * 4;
  const int part = kStreamWaves * 2 * 64 * 16;
  l.bytes = end > part ? end : part;
  return l;
}

// Weight scales of the batch whose first item is block g of local panel q:
// lane l holds the two fp16 scales of columns 2 (l % 8), 2 (l % 8) + 1 of
// item l / 8 (panel clamped to qmax past the range; such items are never
// computed).
__device__ __forceinline__ uint32_t stream_sw(const GemmArgs& p, int pbase, int q, int g,
                                              int qmax) {
  const int lane = threadIdx.x & 63;
  const int NG = p.K / kG;
  int gi = g + (lane >> 3), qi = q;
  if (gi >= NG) {
    gi -= NG;
    ++qi;
  }
  qi = min(qi, qmax);
  return *reinterpret_cast<const uint32_t*>(p.sw + (size_t)gi * p.N + 16 * (pbase + qi) +
                                            2 * (lane & 7));
}

// Weights of items it0 .. it0 + 3 (clamped to ilast): lane r + 16 q reads row
// r's 16-byte chunk q of each item's kilobyte.
__device__ __forceinline__ void stream_w(const uint8_t* wbase, int it0, int ilast,
                                         u32x4 (&w)[kSB]) {
  const int lane = threadIdx.x & 63;
  const uint8_t* b = wbase + (lane & 15) * 64 + (lane >> 4) * 16;
  #pragma unroll
  for (int i = 0; i < kSB; ++i) {
    const int it = min(it0 + i, ilast);
    w[i] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(b + (size_t)it * 1024));
  }
}

__device__ __forceinline__ void stream_store(const GemmArgs& p, int panel, const f32x4& C) {
  const int lane = threadIdx.x & 63;
  const int col = 16 * panel + (lane & 15);
  #pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int row = 4 * (lane >> 4) + i;
    if (row < p.M) p.out[(size_t)row * p.N + col] = __half_as_ushort(__float2half_rn(C[i]));
  }
}

// Activation fragment of block g (offset aoff in units of M * 64 bytes) for
// M <= 8 from L2: rows 8..15 of the operand are padding, so lane r of each
// 16-lane row reads row r & 7: its first 16 bytes, or for an 8-bit block with
// r >= 8 the second 16 bytes of the same 32-byte chunk (moved down eight
// lanes at use).
__device__ __forceinline__ u32x4 stream_a_l2(const GemmArgs& p, int aoff, bool b8) {
  const int lane = threadIdx.x & 63;
  const int r16 = lane & 15, q4 = lane >> 4;
  const uint32_t ub8 = b8 ? 1u : 0u;
  const uint32_t row = (uint32_t)min(r16 & 7, p.M - 1);
  const uint32_t second = ((uint32_t)r16 >> 3) & ub8;
  return *reinterpret_cast<const u32x4*>(p.A + (size_t)p.M * 64 * (size_t)aoff +
                                         (row << (6 + ub8)) + ((uint32_t)q4 << (4 + ub8)) +
                                         (second << 4));
}

// One item: the block sums y of weights wraw (16 columns) against block g's
// activation fragment, from LDS (LDSA: unpacked at aoff KB) or from the L2
// fragment xa; then the dequantization C += y * (sa sw), or (DIAG) the exact
// sums of the window.
template <bool LDSA, bool DIAG>
__device__ __forceinline__ void stream_step(const GemmArgs& p, const uint8_t* sA,
                                            const uint16_t* sSa, const u32x4& wraw,
                                            const u32x4& xa, int g, int aoff, bool b8,
                                            uint32_t swpair, int i, int n0, f32x4& C) {
  const int lane = threadIdx.x & 63;
  const int r16 = lane & 15, q4 = lane >> 4;
  u32x4 wlo, whi;
  unpack4(wraw, wlo, whi);
  const i32x8 wf = {(int)wlo[0], (int)wlo[1], (int)wlo[2], (int)wlo[3],
                    (int)whi[0], (int)whi[1], (int)whi[2], (int)whi[3]};
  f32x4 y;
  if constexpr (LDSA) {
    // row r16 & 7's chunks 2 q4 and 2 q4 + 1, at their swizzled positions
    const int r8 = r16 & 7;
    const uint8_t* fa = sA + (size_t)aoff * 1024 + r8 * 128 + (((2 * q4) ^ r8) << 4);
    const uint8_t* fb = sA + (size_t)aoff * 1024 + r8 * 128 + (((2 * q4 + 1) ^ r8) << 4);
    const u32x4 a0 = *reinterpret_cast<const u32x4*>(fa);
    const u32x4 a1 = *reinterpret_cast<const u32x4*>(fb);
    const i32x8 af = {(int)a0[0], (int)a0[1], (int)a0[2], (int)a0[3],
                      (int)a1[0], (int)a1[1], (int)a1[2], (int)a1[3]};
    if (b8) {
      const u32x4 l0 = *reinterpret_cast<const u32x4*>(fa + 1024);
      const u32x4 l1 = *reinterpret_cast<const u32x4*>(fb + 1024);
      const i32x8 al = {(int)l0[0], (int)l0[1], (int)l0[2], (int)l0[3],
                        (int)l1[0], (int)l1[1], (int)l1[2], (int)l1[3]};
      // exact: integers below 2^24 units
      y = mfma_fp8_x8(af, wf, mfma_fp8(al, wf, f32x4{0.f, 0.f, 0.f, 0.f}));
    } else {
      y = mfma_fp8(af, wf, f32x4{0.f, 0.f, 0.f, 0.f});
    }
  } else {
    if (b8) {
      i32x8 al, ah;
      u32x4 x1;
      #pragma unroll
      for (int k = 0; k < 4; ++k)
        x1[k] = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)xa[k], 0x128, 0xF, 0xF, false);
      #pragma unroll
      for (int k = 0; k < 4; ++k) {
        al[k] = (int)lo8(xa[k]);
        al[4 + k] = (int)lo8(x1[k]);
        ah[k] = (int)hi8(xa[k]);
        ah[4 + k] = (int)hi8(x1[k]);
      }
      y = mfma_fp8_x8(ah, wf, mfma_fp8(al, wf, f32x4{0.f, 0.f, 0.f, 0.f}));
    } else {
      u32x4 alo, ahi;
      unpack4(xa, alo, ahi);
      const i32x8 af = {(int)alo[0], (int)alo[1], (int)alo[2], (int)alo[3],
                        (int)ahi[0], (int)ahi[1], (int)ahi[2], (int)ahi[3]};
      y = mfma_fp8(af, wf, f32x4{0.f, 0.f, 0.f, 0.f});
    }
  }
  if constexpr (DIAG) {
    const int NG = p.K / kG;
    const int col = n0 + r16;
    #pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int row = 4 * q4 + k;
      if (row >= p.win_m0 && row < p.win_m1 && col >= p.win_n0 && col < p.win_n1) {
        const size_t idx = ((size_t)(row - p.win_m0) * (p.win_n1 - p.win_n0) +
                            (col - p.win_n0)) * NG + g;
        p.acc[idx] = (int32_t)(y[k] * kUnit);
      }
    }
  } else {
    // 4x4x1 operands: activation scale of row 4 q4 + (lane & 3), weight scale
    // of column lane % 16 (lane 8 i + c / 2 holds it, half c % 2)
    const uint32_t swb = (uint32_t)__shfl((int)swpair, 8 * i + (r16 >> 1)) >> (16 * (r16 & 1));
    const float sa =
        __half2float(__ushort_as_half(sSa[g * 8 + min(4 * q4 + (lane & 3), p.M - 1)])) * kUnit;
    const float sw = __half2float(__ushort_as_half((unsigned short)swb));
    const f32x4 P = scale_products(sa, sw);
    #pragma unroll
    for (int k = 0; k < 4; ++k) C[k] = __builtin_fmaf(y[k], P[k], C[k]);
  }
}

template <bool LDSA, bool DIAG>
__global__ __launch_bounds__(kStreamWaves * 64) void skinny_stream_kernel(GemmArgs p, int kp,
                                                                          StreamLayout lay) {
  constexpr int NW = kStreamWaves;
  extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int NG = p.K / kG;
  const int items = kp * NG;
  const int pbase = blockIdx.x * kp;  // first panel of the workgroup
  const uint8_t* wbase = p.W + (size_t)pbase * NG * 1024;
  // this wave's items [i0, i1) (local indices) and its first and last panels
  const int i0 = items * wave / NW, i1 = items * (wave + 1) / NW;
  const int q0 = i0 / NG, q1 = (i1 - 1) / NG;
  uint8_t* sA = smem;
  uint16_t* sSa = reinterpret_cast<uint16_t*>(smem + lay.sa_off);
  int* sInfo = reinterpret_cast<int*>(smem + lay.info_off);

  // (panel, block) of the next batch to load, wave-uniform
  int lq = q0, lg = i0 - q0 * NG;
  auto advance = [&]() {
    lg += kSB;
    if (lg >= NG) {
      lg -= NG;
      ++lq;
    }
  };
  u32x4 wa[kSB], wb[kSB];
  uint32_t swa = 0, swb = 0;
  if (i0 < i1) {
    stream_w(wbase, i0, i1 - 1, wa);
    swa = stream_sw(p, pbase, lq, lg, kp - 1);
    advance();
  }
  // per workgroup: activation scales, block table (four entries past the end
  // wrap to blocks 0..3), and with LDSA the unpacked activation operand: for
  // every block and row r < 8 (clamped to M - 1) 128 FP8 bytes at aoff KB +
  // 128 r, 16-byte chunk c at chunk position c ^ r (the eight rows a fragment
  // read touches then sit on distinct banks; unswizzled, the read ran at ~58%
  // of the rate), an 8-bit block's lo parts one KB after its hi parts
  for (int e = threadIdx.x; e < NG * 8; e += NW * 64)
    sSa[e] = p.sa[(size_t)(e >> 3) * p.M + min(e & 7, p.M - 1)];
  for (int e = threadIdx.x; e < NG + kSB; e += NW * 64) {
    const int gi = e < NG ? e : e - NG;
    sInfo[e] = aoff_of(p, gi) | (is8(p, gi) ? 1 << 16 : 0);
  }
  if constexpr (LDSA) {
    for (int e = threadIdx.x; e < NG * 64; e += NW * 64) {
      const int gi = e >> 6, r = (e >> 3) & 7, c = e & 7;  // block, row, 16-code chunk
      const int ao = aoff_of(p, gi);
      const int row = min(r, p.M - 1);
      uint8_t* dst = sA + (size_t)ao * 1024 + r * 128 + ((c ^ r) << 4);
      if (!is8(p, gi)) {
        const uint2 v =
            *reinterpret_cast<const uint2*>(p.A + (size_t)ao * p.M * 64 + row * 64 + c * 8);
        *reinterpret_cast<u32x4*>(dst) =
            u32x4{v.x & kSignMag, rotr4(v.x) & kSignMag, v.y & kSignMag, rotr4(v.y) & kSignMag};
      } else {
        const u32x4 v =
            *reinterpret_cast<const u32x4*>(p.A + (size_t)ao * p.M * 64 + row * 128 + c * 16);
        *reinterpret_cast<u32x4*>(dst) = u32x4{hi8(v[0]), hi8(v[1]), hi8(v[2]), hi8(v[3])};
        *reinterpret_cast<u32x4*>(dst + 1024) = u32x4{lo8(v[0]), lo8(v[1]), lo8(v[2]), lo8(v[3])};
      }
    }
  }
  __syncthreads();

  f32x4 C = f32x4{0.f, 0.f, 0.f, 0.f};
  f32x4 F = C, L = C;  // partials of the first and last panel of the range
  if (i0 < i1) {
    int q = q0, g = i0 - q0 * NG;
    // one batch of four items from weights wc / scales swc while the next
    // batch loads into wn / swn
    auto batch = [&](int ib, const u32x4 (&wc)[kSB], u32x4 (&wn)[kSB], uint32_t swc,
                     uint32_t& swn) {
      // this batch's block table entries (one LDS read, then scalars) and,
      // from L2, its activation fragments
      const int info = sInfo[g + (lane & (kSB - 1))];
      u32x4 xa[kSB];
      if constexpr (!LDSA) {
        #pragma unroll
        for (int i = 0; i < kSB; ++i) {
          const int inf = __builtin_amdgcn_readlane(info, i);
          xa[i] = stream_a_l2(p, inf & 0xFFFF, (inf >> 16) & 1);
        }
      }
      stream_w(wbase, ib + kSB, i1 - 1, wn);
      swn = stream_sw(p, pbase, lq, lg, kp - 1);
      advance();
      issue_point();
      #pragma unroll
      for (int i = 0; i < kSB; ++i) {
        const int it = ib + i;
        const int inf = __builtin_amdgcn_readlane(info, i);
        if (it < i1) {
          stream_step<LDSA, DIAG>(p, sA, sSa, wc[i], xa[LDSA ? 0 : i], g, inf & 0xFFFF,
                                  (inf >> 16) & 1, swc, i, 16 * (pbase + q), C);
          const bool last = g + 1 == NG;
          g = last ? 0 : g + 1;
          if (last || it + 1 == i1) {
            // end of a panel or of the range
            if constexpr (!DIAG) {
              if (q * NG >= i0 && (q + 1) * NG <= i1)
                stream_store(p, pbase + q, C);
              else if (q == q0)
                F = C;
              else
                L = C;
            }
            C = f32x4{0.f, 0.f, 0.f, 0.f};
            ++q;
          }
        }
      }
    };
    for (int ib = i0;;) {
      batch(ib, wa, wb, swa, swb);
      ib += kSB;
      if (ib >= i1) break;
      batch(ib, wb, wa, swb, swa);
      ib += kSB;
      if (ib >= i1) break;
    }
  }
  if constexpr (DIAG) return;
  // partials through LDS (the activation copy is no longer needed)
  __syncthreads();
  f32x4* part = reinterpret_cast<f32x4*>(smem);  // [NW][2][64]
  part[(wave * 2 + 0) * 64 + lane] = F;
  part[(wave * 2 + 1) * 64 + lane] = L;
  __syncthreads();
  for (int q = q0; q <= q1 && i0 < i1; ++q) {
    const int first = q * NG, end = (q + 1) * NG;
    if (first < i0 || end <= i1) continue;  // started by an earlier wave, or complete here
    f32x4 acc = part[(wave * 2 + (q == q0 ? 0 : 1)) * 64 + lane];
    for (int w = wave + 1; w < NW; ++w) {
      const int j0 = items * w / NW, j1 = items * (w + 1) / NW;
      if (j0 >= end) break;
      if (j1 > j0) acc += part[(w * 2) * 64 + lane];
    }
    stream_store(p, pbase + q, acc);
  }
}

template <bool LDSA, bool DIAG>
const void* stream_fn() {
  return reinterpret_cast<const void*>(&skinny_stream_kernel<LDSA, DIAG>);
}

int map_n8(const BlockMap& m) {
  int n = 0;
  for (int w = 0; w < kMaxBlocks / 64; ++w) n += __builtin_popcountll(m.bits[w]);
  return n;
}

// ---------------------------------------------------------------------------
// Chunked weight-stream kernel (8 < M <= 64).  As in the stream kernel above,
// each workgroup owns kp whole 16-column panels (the panels divide evenly over
// the CUs), so the weights leave HBM once, as long contiguous runs, and no
// workgroup waits for another.  With more than eight rows the activation
// operand of a whole row no longer fits in LDS, so the K-blocks are walked in
// chunks of kChC: the workgroup's eight waves stage one chunk's activation
// fragments (all R row blocks, 4-bit codes unpacked once) and scales in LDS
// while computing the previous one, and one barrier per chunk publishes them.
// The chunk's kp * kChC items (panel, K-block) are split evenly over the waves
// in panel-major order, the same way in every chunk, so a wave always works on
// the same (at most three) panels and keeps their accumulators in registers.
// Each item's weights are one 16-byte load per lane, issued a chunk ahead;
// per item the wave runs R MFMAs (2R for an 8-bit block) against the staged
// fragments.  At the end, panels split between waves are added through LDS in
// wave order (deterministic).
constexpr int kChWaves = 8;
constexpr int kChC = 4;                   // K-blocks per chunk
constexpr int kChSeg = 3;                 // panels (segments) per wave
constexpr int kChItems = 2 * kChC;        // most items per wave and chunk
constexpr int kChMaxM = 64;               // rows (four row blocks)

template <int R>
struct ChLayout {
  static constexpr int Frag = 2048;                   // one (K-block, row block): 2 x 64 lanes x 16 B
  static constexpr int Stage = kChC * R * Frag;       // a chunk's activation fragments
  static constexpr int Scales = kChC * 16 * R * 4;    // its fp32 activation scales (x 2^18)
  static constexpr int Buf = Stage + Scales;
  static constexpr int Part = kChWaves * 2 * R * 64 * 16;  // partial panels at the end
  static constexpr int Bytes = 2 * Buf > Part ? 2 * Buf : Part;
  static constexpr int Sets = (kChC * R + kChWaves - 1) / kChWaves;  // fragment sets per wave
};

// One staged fragment set (K-block c of the chunk, row block r): this lane's
// 32 bytes (row 16 r + lane % 16, codes 32 (lane / 16) .. + 31), as loaded.
struct ChSet {
  u32x4 v[2];
  bool b8;
};

// Loads of fragment set f of chunk ch (clamped into range: sets past the
// chunk's end re-read a valid set and are not stored).
template <int R>
__device__ __forceinline__ void ch_set_load(const GemmArgs& p, int ch, int f, ChSet& s) {
  const int lane = threadIdx.x & 63;
  const int NG = p.K / kG;
  const int c = min(f / R, kChC - 1), r = f % R;
  const int g = min(ch * kChC + c, NG - 1);
  s.b8 = is8(p, g);
  const uint32_t b8 = s.b8 ? 1u : 0u;
  const uint32_t row = (uint32_t)min(16 * r + (lane & 15), p.M - 1);
  const uint8_t* base = p.A + (size_t)p.M * 64 * (size_t)aoff_of(p, g) + (row << (6 + b8)) +
                        ((uint32_t)(lane >> 4) << (4 + b8));
  s.v[0] = *reinterpret_cast<const u32x4*>(base);
  s.v[1] = *reinterpret_cast<const u32x4*>(base + (b8 << 4));
}

template <int R>
__device__ __forceinline__ void ch_set_store(const ChSet& s, int f, uint8_t* stage) {
  const int lane = threadIdx.x & 63;
  u32x4 lo = s.v[0], hi = s.v[1];
  if (!s.b8) unpack4(s.v[0], lo, hi);
  uint8_t* dst = stage + f * ChLayout<R>::Frag + lane * 16;  // f = c * R + r
  *reinterpret_cast<u32x4*>(dst) = lo;
  *reinterpret_cast<u32x4*>(dst + 1024) = hi;
}

// Activation scales of chunk ch: entry c * 16 R + row, fp16 loaded here,
// stored as fp32 times 2^18.  Thread t handles entries t and t + 512.
template <int R>
struct ChScales {
  uint32_t v[(kChC * 16 * R + kChWaves * 64 - 1) / (kChWaves * 64)];
};
template <int R>
__device__ __forceinline__ void ch_scales_load(const GemmArgs& p, int ch, ChScales<R>& s) {
  const int NG = p.K / kG;
  #pragma unroll
  for (int i = 0; i < (int)(sizeof(s.v) / sizeof(s.v[0])); ++i) {
    const int e = min((int)threadIdx.x + i * kChWaves * 64, kChC * 16 * R - 1);
    const int c = e / (16 * R), row = e % (16 * R);
    const int g = min(ch * kChC + c, NG - 1);
    s.v[i] = p.sa[(size_t)g * p.M + min(row, p.M - 1)];
  }
}
template <int R>
__device__ __forceinline__ void ch_scales_store(const ChScales<R>& s, float* dst) {
  #pragma unroll
  for (int i = 0; i < (int)(sizeof(s.v) / sizeof(s.v[0])); ++i) {
    const int e = (int)threadIdx.x + i * kChWaves * 64;
    if (e < kChC * 16 * R) dst[e] = __half2float(__ushort_as_half((unsigned short)s.v[i])) * kUnit;
  }
}

// Weights and weight scales of this wave's item k of chunk ch: item t = tb +
// k (clamped below te: a slot past the wave's items re-reads its last item,
// which costs no extra HBM traffic), panel pbase + t / kChC, K-block ch *
// kChC + t % kChC clamped below NG.
struct ChW {
  u32x4 w;
  uint32_t sw;
};
__device__ __forceinline__ void ch_w_load(const GemmArgs& p, int pbase, int tb, int te, int k,
                                          int ch, ChW& x) {
  const int lane = threadIdx.x & 63;
  const int NG = p.K / kG;
  // wave-uniform item, kept in scalar registers: each load is a scalar base
  // plus the lane's constant offset
  const int t = __builtin_amdgcn_readfirstlane(min(tb + k, te - 1));
  const int g = min(ch * kChC + t % kChC, NG - 1);
  const int panel = pbase + t / kChC;
  const uint8_t* wb = p.W + ((size_t)panel * NG + g) * 1024;
  const uint16_t* sb = p.sw + (size_t)g * p.N + 16 * panel;
  x.w = __builtin_nontemporal_load(
      reinterpret_cast<const u32x4*>(wb + (uint32_t)((lane & 15) * 64 + (lane >> 4) * 16)));
  x.sw = sb[lane & 15];
}

// The wave's items at position c of the chunk (K-block g): with at most
// 2 kChC items per wave, two slots kA and kA + kChC (segments sA and sA + 1),
// the second computed only with TWO.  Each staged activation fragment (and
// scale vector) is read once for both items.
template <int R, bool DIAG, bool TWO>
__device__ __forceinline__ void ch_group(const GemmArgs& p, const ChW& xa, const ChW& xb, int g,
                                         int c, int n0a, const uint8_t* sA, const float* sS,
                                         f32x4 (&Ca)[R], f32x4 (&Cb)[R]) {
  const int lane = threadIdx.x & 63;
  const int r16 = lane & 15, q4 = lane >> 4;
  const int NG = p.K / kG;
  const bool b8 = is8(p, g);
  auto wfrag = [](const u32x4& w) {
    u32x4 lo, hi;
    unpack4(w, lo, hi);
    return i32x8{(int)lo[0], (int)lo[1], (int)lo[2], (int)lo[3],
                 (int)hi[0], (int)hi[1], (int)hi[2], (int)hi[3]};
  };
  const i32x8 wa = wfrag(xa.w);
  i32x8 wb = wa;
  if constexpr (TWO) wb = wfrag(xb.w);
  const float swa = __half2float(__ushort_as_half((unsigned short)xa.sw));
  const float swb = __half2float(__ushort_as_half((unsigned short)xb.sw));
  // row block r + 1's fragment is read while row block r computes
  const uint8_t* fr = sA + c * R * ChLayout<R>::Frag + lane * 16;
  u32x4 n0v = *reinterpret_cast<const u32x4*>(fr), n1v = *reinterpret_cast<const u32x4*>(fr + 1024);
  #pragma unroll
  for (int r = 0; r < R; ++r) {
    const u32x4 x0 = n0v, x1 = n1v;
    if (r + 1 < R) {
      n0v = *reinterpret_cast<const u32x4*>(fr + (r + 1) * ChLayout<R>::Frag);
      n1v = *reinterpret_cast<const u32x4*>(fr + (r + 1) * ChLayout<R>::Frag + 1024);
    }
    f32x4 ya, yb = {0.f, 0.f, 0.f, 0.f};  // yb: second panel (TWO) only
    if (b8) {
      i32x8 al, ah;
      #pragma unroll
      for (int k = 0; k < 4; ++k) {
        al[k] = (int)lo8(x0[k]);
        al[4 + k] = (int)lo8(x1[k]);
        ah[k] = (int)hi8(x0[k]);
        ah[4 + k] = (int)hi8(x1[k]);
      }
      // exact: integers below 2^24 units
      ya = mfma_fp8_x8(ah, wa, mfma_fp8(al, wa, f32x4{0.f, 0.f, 0.f, 0.f}));
      if constexpr (TWO) yb = mfma_fp8_x8(ah, wb, mfma_fp8(al, wb, f32x4{0.f, 0.f, 0.f, 0.f}));
    } else {
      const i32x8 af = {(int)x0[0], (int)x0[1], (int)x0[2], (int)x0[3],
                        (int)x1[0], (int)x1[1], (int)x1[2], (int)x1[3]};
      ya = mfma_fp8(af, wa, f32x4{0.f, 0.f, 0.f, 0.f});
      if constexpr (TWO) yb = mfma_fp8(af, wb, f32x4{0.f, 0.f, 0.f, 0.f});
    }
    if constexpr (DIAG) {
      #pragma unroll
      for (int h = 0; h < (TWO ? 2 : 1); ++h) {
        const int col = n0a + 16 * h + r16;
        const f32x4 y = h ? yb : ya;
        #pragma unroll
        for (int k = 0; k < 4; ++k) {
          const int row = 16 * r + 4 * q4 + k;
          if (row >= p.win_m0 && row < p.win_m1 && col >= p.win_n0 && col < p.win_n1) {
            const size_t idx = ((size_t)(row - p.win_m0) * (p.win_n1 - p.win_n0) +
                                (col - p.win_n0)) * NG + g;
            p.acc[idx] = (int32_t)(y[k] * kUnit);
          }
        }
      }
    } else {
      const f32x4 sa4 = *reinterpret_cast<const f32x4*>(sS + c * 16 * R + 16 * r + 4 * q4);
      const f32x4 Pa = sa4 * swa;  // exact: 11-bit by 11-bit significands
      #pragma unroll
      for (int k = 0; k < 4; ++k) Ca[r][k] = __builtin_fmaf(ya[k], Pa[k], Ca[r][k]);
      if constexpr (TWO) {
        const f32x4 Pb = sa4 * swb;
        #pragma unroll
        for (int k = 0; k < 4; ++k) Cb[r][k] = __builtin_fmaf(yb[k], Pb[k], Cb[r][k]);
      }
    }
    __builtin_amdgcn_sched_barrier(0);
  }
}

// The chunk loop for a wave whose first item sits at position A of its
// panel's kChC K-blocks (A = tb % kChC): item k is then position (A + k) %
// kChC of the wave's panel segment (A + k) / kChC, both known at compile time,
// so the accumulators and weight registers are indexed statically.  Items
// are computed by position (K-block) of the chunk, the two items at one
// position together.
template <int R, bool DIAG, int A>
__device__ __forceinline__ void ch_run(const GemmArgs& p, uint8_t* smem, int pbase, int tb, int te,
                                       f32x4 (&C)[kChSeg][R]) {
  using L = ChLayout<R>;
  static_assert(kChItems == 2 * kChC, "two items per chunk position");
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int NG = p.K / kG, NC = (NG + kChC - 1) / kChC;
  const int n = te - tb;  // the wave's items per chunk
  const int q0 = tb / kChC;
  auto stage = [&](int ch) { return smem + (ch & 1) * L::Buf; };
  auto scales = [&](int ch) { return reinterpret_cast<float*>(smem + (ch & 1) * L::Buf + L::Stage); };
  constexpr int H = (L::Sets + 1) / 2;  // fragment sets staged per half chunk

  // weight slot k holds item k; once a position's items are computed their
  // slots load the same items of the next chunk
  ChW w[kChItems];
  #pragma unroll
  for (int k = 0; k < kChItems; ++k) ch_w_load(p, pbase, tb, te, k, 0, w[k]);
  for (int ch = 0; ch < NC; ++ch) {
    const int cc = min(kChC, NG - ch * kChC);  // K-blocks in this chunk
    const int chn = min(ch + 1, NC - 1);      // the chunk loaded ahead (the last re-reads itself)
    const uint8_t* sA = stage(ch);
    const float* sS = scales(ch);
    ChSet st[H];
    ChScales<R> ss;
    #pragma unroll
    for (int j = 0; j < H; ++j) ch_set_load<R>(p, chn, min(wave + kChWaves * j, kChC * R - 1), st[j]);
    ch_scales_load<R>(p, chn, ss);
    issue_point();
    #pragma unroll
    for (int c = 0; c < kChC; ++c) {
      const int ka = (c - A + kChC) % kChC, kb = ka + kChC;  // the position's two slots
      const int sa = (A + ka) / kChC;                        // segment of slot ka
      const ChW xa = w[ka], xb = w[kb];
      ch_w_load(p, pbase, tb, te, ka, chn, w[ka]);
      ch_w_load(p, pbase, tb, te, kb, chn, w[kb]);
      if (c < cc && ka < n) {
        const int g = ch * kChC + c, n0a = 16 * (pbase + q0 + sa);
        if (kb < n)
          ch_group<R, DIAG, true>(p, xa, xb, g, c, n0a, sA, sS, C[sa], C[sa + 1 < kChSeg ? sa + 1 : sa]);
        else
          ch_group<R, DIAG, false>(p, xa, xb, g, c, n0a, sA, sS, C[sa], C[sa]);
      }
      if (c == kChC / 2 - 1 && H < L::Sets) {
        // halfway: store the first half of the next chunk's fragments and
        // load the second
        if (ch + 1 < NC) {
          #pragma unroll
          for (int j = 0; j < H; ++j) {
            const int f = wave + kChWaves * j;
            if (f < kChC * R) ch_set_store<R>(st[j], f, stage(ch + 1));
          }
        }
        #pragma unroll
        for (int j = 0; j < H; ++j)
          ch_set_load<R>(p, chn, min(wave + kChWaves * (H + j), kChC * R - 1), st[j]);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    if (ch + 1 < NC) {
      const int j0 = H < L::Sets ? H : 0;
      #pragma unroll
      for (int j = 0; j < H; ++j) {
        const int f = wave + kChWaves * (j0 + j);
        if (j0 + j < L::Sets && f < kChC * R) ch_set_store<R>(st[j], f, stage(ch + 1));
      }
      ch_scales_store<R>(ss, scales(ch + 1));
    }
    __syncthreads();
  }
}

template <int R, bool DIAG>
__global__ __launch_bounds__(kChWaves * 64) void skinny_chunk_kernel(GemmArgs p, int kp) {
  extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
  using L = ChLayout<R>;
  const int lane = threadIdx.x & 63;
  const int r16 = lane & 15, q4 = lane >> 4;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int T = kp * kChC;
  const int tb = T * wave / kChWaves, te = T * (wave + 1) / kChWaves;
  const int q0 = tb / kChC;
  const int pbase = blockIdx.x * kp;

  f32x4 C[kChSeg][R];
  #pragma unroll
  for (int s = 0; s < kChSeg; ++s)
    #pragma unroll
    for (int r = 0; r < R; ++r) C[s][r] = f32x4{0.f, 0.f, 0.f, 0.f};

  // prologue: chunk 0 staged
  {
    ChSet st[L::Sets];
    ChScales<R> ss;
    #pragma unroll
    for (int j = 0; j < L::Sets; ++j) ch_set_load<R>(p, 0, min(wave + kChWaves * j, kChC * R - 1), st[j]);
    ch_scales_load<R>(p, 0, ss);
    #pragma unroll
    for (int j = 0; j < L::Sets; ++j) {
      const int f = wave + kChWaves * j;
      if (f < kChC * R) ch_set_store<R>(st[j], f, smem);
    }
    ch_scales_store<R>(ss, reinterpret_cast<float*>(smem + L::Stage));
  }
  __syncthreads();
  switch (tb % kChC) {
    case 0: ch_run<R, DIAG, 0>(p, smem, pbase, tb, te, C); break;
    case 1: ch_run<R, DIAG, 1>(p, smem, pbase, tb, te, C); break;
    case 2: ch_run<R, DIAG, 2>(p, smem, pbase, tb, te, C); break;
    default: ch_run<R, DIAG, 3>(p, smem, pbase, tb, te, C); break;
  }
  if constexpr (DIAG) return;

  // Store whole panels; a panel split between waves goes through LDS: the
  // wave holding its first item adds the pieces of the following waves.
  f32x4* part = reinterpret_cast<f32x4*>(smem);  // [waves][2][R][64]
  #pragma unroll
  for (int s = 0; s < kChSeg; ++s) {
    const int q = q0 + s;
    if (q * kChC >= te) continue;
    const bool whole = q * kChC >= tb && (q + 1) * kChC <= te;
    if (whole) {
      const int col = 16 * (pbase + q) + r16;
      #pragma unroll
      for (int r = 0; r < R; ++r)
        #pragma unroll
        for (int k = 0; k < 4; ++k) {
          const int row = 16 * r + 4 * q4 + k;
          if (row < p.M) p.out[(size_t)row * p.N + col] = __half_as_ushort(__float2half_rn(C[s][r][k]));
        }
    } else {
      const int h = s == 0 ? 0 : 1;  // the range's first or last panel
      #pragma unroll
      for (int r = 0; r < R; ++r) part[((wave * 2 + h) * R + r) * 64 + lane] = C[s][r];
    }
  }
  __syncthreads();
  #pragma unroll
  for (int s = 0; s < kChSeg; ++s) {
    const int q = q0 + s;
    if (q * kChC >= te) continue;
    const bool whole = q * kChC >= tb && (q + 1) * kChC <= te;
    if (whole || q * kChC < tb) continue;  // stored above, or started by an earlier wave
    const int h = s == 0 ? 0 : 1;
    f32x4 acc[R];
    #pragma unroll
    for (int r = 0; r < R; ++r) acc[r] = part[((wave * 2 + h) * R + r) * 64 + lane];
    for (int v = wave + 1; v < kChWaves; ++v) {
      const int vb = T * v / kChWaves, ve = T * (v + 1) / kChWaves;
      if (vb >= (q + 1) * kChC) break;
      if (ve > vb) {
        #pragma unroll
        for (int r = 0; r < R; ++r) acc[r] += part[((v * 2 + 0) * R + r) * 64 + lane];
      }
    }
    const int col = 16 * (pbase + q) + r16;
    #pragma unroll
    for (int r = 0; r < R; ++r)
      #pragma unroll
      for (int k = 0; k < 4; ++k) {
        const int row = 16 * r + 4 * q4 + k;
        if (row < p.M) p.out[(size_t)row * p.N + col] = __half_as_ushort(__float2half_rn(acc[r][k]));
      }
  }
}

template <int R>
const void* chunk_fn(bool diag) {
  return diag ? reinterpret_cast<const void*>(&skinny_chunk_kernel<R, true>)
              : reinterpret_cast<const void*>(&skinny_chunk_kernel<R, false>);
}

// Row blocks of the chunk kernel's instantiation for M rows.
int chunk_r(int M) { return (M + 15) / 16; }

const void* chunk_kernel(int R, bool diag) {
  switch (R) {
    case 1: return chunk_fn<1>(diag);
    case 2: return chunk_fn<2>(diag);
    case 3: return chunk_fn<3>(diag);
    case 4: return chunk_fn<4>(diag);
    default: return nullptr;
  }
}

int chunk_lds(int R) {
  switch (R) {
    case 1: return ChLayout<1>::Bytes;
    case 2: return ChLayout<2>::Bytes;
    case 3: return ChLayout<3>::Bytes;
    case 4: return ChLayout<4>::Bytes;
    default: return 0;
  }
}

}  // namespace

bool skinny_stream_eligible(int M, int N, int K, int cus) {
  const int P = N / 16, NG = K / kG;
  if (cus <= 0 || P % cus != 0) return false;
  const int kp = P / cus;
  if (M <= 8) return kp * NG >= kStreamWaves * 2 * kSB;
  // 8 < M <= 64: every wave has at least three items (fewer leave the
  // per-chunk staging and barrier unamortized) and at most kChItems
  return M <= kChMaxM && kp * kChC >= 3 * kChWaves &&
         (kp * kChC + kChWaves - 1) / kChWaves <= kChItems;
}

hipError_t set_skinny_attributes() {
  const void* fns[4] = {stream_fn<true, false>(), stream_fn<true, true>(), stream_fn<false, false>(),
                        stream_fn<false, true>()};
  for (const void* f : fns) {
    hipError_t e = hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, kStreamMaxLds);
    if (e != hipSuccess) return e;
  }
  for (int R : {1, 2, 3, 4})
    for (bool diag : {false, true}) {
      hipError_t e = hipFuncSetAttribute(chunk_kernel(R, diag),
                                         hipFuncAttributeMaxDynamicSharedMemorySize, chunk_lds(R));
      if (e != hipSuccess) return e;
    }
  return hipSuccess;
}

hipError_t launch_gemm_skinny(const GemmArgs& a, bool diag, hipStream_t stream) {
  if (a.M > 8 && skinny_stream_eligible(a.M, a.N, a.K, a.cus)) {
    const int R = chunk_r(a.M), kp = a.N / 16 / a.cus;
    const void* fn = chunk_kernel(R, diag);
    if (!fn) return hipErrorInvalidValue;
    GemmArgs args = a;
    void* params[] = {&args, const_cast<int*>(&kp)};
    return hipLaunchKernel(fn, dim3(a.cus), dim3(kChWaves * 64), params, chunk_lds(R), stream);
  }
  if (skinny_stream_eligible(a.M, a.N, a.K, a.cus)) {
    const int NG = a.K / kG, kp = a.N / 16 / a.cus;
    // the unpacked operand in LDS pays when it fits and a workgroup has
    // enough items to amortise unpacking it
    StreamLayout lay = stream_layout(NG, map_n8(a.map), true);
    const bool ldsa = lay.bytes <= kStreamMaxLds && kp * NG >= 512;
    if (!ldsa) lay = stream_layout(NG, 0, false);
    const dim3 grid(a.cus), block(kStreamWaves * 64);
    if (ldsa) {
      if (diag)
        hipLaunchKernelGGL((skinny_stream_kernel<true, true>), grid, block, lay.bytes, stream, a, kp, lay);
      else
        hipLaunchKernelGGL((skinny_stream_kernel<true, false>), grid, block, lay.bytes, stream, a, kp, lay);
    } else {
      if (diag)
        hipLaunchKernelGGL((skinny_stream_kernel<false, true>), grid, block, lay.bytes, stream, a, kp, lay);
      else
        hipLaunchKernelGGL((skinny_stream_kernel<false, false>), grid, block, lay.bytes, stream, a, kp, lay);
    }
    return hipGetLastError();
  }

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
