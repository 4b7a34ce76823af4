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
// Dequantization (Sec. 4.3: the scale absorbs the conversion factor):
//     C += Y * P,  P = (sa * 2^18) * sw      in fp32, once per output and K-block.
// The scale products P of a 16x16 block are one v_mfma_f32_4x4x1_16b_f32
// (16 outer products of 4 activation scales and 4 weight scales, K = 1, exact
// in fp32), laid out lane for lane like Y, so the vector ALUs only do the
// fused multiply-add; they are the co-bottleneck of this kernel.
//
// Kernel structure (the gfx950 form of the paper's software pipeline,
// Sec. 4.2, and of its tile decomposition, Sec. 4.4):
//   * persistent workgroups of 8 waves walk a host-built list of work units
//     (tile, K-block range); full tiles go to one workgroup, the fractional
//     last wave of tiles is split over all of them by cost;
//   * per K-block the workgroup stages its 256x256 tile's operands
//     HBM -> VGPR (128-bit loads) -> unpack -> LDS (double-buffered, XOR
//     swizzled rows), so every nibble is unpacked once per workgroup, and one
//     barrier per K-block separates the stages;
//   * each wave computes a 128x64 quadrant: 8x4 MFMA blocks per K-block, fed
//     from LDS, with the fp32 dequantization interleaved;
//   * split tiles write fp32 partials; the last workgroup to finish a tile
//     (arrival counter, no waiting) adds the partials in slot order and
//     stores fp16, so the result does not depend on arrival order.
#include <hip/hip_runtime.h>
#include <hip/hip_fp16.h>
#include <stdint.h>

#include "kernels.h"
#include "operand.h"

namespace comet {

namespace {

constexpr int kThreads = 512;            // 8 waves
constexpr int kWM = 128, kWN = 64;       // wave quadrant
constexpr int kRB = kWM / 16, kCB = kWN / 16;
constexpr int kA = kTileM * 128;         // LDS bytes of one A stage (fp8 or raw 8-bit codes)
constexpr int kW = kTileN * 128;         // LDS bytes of one W stage (fp8)
constexpr int kBuf = kA + kW + 4 * kTileM + 4 * kTileN;
constexpr int kLds = 2 * kBuf;

static_assert(kTileM == 2 * kWM && kTileN == 4 * kWN, "8 waves as 2 x 4 quadrants");

// LDS layout of one stage buffer: A (kTileM rows x 128 B), W (kTileN rows x
// 128 B), then the tile's fp32 activation scales (times 2^18) and weight
// scales.  Row r's 16-byte chunk c sits at r*128 + ((c ^ g(r)) << 4) with
// g(r) = (r ^ (r >> 1)) & 7.  With this swizzle the 16 rows of one MFMA
// operand fetch (ds_read_b128) are bank-conflict free on gfx950 (measured:
// the plain c ^ (r & 7) swizzle runs at 60% of the read bandwidth).
__device__ __forceinline__ int swz(int r, int c) { return r * 128 + ((c ^ ((r ^ (r >> 1)) & 7)) << 4); }

__device__ __forceinline__ i32x8 lds_frag(const uint8_t* p0, const uint8_t* p1) {
  const u32x4 x = *reinterpret_cast<const u32x4*>(p0);
  const u32x4 y = *reinterpret_cast<const u32x4*>(p1);
  i32x8 f;
  f[0] = (int)x[0]; f[1] = (int)x[1]; f[2] = (int)x[2]; f[3] = (int)x[3];
  f[4] = (int)y[0]; f[5] = (int)y[1]; f[6] = (int)y[2]; f[7] = (int)y[3];
  return f;
}

// Per-lane LDS offsets, fixed for the whole kernel.  Fragment reads of row
// block rb (column block cb) add rb*2048 (cb*2048): 16 rows of 128 bytes, and
// the swizzle term depends only on the row's low 4 bits, which do not change.
struct LaneOffsets {
  int fa0, fa1;   // A fragment chunks (2*q4, 2*q4+1) of row wr + r16
  int fw0, fw1;   // W fragment chunks of row wc + r16
};

__device__ __forceinline__ LaneOffsets lane_offsets() {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r16 = lane & 15, q4 = lane >> 4;
  const int wr = (wave >> 2) * kWM, wc = (wave & 3) * kWN;
  LaneOffsets o;
  o.fa0 = swz(wr + r16, 2 * q4);
  o.fa1 = swz(wr + r16, 2 * q4 + 1);
  o.fw0 = kA + swz(wc + r16, 2 * q4);
  o.fw1 = kA + swz(wc + r16, 2 * q4 + 1);
  (void)tid;
  return o;
}

// One K-block position of the schedule, decoded from the host's encoding:
// bits 0..9 block index g, bit 10 set for an 8-bit activation block, bits
// 11.. the block's offset in A_packed in units of M*64 bytes.
struct KBlock {
  int g;
  bool b8;
  int aoff;
};

__device__ __forceinline__ KBlock kblock(int e) { return KBlock{e & 1023, ((e >> 10) & 1) != 0, e >> 11}; }

// Registers holding one K-block's packed operands between load and LDS store.
struct Stage {
  u32x4 a[4];
  u32x4 w[2];
  uint32_t s;
};

// Global loads of one K-block's packed operands for the tile at (m0, n0).
// Rows and columns are clamped into range, so edge tiles never read out of
// bounds; clamped rows and columns compute values that are never stored.
__device__ __forceinline__ void stage_load(const GemmArgs& p, const KBlock& kb, int m0, int n0,
                                           Stage& st) {
  const int tid = threadIdx.x;
  const uint8_t* A = p.A + (size_t)p.M * 64 * (size_t)kb.aoff;
  // 4-bit block: lane chunk tid%4 of rows tid/4 + 128 i (i < 2), 64 bytes a row;
  // 8-bit block: lane chunk tid%8 of rows tid/8 + 64 i (i < 4), 128 bytes a row.
  // The first two loads only switch offsets (arithmetic select, so that the
  // staging registers are not forced into memory by a branch merge).
  const uint32_t b8 = kb.b8 ? 1u : 0u;
  #pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int r = b8 ? (tid >> 3) + 64 * i : (tid >> 2) + 128 * i;
    const uint32_t row = (uint32_t)min(m0 + r, p.M - 1);
    const uint32_t off = (row << (6 + b8)) + ((uint32_t)tid & (3u | (b8 << 2))) * 16u;
    st.a[i] = *reinterpret_cast<const u32x4*>(A + off);
  }
  if (kb.b8) {
    #pragma unroll
    for (int i = 2; i < 4; ++i) {
      const uint32_t row = (uint32_t)min(m0 + (tid >> 3) + 64 * i, p.M - 1);
      st.a[i] = *reinterpret_cast<const u32x4*>(A + row * 128u + (tid & 7) * 16u);
    }
  }
  const uint8_t* W = p.W + (size_t)kb.g * 64;
  #pragma unroll
  for (int i = 0; i < 2; ++i) {
    const uint32_t col = (uint32_t)min(n0 + (tid >> 2) + 128 * i, p.N - 1);
    st.w[i] = *reinterpret_cast<const u32x4*>(W + col * (uint32_t)(p.K / 2) + (tid & 3) * 16u);
  }
  if (tid < kTileM)
    st.s = p.sa[(size_t)kb.g * p.M + min(m0 + tid, p.M - 1)];
  else
    st.s = p.sw[(size_t)kb.g * p.N + min(n0 + tid - kTileM, p.N - 1)];
}

__device__ __forceinline__ void stage_store(const Stage& st, bool b8, uint8_t* buf) {
  const int tid = threadIdx.x;
  const int st4a = swz(tid >> 2, 2 * (tid & 3)), st4b = swz(tid >> 2, 2 * (tid & 3) + 1);
  const int st8 = swz(tid >> 3, tid & 7);
  if (!b8) {
    #pragma unroll
    for (int i = 0; i < 2; ++i) {
      u32x4 lo, hi;
      unpack4(st.a[i], lo, hi);
      *reinterpret_cast<u32x4*>(buf + st4a + i * 16384) = lo;
      *reinterpret_cast<u32x4*>(buf + st4b + i * 16384) = hi;
    }
  } else {
    #pragma unroll
    for (int i = 0; i < 4; ++i) *reinterpret_cast<u32x4*>(buf + st8 + i * 8192) = st.a[i];
  }
  #pragma unroll
  for (int i = 0; i < 2; ++i) {
    u32x4 lo, hi;
    unpack4(st.w[i], lo, hi);
    *reinterpret_cast<u32x4*>(buf + kA + st4a + i * 16384) = lo;
    *reinterpret_cast<u32x4*>(buf + kA + st4b + i * 16384) = hi;
  }
  // Scales, permuted so that each lane later reads its values with one or two
  // 16-byte LDS reads.  Activation scale of tile row r = 128h + 16rb + 4j + i
  // goes to (16h + 4j + i) * 8 + rb (the 8 row blocks of one 4x4x1 operand
  // lane); weight scale of tile column c = 64q + 16cb + x to
  // kTileM + (16q + x) * 4 + cb.
  const float f = __half2float(__ushort_as_half((unsigned short)st.s));
  float* scales = reinterpret_cast<float*>(buf + kA + kW);
  if (tid < kTileM) {
    const int r = tid, h = r >> 7, rb = (r >> 4) & 7, j = (r >> 2) & 3, i = r & 3;
    scales[(16 * h + 4 * j + i) * 8 + rb] = f * kUnit;
  } else {
    const int c = tid - kTileM, q = c >> 6, cb = (c >> 4) & 3, x = c & 15;
    scales[kTileM + (16 * q + x) * 4 + cb] = f;
  }
}

template <bool DIAG, bool B8>
__device__ __forceinline__ void compute_block(const uint8_t* buf, const LaneOffsets& o, int g, int NG,
                                              int m0, int n0, const GemmArgs& p,
                                              f32x4 (&C)[kRB][kCB]) {
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int r16 = lane & 15, q4 = lane >> 4;
  const int wr = (wave >> 2) * kWM;
  const int wc = (wave & 3) * kWN;
  // this lane's 4x4x1 operands: activation scale of row wr + 16rb + 4*q4 + (lane & 3)
  // for every rb, weight scale of column wc + 16cb + r16 for every cb
  const float* scales = reinterpret_cast<const float*>(buf + kA + kW);
  const float* sal = scales + (16 * (wave >> 2) + 4 * q4 + (lane & 3)) * 8;
  const f32x4 swl = *reinterpret_cast<const f32x4*>(scales + kTileM + (16 * (wave & 3) + r16) * 4);

  i32x8 wf[kCB];
  #pragma unroll
  for (int cb = 0; cb < kCB; ++cb) wf[cb] = lds_frag(buf + o.fw0 + cb * 2048, buf + o.fw1 + cb * 2048);
  // the A fragment and activation scale of row block rb + 1 are fetched while
  // row block rb computes
  i32x8 an = lds_frag(buf + o.fa0, buf + o.fa1);
  float san = sal[0];
  #pragma unroll
  for (int rb = 0; rb < kRB; ++rb) {
    i32x8 af = an;
    const float sa_rb = san;
    if (rb + 1 < kRB) {
      an = lds_frag(buf + o.fa0 + (rb + 1) * 2048, buf + o.fa1 + (rb + 1) * 2048);
      san = sal[rb + 1];
    }
    i32x8 ah;
    if constexpr (B8) {
      #pragma unroll
      for (int i = 0; i < 8; ++i) {
        ah[i] = (int)hi8((uint32_t)af[i]);
        af[i] = (int)lo8((uint32_t)af[i]);
      }
    }
    #pragma unroll
    for (int cb = 0; cb < kCB; ++cb) {
      f32x4 y = mfma_fp8(af, wf[cb], f32x4{0.f, 0.f, 0.f, 0.f});
      if constexpr (B8) {
        const f32x4 yh = mfma_fp8(ah, wf[cb], f32x4{0.f, 0.f, 0.f, 0.f});
        #pragma unroll
        for (int i = 0; i < 4; ++i) y[i] = __builtin_fmaf(yh[i], 8.0f, y[i]);  // exact
      }
      if constexpr (DIAG) {
        const int col = n0 + wc + cb * 16 + r16;
        #pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int row = m0 + wr + rb * 16 + 4 * q4 + i;
          if (row >= p.win_m0 && row < p.win_m1 && col >= p.win_n0 && col < p.win_n1) {
            const size_t idx = ((size_t)(row - p.win_m0) * (p.win_n1 - p.win_n0) +
                                (col - p.win_n0)) * NG + g;
            p.acc[idx] = (int32_t)(y[i] * kUnit);
          }
        }
      } else {
        const f32x4 P = scale_products(sa_rb, swl[cb]);
        #pragma unroll
        for (int i = 0; i < 4; ++i) C[rb][cb][i] = __builtin_fmaf(y[i], P[i], C[rb][cb][i]);
      }
    }
    // Pin this row block's accumulator updates here.  Without it the
    // optimizer sinks the FMAs past the barrier into the next K-block, keeping
    // all 32 MFMA results of the K-block live at once (and spilling them).
    if constexpr (!DIAG)
      asm volatile("" : "+v"(C[rb][0]), "+v"(C[rb][1]), "+v"(C[rb][2]), "+v"(C[rb][3]));
  }
}

// Pipelined K-loop over schedule positions [pos, end), all of precision B8:
// K-block k is computed from one LDS buffer while k+1 (whatever its
// precision) is loaded into registers and then stored to the other buffer.
template <bool DIAG, bool B8>
__device__ __forceinline__ void kloop(const GemmArgs& p, const LaneOffsets& o,
                                      uint8_t* smem, int g_begin, int pos,
                                      int end, int g_end, int NG, int m0, int n0, Stage& st,
                                      f32x4 (&C)[kRB][kCB]) {
  for (; pos < end; ++pos) {
    const int cur = (pos - g_begin) & 1;
    const bool more = pos + 1 < g_end;
    const KBlock kb = kblock(p.order[pos]);
    const KBlock kn = kblock(p.order[more ? pos + 1 : pos]);
    if (more) stage_load(p, kn, m0, n0, st);
    compute_block<DIAG, B8>(smem + cur * kBuf, o, kb.g, NG, m0, n0, p, C);
    if (more) stage_store(st, kn.b8, smem + (cur ^ 1) * kBuf);
    __syncthreads();
  }
}

template <bool DIAG>
__global__ __launch_bounds__(kThreads) void gemm_kernel(GemmArgs p) {
  extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
  __shared__ int s_last;
  const int NG = p.K / kG;
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int r16 = lane & 15, q4 = lane >> 4;
  const LaneOffsets o = lane_offsets();
  const int u_end = p.wg_begin[blockIdx.x + 1];

  for (int u = p.wg_begin[blockIdx.x]; u < u_end; ++u) {
    const WorkUnit unit = p.units[u];
    const int tm = unit.tile / p.tiles_n, tn = unit.tile % p.tiles_n;
    const int m0 = tm * kTileM, n0 = tn * kTileN;

    f32x4 C[kRB][kCB];
    #pragma unroll
    for (int i = 0; i < kRB; ++i)
      #pragma unroll
      for (int j = 0; j < kCB; ++j) C[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    // software pipeline over the unit's K-blocks; the schedule lists all
    // 4-bit blocks before the 8-bit ones, so each precision runs its own loop
    Stage st;
    const KBlock k0 = kblock(p.order[unit.g_begin]);
    stage_load(p, k0, m0, n0, st);
    stage_store(st, k0.b8, smem);
    __syncthreads();
    const int split = min(max(p.n4, unit.g_begin), unit.g_end);
    kloop<DIAG, false>(p, o, smem, unit.g_begin, unit.g_begin, split, unit.g_end, NG, m0, n0,
                       st, C);
    kloop<DIAG, true>(p, o, smem, unit.g_begin, split, unit.g_end, unit.g_end, NG, m0, n0, st,
                      C);
    if (DIAG) continue;

    const int wr = (wave >> 2) * kWM, wc = (wave & 3) * kWN;
    if (unit.nslots > 1) {
      // split tile: publish this slot's partial, then the last arriver reduces
      const int base = p.split_index[unit.tile];
      float* part = p.partials + (size_t)(base + unit.slot) * (kTileM * kTileN);
      #pragma unroll
      for (int rb = 0; rb < kRB; ++rb)
        #pragma unroll
        for (int cb = 0; cb < kCB; ++cb)
          *reinterpret_cast<f32x4*>(part + (((wave * kRB + rb) * kCB + cb) * 64 + lane) * 4) =
              C[rb][cb];
      __threadfence();
      __syncthreads();
      if (threadIdx.x == 0) s_last = atomicAdd(p.counters + base, 1) == unit.nslots - 1;
      __syncthreads();
      if (!s_last) continue;
      __threadfence();
      #pragma unroll
      for (int rb = 0; rb < kRB; ++rb)
        #pragma unroll
        for (int cb = 0; cb < kCB; ++cb) C[rb][cb] = f32x4{0.f, 0.f, 0.f, 0.f};
      for (int s = 0; s < unit.nslots; ++s) {
        const float* src = p.partials + (size_t)(base + s) * (kTileM * kTileN);
        #pragma unroll
        for (int rb = 0; rb < kRB; ++rb) {
          #pragma unroll
          for (int cb = 0; cb < kCB; ++cb)
            C[rb][cb] += *reinterpret_cast<const f32x4*>(
                src + (((wave * kRB + rb) * kCB + cb) * 64 + lane) * 4);
          __builtin_amdgcn_sched_barrier(0);
        }
      }
      if (threadIdx.x == 0) p.counters[base] = 0;  // ready for the next launch
    }
    #pragma unroll
    for (int rb = 0; rb < kRB; ++rb)
      #pragma unroll
      for (int cb = 0; cb < kCB; ++cb) {
        const int col = n0 + wc + cb * 16 + r16;
        #pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int row = m0 + wr + rb * 16 + 4 * q4 + i;
          if (row < p.M && col < p.N)
            p.out[(size_t)row * p.N + col] = __half_as_ushort(__float2half_rn(C[rb][cb][i]));
        }
      }
  }
}

}  // namespace

int gemm_lds_bytes() { return kLds; }

hipError_t launch_gemm(const GemmArgs& a, int num_wgs, bool diag, hipStream_t stream) {
  if (diag)
    hipLaunchKernelGGL(gemm_kernel<true>, dim3(num_wgs), dim3(kThreads), kLds, stream, a);
  else
    hipLaunchKernelGGL(gemm_kernel<false>, dim3(num_wgs), dim3(kThreads), kLds, stream, a);
  return hipGetLastError();
}

hipError_t set_gemm_attributes() {
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&gemm_kernel<false>),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, kLds);
  if (e != hipSuccess) return e;
  return hipFuncSetAttribute(reinterpret_cast<const void*>(&gemm_kernel<true>),
                             hipFuncAttributeMaxDynamicSharedMemorySize, kLds);
}

}  // namespace comet
