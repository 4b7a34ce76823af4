// gemm.hip -- W4Ax mixed-precision GEMM for gfx950 (paper Sec. 4).
//
// Operand path.  Both operands arrive as sign-magnitude codes.  A 4-bit chunk
// becomes FP8-E4M3 subnormal bytes (code * 2^-9) with two masks and one
// rotate per 8 codes; an 8-bit activation byte (sign, 7-bit magnitude m)
// becomes two such FP8 bytes, hi = m >> 3 (0..15) and lo = m & 7, so that
// code = 8 * hi + lo.  Each 16x16 output block of one K-block is one
// v_mfma_f32_16x16x128_f8f6f4 (K = 128 = one block) for W4A4 and two for
// W4A8, the second (hi) chained on the first's result with an E8M0 block
// scale of 2^3 on A.  Products of such codes are integers times 2^-18 and
// their sums stay below 2^24 units, so the fp32 MFMA result is the exact
// block sum (the paper's integer tile result, Sec. 4.1) and needs no
// int->float convert.
// Dequantization (Sec. 4.3: the scale absorbs the conversion factor) runs on
// the vector ALUs, once per output and K-block:
//     C += Y * P,   P = (sa * 2^18) * sw      (fp32; sa * sw is exact),
// two VALU operations per output and K-block: as much vector work as the
// MFMAs have matrix work.  Each step's dequantization is issued one step
// late, behind the next step's MFMA, so it never waits for an MFMA result.
//
// Kernel structure (the gfx950 form of the paper's software pipeline,
// Sec. 4.2, and of its tile decomposition, Sec. 4.4):
//   * persistent workgroups of 8 waves walk a host-built list of work units
//     (tile, K-block range); full tiles go to one workgroup, the fractional
//     last wave of tiles is split over all of them by cost;
//   * the tile's packed 4-bit weights stream HBM -> LDS with direct
//     (register-free) 128-bit loads into a ring of three K-block slots,
//     issued two K-blocks ahead by waves 4-7; each wave unpacks the weight
//     fragments it uses when it reads them;
//   * the tile's activation codes stream HBM -> LDS one K-block ahead with
//     direct loads by waves 0-3, which then unpack 4-bit codes once per
//     workgroup into a double-buffered stage of FP8 bytes (XOR swizzled
//     rows); 8-bit codes land in the stage directly.  Waves 0-3 also stage
//     both scale vectors.  Waves 0-3 win issue arbitration over the waves
//     that share their SIMDs, so their extra work runs while waves 4-7 finish
//     computing;
//   * one barrier per K-block separates the stages;
//   * each wave computes a 128x64 quadrant: 8x4 MFMA blocks per K-block;
//   * split tiles write fp32 partials; the last workgroup to finish a tile
//     (arrival counter, no waiting) adds the partials in slot order and
//     stores fp16, so the result does not depend on arrival order.
#include <hip/hip_runtime.h>
#include <hip/hip_fp16.h>
#include <stdint.h>

#include "fmpq.h"
#include "kernels.h"
#include "operand.h"
#include "swiglu.h"

namespace comet {

namespace {

constexpr int kThreads = 512;            // 8 waves
constexpr int kWN = 64;                  // wave quadrant width
constexpr int kCB = kWN / 16;
constexpr int kWr = kTileN * 64;          // one packed weight K-block, ring of three
static_assert(kTileN == 4 * kWN, "8 waves as 2 x 4 quadrants");

// Geometry of a tile of TM rows (TM = 256, or 128: for 64 < M <= 128, where a
// 256-row tile would leave half of every MFMA idle, and for larger M where
// comet::choose_tile_m finds 128-row tiles faster): 8 waves as 2 x 4
// quadrants of (TM / 2) x 64.
template <int TM>
struct Geo {
  static constexpr int WM = TM / 2;                // wave quadrant rows
  static constexpr int RB = WM / 16;               // row blocks per wave
  static constexpr int A = TM * 128;               // LDS bytes of one A stage (fp8 or raw 8-bit codes)
  static constexpr int S = 4 * (TM + kTileN);      // LDS bytes of one stage's scales (fp32)
  static constexpr int Buf = A + S;                // one activation stage, double-buffered
  static constexpr int Raw = TM * 64;              // packed 4-bit codes of the next K-block
  static constexpr int Lds = 2 * Buf + 3 * kWr + Raw;
  static_assert(TM == 256 || TM == 128, "tile heights");
  static_assert(TM * 136 * 2 <= Lds, "SwiGLU epilogue buffer fits in LDS");
};

// LDS layout of one activation stage: A (TM rows x 128 B), then the
// tile's fp32 activation scales (times 2^18) and weight scales.  Row r's
// 16-byte chunk c sits at r*128 + ((c ^ g(r)) << 4) with g(r) = (r ^ (r >> 1))
// & 7.  With this swizzle the 16 rows of one MFMA operand fetch
// (ds_read_b128) are bank-conflict free on gfx950 (measured: the plain
// c ^ (r & 7) swizzle runs at 60% of the read bandwidth).
__device__ __forceinline__ int swz(int r, int c) { return r * 128 + ((c ^ ((r ^ (r >> 1)) & 7)) << 4); }

// Packed weights in a ring slot: one kilobyte per 16-column panel (one
// K-block of it), chunk-major inside: tile column c's 16-byte chunk j (32
// codes) at (c / 16) * 1024 + (16 j + c % 16) * 16.  A fragment read (lane
// r16 + 16 q4 takes chunk q4 of column r16 of a panel) is then one linear
// kilobyte, free of bank conflicts on gfx950 (measured: a column-major panel
// with swizzled chunks read at 60% of the LDS bandwidth).
__device__ __forceinline__ int wpos(int c, int j) { return (c >> 4) * 1024 + ((j << 4) + (c & 15)) * 16; }

// Scales of one stage (floats after the A codes): the activation scale of
// tile row r at r, so a lane's four rows 4 j .. 4 j + 3 of a row block are one
// 16-byte read; the weight scale of tile column c = 64 q + 16 cb + x at
// TM + (16 q + x) * 4 + cb, so a lane's column in all four column blocks is
// one 16-byte read.
template <int TM>
__device__ __forceinline__ int sw_slot(int c) {
  return TM + (16 * (c >> 6) + (c & 15)) * 4 + ((c >> 4) & 3);
}

__device__ __forceinline__ i32x8 lds_frag(const uint8_t* p0, const uint8_t* p1) {
  const u32x4 x = *reinterpret_cast<const u32x4*>(p0);
  const u32x4 y = *reinterpret_cast<const u32x4*>(p1);
  i32x8 f;
  f[0] = (int)x[0]; f[1] = (int)x[1]; f[2] = (int)x[2]; f[3] = (int)x[3];
  f[4] = (int)y[0]; f[5] = (int)y[1]; f[6] = (int)y[2]; f[7] = (int)y[3];
  return f;
}

// Per-lane LDS offsets, fixed for the whole kernel.  Fragment reads of row
// block rb add rb*2048 (16 rows of 128 bytes; the swizzle term depends only on
// the row's low 4 bits, which do not change), of column block cb cb*1024 (one
// weight panel).
struct LaneOffsets {
  int fa0, fa1;   // A fragment chunks (2*q4, 2*q4+1) of row wr + r16
  int fw;         // packed weight chunk q4 of column wc + r16 (in a ring slot)
};

template <int TM>
__device__ __forceinline__ LaneOffsets lane_offsets() {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r16 = lane & 15, q4 = lane >> 4;
  const int wr = (wave >> 2) * Geo<TM>::WM, wc = (wave & 3) * kWN;
  LaneOffsets o;
  o.fa0 = swz(wr + r16, 2 * q4);
  o.fa1 = swz(wr + r16, 2 * q4 + 1);
  o.fw = wpos(wc + r16, q4);
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

// End of the run of K-blocks of equal precision that starts at schedule
// position pos (an LDS copy of the order; the run ends at `end` at the
// latest).  The precision-batched order has two runs, 4-bit then 8-bit; the
// natural order has as many as the map.
__device__ __forceinline__ int run_end(const int* order, int pos, int end) {
  const int b = __builtin_amdgcn_readfirstlane(order[pos]) & 1024;
  int e = pos + 1;
  while (e < end && (__builtin_amdgcn_readfirstlane(order[e]) & 1024) == b) ++e;
  return e;
}

// The plan (schedule, work units, split table) is read-only while the kernel
// runs.  Reading it through the constant address space keeps its loads on the
// scalar unit: a vector load here would come with a wait on the vector-memory
// counter, which also waits for every weight load in flight.
typedef const __attribute__((address_space(4))) int* cint_ptr;
__device__ __forceinline__ int plan_at(const int* a, int i) {
  return ((cint_ptr)a)[i];
}
__device__ __forceinline__ int order_at(const GemmArgs& p, int i) { return plan_at(p.order, i); }

// Registers holding one K-block's activation codes and a scale between load
// and LDS store (the mid-size kernel's activation waves).
struct Stage {
  u32x4 a[4];
  uint32_t s;
};

// Direct global -> LDS load of 16 bytes per lane: the wave's 64 chunks land
// at LDS bytes lds .. lds + 1023, lane by lane.  Issued as inline assembly so
// that the compiler does not wait for it at LDS reads of other ring slots;
// the K-loop waits for it explicitly before the barrier that publishes it.
__device__ __forceinline__ void dma16(const void* g, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off"
               :: "v"(g), "s"(lds) : "memory", "m0");
}
// The same with the non-temporal hint, for data used once (the mid-size
// kernel's weights): it does not displace the activation codes, which every
// workgroup reads, from L2.
__device__ __forceinline__ void dma16nt(const void* g, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off nt"
               :: "v"(g), "s"(lds) : "memory", "m0");
}

// Source of one 1 KB wave load of packed weights: K-block g of the 16-column
// panel j of the tile at n0 (one contiguous kilobyte of W_packed).  Lane L
// fills the ring layout's position L * 16 of the panel: chunk L / 16 of the
// panel's column L % 16.  Panels past N are clamped (their outputs are never
// stored).
__device__ __forceinline__ const uint8_t* w_src(const GemmArgs& p, int g, int n0, int j) {
  const int lane = threadIdx.x & 63;
  const int NG = p.K / kG;
  const int panel = min(n0 / 16 + j, p.N / 16 - 1);
  return p.W + ((size_t)panel * NG + g) * 1024 + (lane & 15) * 64 + (lane >> 4) * 16;
}

// Direct load with a scalar base and a 32-bit per-lane byte offset.
__device__ __forceinline__ void dma16s(const uint8_t* base, uint32_t voff, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1"
               :: "v"(voff), "s"(base), "s"(lds) : "m0");
}

// Weight loads of waves 4-7: wave 4 + w loads panels 4 w .. 4 w + 3 of the
// tile (clamped to the last panel past N).  Per tile, the panels' bases;
// per lane, the source offset of its ring position within a 1 KB K-block
// (the ring layout of wpos(): column lane % 16, chunk lane / 16).
struct WPanels {
  const uint8_t* b[4];
};
__device__ __forceinline__ WPanels w_panels(const GemmArgs& p, int n0) {
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6) - 4;
  const int NG = p.K / kG;
  WPanels wp;
  #pragma unroll
  for (int i = 0; i < 4; ++i)
    wp.b[i] = p.W + (size_t)min(n0 / 16 + 4 * w + i, p.N / 16 - 1) * NG * 1024;
  return wp;
}
__device__ __forceinline__ uint32_t w_lane_off() {
  const int lane = threadIdx.x & 63;
  return (lane & 15) * 64 + (lane >> 4) * 16;
}

// Packed weights of K-block g for the tile's 256 columns into a ring slot:
// 16 KB, four 1 KB wave loads by each of waves 4-7.
__device__ __forceinline__ void dma_w(const WPanels& wp, uint32_t voff, int g, uint32_t slot) {
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6) - 4;
  #pragma unroll
  for (int i = 0; i < 4; ++i) dma16s(wp.b[i] + (size_t)g * 1024, voff, slot + (4 * w + i) * 1024);
}

// Activation codes of K-block kb for the tile's 256 rows, by waves 0-3 (wave
// w: rows 64 w .. 64 w + 63), straight into LDS.  A 4-bit block lands packed
// in the raw slot (row r at r * 64), to be unpacked by act_unpack; an 8-bit
// block lands in activation stage `stage` in its final swizzled layout (LDS
// chunk slot s of row r holds code chunk s ^ g(r)).  Rows past M re-read row
// M - 1.
// Load i (i < 4) of a 4-bit block: rows 64 w + 16 i .. + 15.  A is the block's
// base; byte offsets within a block stay below 2^32 (at most 2^21 rows of
// 128 bytes).
__device__ __forceinline__ void act_dma4(const uint8_t* A, int M, int m0, int i, uint32_t raw) {
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int r = 64 * wave + 16 * i + (lane >> 2);
  const uint32_t off = (uint32_t)min(m0 + r, M - 1) * 64u + (lane & 3) * 16u;
  dma16s(A, off, raw + (4 * wave + i) * 1024);
}
// Load i (i < 8) of an 8-bit block: rows 64 w + 8 i .. + 7.
__device__ __forceinline__ void act_dma8(const uint8_t* A, int M, int m0, int i, uint32_t stage) {
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int r = 64 * wave + 8 * i + (lane >> 3);
  const int c = (lane & 7) ^ ((r ^ (r >> 1)) & 7);
  const uint32_t off = (uint32_t)min(m0 + r, M - 1) * 128u + c * 16u;
  dma16s(A, off, stage + (8 * wave + i) * 1024);
}
// Loads of a tile that lies inside M (m0 + 256 <= M): no row is clamped, so a
// load is a scalar base and a per-lane constant.  4-bit load i of wave w
// covers rows 64 w + 16 i .. + 15 (lane offset lane * 16); 8-bit load i rows
// 64 w + 8 i .. + 7, whose swizzle depends on i only through i & 1 (lane
// offsets a8[0], a8[1]).
struct ActLane {
  uint32_t a4, a8[2];
};
__device__ __forceinline__ ActLane act_lane() {
  const int lane = threadIdx.x & 63;
  ActLane l;
  l.a4 = lane * 16;
  #pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int r = 8 * h + (lane >> 3);  // row modulo 16
    l.a8[h] = (lane >> 3) * 128 + (((lane & 7) ^ ((r ^ (r >> 1)) & 7)) << 4);
  }
  return l;
}
__device__ __forceinline__ void act_dma4_in(const uint8_t* A, int m0, int i, const ActLane& l,
                                            uint32_t raw) {
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  dma16s(A + (size_t)(m0 + 64 * wave) * 64 + i * 1024, l.a4, raw + (4 * wave + i) * 1024);
}
__device__ __forceinline__ void act_dma8_in(const uint8_t* A, int m0, int i, const ActLane& l,
                                            uint32_t stage) {
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  dma16s(A + (size_t)(m0 + 64 * wave) * 128 + i * 1024, l.a8[i & 1],
         stage + (8 * wave + i) * 1024);
}

__device__ __forceinline__ void act_dma(const GemmArgs& p, const KBlock& kb, int m0, uint32_t raw,
                                        uint32_t stage) {
  const uint8_t* A = p.A + (size_t)p.M * 64 * (size_t)kb.aoff;
  if (!kb.b8) {
    #pragma unroll
    for (int i = 0; i < 4; ++i) act_dma4(A, p.M, m0, i, raw);
  } else {
    #pragma unroll
    for (int i = 0; i < 8; ++i) act_dma8(A, p.M, m0, i, stage);
  }
}

// Waves 0-3: unpack the 4-bit codes that this wave loaded into the raw slot
// into activation stage `buf` (FP8 bytes, swizzled rows).
__device__ __forceinline__ void act_unpack(const uint8_t* raw, uint8_t* buf) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  // all four reads first: one LDS round trip instead of four
  u32x4 v[4];
  #pragma unroll
  for (int i = 0; i < 4; ++i)
    v[i] = *reinterpret_cast<const u32x4*>(raw + (4 * wave + i) * 1024 + lane * 16);
  #pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int r = 64 * wave + 16 * i + (lane >> 2), c = lane & 3;
    u32x4 lo, hi;
    unpack4(v[i], lo, hi);
    *reinterpret_cast<u32x4*>(buf + swz(r, 2 * c)) = lo;
    *reinterpret_cast<u32x4*>(buf + swz(r, 2 * c + 1)) = hi;
  }
}

// Waves 0-3 (thread t): the fp16 scales of tile row t and tile column t for
// K-block g, loaded ahead into registers and stored as fp32 into a stage.
struct StageScales {
  uint32_t sa, sw;  // zero-extended fp16 bits, kept apart so that no wait is forced at the load
};
__device__ __forceinline__ StageScales scales_load(const GemmArgs& p, int g, int m0, int n0) {
  const int t = threadIdx.x;
  return StageScales{(uint32_t)p.sa[(size_t)g * p.M + min(m0 + t, p.M - 1)],
                     (uint32_t)p.sw[(size_t)g * p.N + min(n0 + t, p.N - 1)]};
}
template <int TM>
__device__ __forceinline__ void scales_store(StageScales sc, uint8_t* buf) {
  const int t = threadIdx.x;
  float* scales = reinterpret_cast<float*>(buf + Geo<TM>::A);
  scales[t] = __half2float(__ushort_as_half((unsigned short)sc.sa)) * kUnit;
  scales[sw_slot<TM>(t)] = __half2float(__ushort_as_half((unsigned short)sc.sw));
}

__device__ __forceinline__ void wait_vm_all() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

// Barrier that publishes this wave's LDS writes (ds_write completion) but
// leaves its outstanding global loads in flight.
__device__ __forceinline__ void barrier_lds() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// 16 bytes of 4-bit codes (32 channels) -> one MFMA operand of 32 FP8 bytes.
__device__ __forceinline__ i32x8 unpack_frag(u32x4 v) {
  i32x8 f;
  #pragma unroll
  for (int i = 0; i < 4; ++i) {
    f[2 * i] = (int)(v[i] & kSignMag);
    f[2 * i + 1] = (int)(rotr4(v[i]) & kSignMag);
  }
  return f;
}

// The lane's weight scales (column wc + 16 cb + r16, cb < 4) from an
// activation stage's fp32 scale table.
template <int TM>
__device__ __forceinline__ f32x4 stage_sw(const uint8_t* buf) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const float* scales = reinterpret_cast<const float*>(buf + Geo<TM>::A);
  return *reinterpret_cast<const f32x4*>(scales + TM + (16 * (wave & 3) + (lane & 15)) * 4);
}

// One K-block of the wave's quadrant: activation stage `buf` (fp8 or raw
// 8-bit codes, then activation scales), packed weights in ring slot `wbuf`,
// the lane's weight scales in swl.
struct NoHook {
  __device__ void operator()(int) const {}
};

// hook(s) runs after the MFMA issue of step s (s < RB * 4): loads spread over
// the K-block instead of issued in one burst.
template <int TM, bool DIAG, bool B8, class Hook = NoHook>
__device__ __forceinline__ void compute_block(const uint8_t* buf, const uint8_t* wbuf, f32x4 swl,
                                              const LaneOffsets& o, int g, int NG, int m0, int n0,
                                              const GemmArgs& p,
                                              f32x4 (&C)[Geo<TM>::RB][kCB],
                                              Hook&& hook = NoHook()) {
  constexpr int kRB = Geo<TM>::RB;
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int r16 = lane & 15, q4 = lane >> 4;
  const int wr = (wave >> 2) * Geo<TM>::WM;
  const int wc = (wave & 3) * kWN;
  // this lane's rows wr + 16 rb + 4 q4 + i (i < 4) and column wc + 16 cb + r16
  const float* scales = reinterpret_cast<const float*>(buf + Geo<TM>::A);
  const float* sal = scales + wr + 4 * q4;  // + 16 rb

  i32x8 wf[kCB];
  #pragma unroll
  for (int cb = 0; cb < kCB; ++cb)
    wf[cb] = unpack_frag(*reinterpret_cast<const u32x4*>(wbuf + o.fw + cb * 1024));
  // the A fragment and activation scales of row block rb + 1 are fetched
  // while row block rb computes
  i32x8 af = lds_frag(buf + o.fa0, buf + o.fa1);
  f32x4 san = *reinterpret_cast<const f32x4*>(sal);
  i32x8 ah;
  f32x4 sa_rb = san;
  // Step s = (rb, cb).  The dequantization of step s - 1 is issued after the
  // MFMA of step s, so the vector ALU works while the matrix core does.
  f32x4 yq = {0.f, 0.f, 0.f, 0.f}, pq = {0.f, 0.f, 0.f, 0.f};
  #pragma unroll
  for (int s = 0; s < kRB * kCB; ++s) {
    const int rb = s / kCB, cb = s % kCB;
    if (cb == 0) {
      sa_rb = san;
      if (rb + 1 < kRB) san = *reinterpret_cast<const f32x4*>(sal + (rb + 1) * 16);
      if constexpr (B8) {
        #pragma unroll
        for (int i = 0; i < 8; ++i) {
          ah[i] = (int)hi8((uint32_t)af[i]);
          af[i] = (int)lo8((uint32_t)af[i]);
        }
      }
    }
    f32x4 y = mfma_fp8(af, wf[cb], f32x4{0.f, 0.f, 0.f, 0.f});
    if constexpr (B8) y = mfma_fp8_x8(ah, wf[cb], y);  // + 8 * hi, exact
    hook(s);
    if (cb == kCB - 1 && rb + 1 < kRB) {
      // the next row block's fragment replaces this one in the same registers
      __builtin_amdgcn_sched_barrier(0);
      af = lds_frag(buf + o.fa0 + (rb + 1) * 2048, buf + o.fa1 + (rb + 1) * 2048);
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
      const f32x4 P = sa_rb * swl[cb];  // exact: 11-bit by 11-bit significands
      if (s > 0) {
        const int pr = (s - 1) / kCB, pc = (s - 1) % kCB;
        #pragma unroll
        for (int i = 0; i < 4; ++i) C[pr][pc][i] = __builtin_fmaf(yq[i], pq[i], C[pr][pc][i]);
        // pin each row block's updates here; otherwise the optimizer sinks
        // the FMAs past the barrier and keeps all the K-block's MFMA results
        // live at once
        if (pc == kCB - 1)
          asm volatile("" : "+v"(C[pr][0]), "+v"(C[pr][1]), "+v"(C[pr][2]), "+v"(C[pr][3]));
      }
      yq = y;
      pq = P;
    }
  }
  if constexpr (!DIAG) {
    #pragma unroll
    for (int i = 0; i < 4; ++i)
      C[kRB - 1][kCB - 1][i] = __builtin_fmaf(yq[i], pq[i], C[kRB - 1][kCB - 1][i]);
    asm volatile("" : "+v"(C[kRB - 1][0]), "+v"(C[kRB - 1][1]), "+v"(C[kRB - 1][2]),
                 "+v"(C[kRB - 1][3]));
  }
}

// Pipelined K-loop over schedule positions [pos, end), all of precision B8.
// Relative position j = pos - g_begin computes from activation stage j % 2
// and weight ring slot j % 3.  The waves split the loads by role:
//   * waves 0-3 load the scales of j + 1 and start the direct loads of its
//     activation codes (into the raw slot, or for an 8-bit block into stage
//     (j + 1) % 2, read last at j - 1), compute j, then wait for their own
//     loads and unpack the codes into stage (j + 1) % 2.  They are the waves
//     that win issue arbitration, so this work runs while waves 4-7 still
//     compute;
//   * waves 4-7 start the direct loads of the weights of j + 2 into ring slot
//     (j + 2) % 3 (read last at j - 1), compute j, and wait only for the
//     weights of j + 1 (loads complete in order: at most the four of j + 2
//     stay in flight).
// The direct loads are issued a few MFMA steps into the K-block, those of
// waves 4-7 one step before those of waves 0-3: issued at the top all at once
// they queue for the memory pipeline, and the waves wait for the issue with
// idle matrix cores.  Tiles that cross M (clamped rows) issue their activation
// loads at the top.  One barrier per K-block publishes the stage and the
// weights.
template <int TM, bool DIAG, bool B8>
__device__ __forceinline__ void kloop(const GemmArgs& p, const LaneOffsets& o, uint8_t* smem,
                                      uint32_t lds, const int* order, int g_begin, int pos,
                                      int end, int g_end, int NG, int m0, int n0,
                                      const WPanels& wp, uint32_t wvoff,
                                      f32x4 (&C)[Geo<TM>::RB][kCB]) {
  constexpr int kBuf = Geo<TM>::Buf, kRaw = 2 * kBuf + 3 * kWr;
  const bool awave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6) < 4;
  const bool inside = m0 + TM <= p.M;
  const ActLane al = act_lane();
  // schedule entries of pos, pos + 1 and pos + 2 (clamped to the unit),
  // each read from the LDS copy one K-block ahead
  int e0 = order[pos], e1 = order[min(pos + 1, g_end - 1)], e2 = order[min(pos + 2, g_end - 1)];
  for (; pos < end; ++pos) {
    const int j = pos - g_begin;
    const int cur = j & 1, wslot = j % 3;
    const bool more = pos + 1 < g_end, wnext = pos + 2 < g_end;
    const KBlock kb = kblock(__builtin_amdgcn_readfirstlane(e0));
    const KBlock kn = kblock(__builtin_amdgcn_readfirstlane(e1));
    const int g2 = kblock(__builtin_amdgcn_readfirstlane(e2)).g;
    StageScales sc;
    const int e3 = order[min(pos + 3, g_end - 1)];
    const uint8_t* Anext = p.A + (size_t)p.M * 64 * (size_t)kn.aoff;
    const uint32_t wdst = lds + 2 * kBuf + (wslot == 0 ? 2 : wslot - 1) * kWr;  // slot (j + 2) % 3
    if (awave && more) {
      sc = scales_load(p, kn.g, m0, n0);
      if (!inside) act_dma(p, kn, m0, lds + kRaw, lds + (cur ^ 1) * kBuf);
    }
    auto hook = [&](int s) {
      if (s == 1 && !awave && wnext) dma_w(wp, wvoff, g2, wdst);
      if (s == 2 && awave && more && inside) {
        if (!kn.b8) {
          #pragma unroll
          for (int i = 0; i < 4; ++i) act_dma4_in(Anext, m0, i, al, lds + kRaw);
        } else {
          #pragma unroll
          for (int i = 0; i < 8; ++i) act_dma8_in(Anext, m0, i, al, lds + (cur ^ 1) * kBuf);
        }
      }
    };
    compute_block<TM, DIAG, B8>(smem + cur * kBuf, smem + 2 * kBuf + wslot * kWr,
                                stage_sw<TM>(smem + cur * kBuf), o, kb.g, NG, m0, n0, p, C, hook);
    if (awave) {
      if (more) {
        wait_vm_all();
        if (!kn.b8) act_unpack(smem + kRaw, smem + (cur ^ 1) * kBuf);
        scales_store<TM>(sc, smem + (cur ^ 1) * kBuf);
      }
    } else if (wnext) {
      asm volatile("s_waitcnt vmcnt(4)" ::: "memory");
    } else {
      wait_vm_all();
    }
    e0 = e1;
    e1 = e2;
    e2 = e3;
    barrier_lds();
  }
}

// Epilogue of a work unit: a whole tile is stored as fp16; a split tile
// publishes this slot's fp32 partial, and the last workgroup to arrive adds
// the partials in slot order and stores fp16.
// SwiGLU epilogue (the step after the path, fused): the tile's columns 0-127
// are the gate and 128-255 the up outputs of channels 128 j .. 128 j + 127
// (j = n0 / 256).  The up waves put fp16(up) into LDS, the gate waves turn
// each entry into h = SiLU(fp16(gate)) * up (fp16), and then 16 lanes per row
// quantize the row's 128 channels of h as the activation quantizer does,
// into block j of the next layer's A_packed.  `lds` is free by now.
template <int TM>
__device__ __forceinline__ void swiglu_tile(const GemmArgs& p, int m0, int n0,
                                            f32x4 (&C)[Geo<TM>::RB][kCB], uint8_t* lds) {
  constexpr int kRB = Geo<TM>::RB;
  constexpr int kHP = 136;  // row pitch in halves: 128 channels + 16 bytes
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int r16 = lane & 15, q4 = lane >> 4;
  const int wr = (wave >> 2) * Geo<TM>::WM, wq = wave & 3;
  uint16_t* H = reinterpret_cast<uint16_t*>(lds);
  __syncthreads();
  if (wq >= 2) {
    #pragma unroll
    for (int rb = 0; rb < kRB; ++rb)
      #pragma unroll
      for (int cb = 0; cb < kCB; ++cb)
        #pragma unroll
        for (int i = 0; i < 4; ++i)
          H[(wr + rb * 16 + 4 * q4 + i) * kHP + (wq - 2) * 64 + cb * 16 + r16] =
              __half_as_ushort(__float2half_rn(C[rb][cb][i]));
  }
  __syncthreads();
  if (wq < 2) {
    #pragma unroll
    for (int rb = 0; rb < kRB; ++rb)
      #pragma unroll
      for (int cb = 0; cb < kCB; ++cb)
        #pragma unroll
        for (int i = 0; i < 4; ++i) {
          uint16_t* h = H + (wr + rb * 16 + 4 * q4 + i) * kHP + wq * 64 + cb * 16 + r16;
          *h = swiglu_f16(__half_as_ushort(__float2half_rn(C[rb][cb][i])), *h);
        }
  }
  __syncthreads();
  const int j = n0 / kTileN;
  const bool b8 = (p.out_map.bits[j >> 6] >> (j & 63)) & 1;
  const size_t base = (size_t)p.M * 64 * (size_t)(j + n8_before(p.out_map, j));
  const int lane16 = threadIdx.x & 15;
  for (int r = threadIdx.x >> 4; r < TM; r += kThreads / 16) {
    float x[8];
    load8(H + r * kHP + 8 * lane16, x);
    float a = 0.0f;
    #pragma unroll
    for (int i = 0; i < 8; ++i) a = fmaxf(a, fabsf(x[i]));
    a = max16(a);
    Codes c;
    const uint16_t s16 = quantize8(x, a, b8 ? 127.0f : 7.0f, c);
    const int m = m0 + r;
    if (m >= p.M) continue;
    if (b8)
      *reinterpret_cast<uint2*>(p.out_A + base + (size_t)m * 128 + 8 * lane16) = pack8(c);
    else
      *reinterpret_cast<uint32_t*>(p.out_A + base + (size_t)m * 64 + 4 * lane16) = pack4(c);
    if (lane16 == 0) p.out_sa[(size_t)j * p.M + m] = s16;
  }
}

template <int TM, bool SWIGLU>
__device__ __forceinline__ void store_tile(const GemmArgs& p, const WorkUnit& unit, int m0, int n0,
                                           f32x4 (&C)[Geo<TM>::RB][kCB], int* s_last,
                                           uint8_t* lds) {
  constexpr int kRB = Geo<TM>::RB;
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int r16 = lane & 15, q4 = lane >> 4;
  const int wr = (wave >> 2) * Geo<TM>::WM, wc = (wave & 3) * kWN;
  if (unit.nslots > 1) {
    // Split tile.  Each slot publishes its fp32 partial and counts in;
    // whichever counts in last adds the partials in slot order.  A tile of
    // two slots needs only the other slot's partial: the plan puts the
    // first slot early in its workgroup's list and the second at the end, so
    // the second usually finds the first arrived and then skips publishing
    // its own.  One device-scope release and one acquire per tile slot, by
    // one thread: on this multi-XCD part each is a write-back or invalidate
    // of the whole L2, too costly to issue from every wave.
    const int base = plan_at(p.split_index, unit.tile);
    const bool pair = unit.nslots == 2;
    if (threadIdx.x == 0) {
      *s_last = pair && __hip_atomic_load(p.counters + base, __ATOMIC_RELAXED,
                                          __HIP_MEMORY_SCOPE_AGENT) == 1;
      if (*s_last) __threadfence();  // acquire the other slot's partial
    }
    __syncthreads();
    if (!*s_last) {
      float* part = p.partials + (size_t)(base + unit.slot) * (TM * kTileN);
      #pragma unroll
      for (int rb = 0; rb < kRB; ++rb)
        #pragma unroll
        for (int cb = 0; cb < kCB; ++cb)
          *reinterpret_cast<f32x4*>(part + (((wave * kRB + rb) * kCB + cb) * 64 + lane) * 4) =
              C[rb][cb];
      // the barrier completes every wave's partial stores into L2
      __syncthreads();
      if (threadIdx.x == 0) {
        __threadfence();
        const bool last = atomicAdd(p.counters + base, 1) == unit.nslots - 1;
        if (last) __threadfence();
        *s_last = last;
      }
      __syncthreads();
      if (!*s_last) return;
    }
    // A pair adds the other slot's partial to its registers (two terms: the
    // same sum whichever slot adds it); otherwise all partials in slot order.
    const int s_first = pair ? unit.slot ^ 1 : 0;
    const int s_end = pair ? s_first + 1 : unit.nslots;
    if (!pair) {
      #pragma unroll
      for (int rb = 0; rb < kRB; ++rb)
        #pragma unroll
        for (int cb = 0; cb < kCB; ++cb) C[rb][cb] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
    for (int s = s_first; s < s_end; ++s) {
      const float* src = p.partials + (size_t)(base + s) * (TM * kTileN);
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
  if constexpr (SWIGLU) {
    swiglu_tile<TM>(p, m0, n0, C, lds);
    return;
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

// NAT: the schedule lists the K-blocks in the map's own order (the ablation
// baseline without tile remapping); otherwise all 4-bit blocks come first.
template <int TM, bool DIAG, bool SWIGLU, bool NAT>
__global__ __launch_bounds__(kThreads) void gemm_kernel(GemmArgs p) {
  constexpr int kRB = Geo<TM>::RB, kBuf = Geo<TM>::Buf;
  extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
  __shared__ int s_last;
  __shared__ int s_order[kMaxBlocks];
  const int NG = p.K / kG;
  const LaneOffsets o = lane_offsets<TM>();
  const uint32_t lds = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)smem);
  const int u_end = plan_at(p.wg_begin, blockIdx.x + 1);
  for (int i = threadIdx.x; i < NG; i += kThreads) s_order[i] = p.order[i];
  __syncthreads();
  const uint32_t wvoff = w_lane_off();

  const bool awave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6) < 4;
  // The unit whose first K-block loads are in flight: they are issued before
  // the previous unit's epilogue, so their latency overlaps its stores.
  WorkUnit unit{};
  int m0 = 0, n0 = 0;
  KBlock k0{};
  WPanels wp{};
  StageScales sc{};
  auto issue = [&](int uu) {
    const int* ue = reinterpret_cast<const int*>(p.units) + 5 * uu;
    unit = WorkUnit{plan_at(ue, 0), plan_at(ue, 1), plan_at(ue, 2), plan_at(ue, 3),
                    plan_at(ue, 4)};
    m0 = (unit.tile / p.tiles_n) * TM;
    n0 = (unit.tile % p.tiles_n) * kTileN;
    k0 = kblock(order_at(p, unit.g_begin));
    wp = w_panels(p, n0);
    if (awave) {
      act_dma(p, k0, m0, lds + 2 * kBuf + 3 * kWr, lds);
      sc = scales_load(p, k0.g, m0, n0);
    } else {
      dma_w(wp, wvoff, k0.g, lds + 2 * kBuf);
      if (unit.g_begin + 1 < unit.g_end)
        dma_w(wp, wvoff, kblock(order_at(p, unit.g_begin + 1)).g, lds + 2 * kBuf + kWr);
    }
  };
  int u = plan_at(p.wg_begin, blockIdx.x);
  if (u < u_end) issue(u);
  for (; u < u_end; ++u) {
    // the unit's first K-block in place (and its second's weights in flight)
    if (awave) {
      wait_vm_all();
      if (!k0.b8) act_unpack(smem + 2 * kBuf + 3 * kWr, smem);
      scales_store<TM>(sc, smem);
    } else if (unit.g_begin + 1 < unit.g_end) {
      asm volatile("s_waitcnt vmcnt(4)" ::: "memory");
    } else {
      wait_vm_all();
    }
    barrier_lds();

    f32x4 C[kRB][kCB];
    #pragma unroll
    for (int i = 0; i < kRB; ++i)
      #pragma unroll
      for (int j = 0; j < kCB; ++j) C[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    // software pipeline over the unit's K-blocks; the schedule lists all
    // 4-bit blocks before the 8-bit ones, so each precision runs its own loop
    if constexpr (NAT) {
      // natural order: one K-loop per run of equal precision, the loads
      // running on across runs
      for (int pos = unit.g_begin; pos < unit.g_end;) {
        const int end = run_end(s_order, pos, unit.g_end);
        if (s_order[pos] & 1024)
          kloop<TM, DIAG, true>(p, o, smem, lds, s_order, unit.g_begin, pos, end, unit.g_end, NG,
                                m0, n0, wp, wvoff, C);
        else
          kloop<TM, DIAG, false>(p, o, smem, lds, s_order, unit.g_begin, pos, end, unit.g_end,
                                 NG, m0, n0, wp, wvoff, C);
        pos = end;
      }
    } else {
      // precision-batched order: the 4-bit run, then the 8-bit run, as two
      // straight-line loops (a loop over runs holding both bodies makes the
      // register allocator spill)
      const int split = min(max(p.n4, unit.g_begin), unit.g_end);
      if (unit.g_begin < split)
        kloop<TM, DIAG, false>(p, o, smem, lds, s_order, unit.g_begin, unit.g_begin, split,
                               unit.g_end, NG, m0, n0, wp, wvoff, C);
      if (split < unit.g_end)
        kloop<TM, DIAG, true>(p, o, smem, lds, s_order, unit.g_begin, split, unit.g_end,
                              unit.g_end, NG, m0, n0, wp, wvoff, C);
    }
    const WorkUnit cur = unit;
    const int cm0 = m0, cn0 = n0;
    if (u + 1 < u_end) issue(u + 1);  // LDS is free: the K-loop ended on a barrier
    if (DIAG) continue;

    store_tile<TM, SWIGLU>(p, cur, cm0, cn0, C, &s_last, smem);
  }
}


// ---------------------------------------------------------------------------
// Mid-size GEMM: 128-row tiles (up to 128 rows, and above where
// comet::choose_tile_m finds them faster), with the workgroup's waves split
// by role so that no load is waited for early.  With this few rows the
// weights come from HBM exactly once and a K-block computes briefly, so the
// loads need several K-blocks of lead, and a wait on the vector-memory counter
// covers every older load of the wave:
//   * waves 0-3 stage the activation codes and scales (few rows, written just
//     before by the quantizer, so they come from L2) through registers one
//     K-block ahead, unpack 4-bit codes once and store them to a
//     double-buffered LDS stage.  They win issue arbitration over the waves
//     sharing their SIMDs, so this extra work runs while waves 4-7 still
//     compute (as in the tile kernel; with the roles the other way round the
//     kernel ran 2-6% slower);
//   * waves 4-7 only issue direct loads: a K-block's packed weights and its
//     fp16 weight scales, into a ring of four slots three K-blocks ahead, and
//     wait for them with counted waits;
//   * all eight waves compute their 64 x 64 quadrant with the tile kernel's
//     K-block step.
// As in the tile kernel, both roles issue their loads a few MFMA steps into
// the K-block (not in a burst at its top), and the K-block order is read
// from an LDS copy.
constexpr int kMidTM = 128;
constexpr int kMidD = 4;                                // weight ring slots
constexpr int kMidSlot = kWr + 2 * kTileN;              // packed weights + fp16 weight scales
constexpr int kMidStage = Geo<kMidTM>::A + 4 * kMidTM;  // codes + fp32 activation scales
constexpr int kMidLds = 2 * kMidStage + kMidD * kMidSlot;
static_assert(kMidTM * 136 * 2 <= kMidLds, "SwiGLU epilogue buffer fits in the mid kernel's LDS");
constexpr int kMidVm = 5;  // direct loads per K-block and weight wave

// Waves 4-7 (w = wave - 4): packed weights of K-block g (16 KB, four 1 KB
// loads per wave, in the ring layout of wpos()) and the fp16 scales of the
// slot's 256 columns (lanes 0-7 of each wave: columns n0 + 64 w + 8 lane
// .. + 7, at byte kWr + 2 * (column - n0)).  Columns past N re-read the last
// valid ones.
__device__ __forceinline__ void mid_dma(const GemmArgs& p, int g, int n0, uint32_t slot) {
  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6) & 3;
  #pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int j = 4 * w + i;
    dma16nt(w_src(p, g, n0, j), slot + j * 1024);
  }
  const int c0 = min(n0 + 64 * w + 8 * (lane & 7), p.N - 8);
  if (lane < 8) dma16(p.sw + (size_t)g * p.N + c0, slot + kWr + 128 * w);
}

// Wait until at most n of this wave's direct loads are in flight (n = 0, 5
// or 10: the loads of the next zero, one or two K-blocks).
__device__ __forceinline__ void mid_wait(int n) {
  if (n >= 2 * kMidVm)
    asm volatile("s_waitcnt vmcnt(10)" ::: "memory");
  else if (n >= kMidVm)
    asm volatile("s_waitcnt vmcnt(5)" ::: "memory");
  else
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
}

// The lane's weight scales (column wc + 16 cb + r16, cb < 4) from a ring slot.
__device__ __forceinline__ f32x4 slot_sw(const uint8_t* slot) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const uint16_t* sw =
      reinterpret_cast<const uint16_t*>(slot + kWr) + 64 * (wave & 3) + (lane & 15);
  return f32x4{__half2float(__ushort_as_half(sw[0])), __half2float(__ushort_as_half(sw[16])),
               __half2float(__ushort_as_half(sw[32])), __half2float(__ushort_as_half(sw[48]))};
}

// Waves 0-3 (t = threadIdx.x): one K-block's activation codes and scale.
// 4-bit block: chunk t % 4 of rows t / 4 + 64 i (i < 2); 8-bit block: chunk
// t % 8 of rows t / 8 + 32 i (i < 4).  Rows past M are clamped.
__device__ __forceinline__ void mid_load(const GemmArgs& p, const KBlock& kb, int m0, Stage& st) {
  const int t = threadIdx.x;
  const uint8_t* A = p.A + (size_t)p.M * 64 * (size_t)kb.aoff;
  const uint32_t b8 = kb.b8 ? 1u : 0u;
  #pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int r = b8 ? (t >> 3) + 32 * i : (t >> 2) + 64 * i;
    const uint32_t row = (uint32_t)min(m0 + r, p.M - 1);
    const uint32_t off = (row << (6 + b8)) + ((uint32_t)t & (3u | (b8 << 2))) * 16u;
    st.a[i] = *reinterpret_cast<const u32x4*>(A + off);
  }
  if (kb.b8) {
    #pragma unroll
    for (int i = 2; i < 4; ++i) {
      const uint32_t row = (uint32_t)min(m0 + (t >> 3) + 32 * i, p.M - 1);
      st.a[i] = *reinterpret_cast<const u32x4*>(A + row * 128u + (t & 7) * 16u);
    }
  }
  st.s = p.sa[(size_t)kb.g * p.M + min(m0 + (t & (kMidTM - 1)), p.M - 1)];
}

__device__ __forceinline__ void mid_store(const Stage& st, bool b8, uint8_t* buf) {
  const int t = threadIdx.x;
  if (!b8) {
    const int r = t >> 2, c = t & 3;
    #pragma unroll
    for (int i = 0; i < 2; ++i) {
      u32x4 lo, hi;
      unpack4(st.a[i], lo, hi);
      *reinterpret_cast<u32x4*>(buf + swz(r, 2 * c) + i * 8192) = lo;
      *reinterpret_cast<u32x4*>(buf + swz(r, 2 * c + 1) + i * 8192) = hi;
    }
  } else {
    const int off = swz(t >> 3, t & 7);
    #pragma unroll
    for (int i = 0; i < 4; ++i) *reinterpret_cast<u32x4*>(buf + off + i * 4096) = st.a[i];
  }
  if (t < kMidTM)
    reinterpret_cast<float*>(buf + Geo<kMidTM>::A)[t] =
        __half2float(__ushort_as_half((unsigned short)st.s)) * kUnit;
}

// One K-block position of the mid-size loop: weights of pos + 3 issued after
// MFMA step 2, activations of pos + 1 loaded after step 3 and stored to the
// other stage after the compute.
template <bool DIAG, bool B8>
__device__ __forceinline__ void mid_loop(const GemmArgs& p, const LaneOffsets& o, uint8_t* smem,
                                         uint32_t lds, const int* order, int pos, int end, int gb,
                                         int ge, int NG, int m0, int n0, Stage& st,
                                         f32x4 (&C)[Geo<kMidTM>::RB][kCB]) {
  const bool wwave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6) >= 4;
  for (; pos < end; ++pos) {
    const int j = pos - gb;
    const KBlock kb = kblock(__builtin_amdgcn_readfirstlane(order[pos]));
    const bool more = pos + 1 < ge;
    const KBlock kn = kblock(__builtin_amdgcn_readfirstlane(order[more ? pos + 1 : pos]));
    const int g3 = kblock(__builtin_amdgcn_readfirstlane(order[min(pos + 3, ge - 1)])).g;
    const uint8_t* slot = smem + 2 * kMidStage + (j & 3) * kMidSlot;
    auto hook = [&](int s) {
      if (s == 2 && wwave && pos + 3 < ge)
        mid_dma(p, g3, n0, lds + 2 * kMidStage + ((j + 3) & 3) * kMidSlot);
      if (s == 3 && !wwave && more) mid_load(p, kn, m0, st);
    };
    compute_block<kMidTM, DIAG, B8>(smem + (j & 1) * kMidStage, slot, slot_sw(slot), o, kb.g, NG,
                                    m0, n0, p, C, hook);
    if (wwave)
      mid_wait(kMidVm * min(max(ge - pos - 2, 0), 2));
    else if (more)
      mid_store(st, kn.b8, smem + ((j + 1) & 1) * kMidStage);
    barrier_lds();
  }
}

template <bool DIAG, bool SWIGLU, bool NAT>
__global__ __launch_bounds__(kThreads) void gemm_mid_kernel(GemmArgs p) {
  constexpr int TM = kMidTM, kRB = Geo<TM>::RB;
  extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
  __shared__ int s_last;
  __shared__ int s_order[kMaxBlocks];
  const int NG = p.K / kG;
  const LaneOffsets o = lane_offsets<TM>();
  const uint32_t lds = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)smem);
  const bool wwave = threadIdx.x >= 256;
  const int u_end = plan_at(p.wg_begin, blockIdx.x + 1);
  for (int i = threadIdx.x; i < NG; i += kThreads) s_order[i] = p.order[i];
  __syncthreads();

  for (int u = plan_at(p.wg_begin, blockIdx.x); u < u_end; ++u) {
    const int* ue = reinterpret_cast<const int*>(p.units) + 5 * u;
    const WorkUnit unit{plan_at(ue, 0), plan_at(ue, 1), plan_at(ue, 2), plan_at(ue, 3),
                        plan_at(ue, 4)};
    const int tm = unit.tile / p.tiles_n, tn = unit.tile % p.tiles_n;
    const int m0 = tm * TM, n0 = tn * kTileN;
    const int gb = unit.g_begin, ge = unit.g_end;

    f32x4 C[kRB][kCB];
    #pragma unroll
    for (int i = 0; i < kRB; ++i)
      #pragma unroll
      for (int j = 0; j < kCB; ++j) C[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    // prologue: weights of the first three K-blocks in flight, activations
    // of the first stored
    Stage st;
    if (wwave) {
      for (int d = 0; d < 3 && gb + d < ge; ++d)
        mid_dma(p, kblock(order_at(p, gb + d)).g, n0, lds + 2 * kMidStage + d * kMidSlot);
      mid_wait(kMidVm * min(ge - gb - 1, 2));
    } else {
      const KBlock k0 = kblock(order_at(p, gb));
      mid_load(p, k0, m0, st);
      mid_store(st, k0.b8, smem);
    }
    barrier_lds();
    if constexpr (NAT) {
      for (int pos = gb; pos < ge;) {
        const int end = run_end(s_order, pos, ge);
        if (s_order[pos] & 1024)
          mid_loop<DIAG, true>(p, o, smem, lds, s_order, pos, end, gb, ge, NG, m0, n0, st, C);
        else
          mid_loop<DIAG, false>(p, o, smem, lds, s_order, pos, end, gb, ge, NG, m0, n0, st, C);
        pos = end;
      }
    } else {
      const int split = min(max(p.n4, gb), ge);
      if (gb < split)
        mid_loop<DIAG, false>(p, o, smem, lds, s_order, gb, split, gb, ge, NG, m0, n0, st, C);
      if (split < ge)
        mid_loop<DIAG, true>(p, o, smem, lds, s_order, split, ge, gb, ge, NG, m0, n0, st, C);
    }
    if (DIAG) continue;

    store_tile<TM, SWIGLU>(p, unit, m0, n0, C, &s_last, smem);
  }
}

typedef void (*GemmKernelFn)(GemmArgs);

// The instantiations: production (plain, diagnostic; the SwiGLU epilogue for
// the 128-row kernel only) and the natural-order ablation (plain,
// diagnostic), for both tile heights.  nullptr: not instantiated.
GemmKernelFn gemm_kernel_fn(int tile_m, bool diag, bool swiglu, bool natural) {
  if (tile_m == kMidTM) {
    if (natural) return diag ? gemm_mid_kernel<true, false, true> : gemm_mid_kernel<false, false, true>;
    if (diag) return gemm_mid_kernel<true, false, false>;
    return swiglu ? gemm_mid_kernel<false, true, false> : gemm_mid_kernel<false, false, false>;
  }
  if (natural) return diag ? gemm_kernel<256, true, false, true> : gemm_kernel<256, false, false, true>;
  if (swiglu) return nullptr;  // the 256-row kernel's SwiGLU runs as its own kernel
  return diag ? gemm_kernel<256, true, false, false> : gemm_kernel<256, false, false, false>;
}

}  // namespace

int gemm_lds_bytes(int tile_m) { return tile_m == kMidTM ? kMidLds : Geo<256>::Lds; }

hipError_t launch_gemm(const GemmArgs& a, int num_wgs, bool diag, bool swiglu, bool natural,
                       int tile_m, hipStream_t stream) {
  const dim3 grid(num_wgs), block(kThreads);
  const GemmKernelFn fn = swiglu && natural ? nullptr : gemm_kernel_fn(tile_m, diag, swiglu, natural);
  if (!fn) return hipErrorInvalidValue;  // not instantiated
  const int lds = tile_m == kMidTM ? kMidLds : Geo<256>::Lds;
  hipLaunchKernelGGL(fn, grid, block, lds, stream, a);
  return hipGetLastError();
}

hipError_t set_gemm_attributes() {
  for (int tm : {256, kMidTM})
    for (int v = 0; v < 5; ++v) {
      const bool diag = v == 1 || v == 4, swiglu = v == 2, natural = v >= 3;
      const GemmKernelFn fn = gemm_kernel_fn(tm, diag, swiglu, natural);
      if (!fn) continue;
      hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(fn),
                                         hipFuncAttributeMaxDynamicSharedMemorySize,
                                         tm == kMidTM ? kMidLds : Geo<256>::Lds);
      if (e != hipSuccess) return e;
    }
  return hipSuccess;
}

}  // namespace comet
