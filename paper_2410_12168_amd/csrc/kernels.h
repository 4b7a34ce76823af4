// kernels.h -- internal launchers of libcomet's gfx950 kernels (not part of
// the public C ABI; see include/comet.h for that).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace comet {

constexpr int kG = 128;          // block size along K (the paper's k = 128)
constexpr int kMaxBlocks = 512;  // blocks per row supported by the bit map (K <= 65536)
constexpr int kOrderPad = 16;    // entries after the K-block order that repeat its last entry

// Precision of every K-block as a bit set (bit g = 1: block g is 8-bit),
// passed by value as a kernel argument so no device table is needed.
struct BlockMap {
  uint64_t bits[kMaxBlocks / 64];
};

// One unit of GEMM work: blocks [g_begin, g_end) (positions in the schedule's
// block order) of output tile `tile`, written as partial `slot` of `nslots`.
struct WorkUnit {
  int tile;
  int g_begin;
  int g_end;
  int slot;
  int nslots;
};

struct GemmArgs {
  const uint8_t* A;
  const uint16_t* sa;
  const uint8_t* W;
  const uint16_t* sw;
  uint16_t* out;
  int32_t* acc;       // diagnostic window output (or null)
  float* partials;    // split-tile fp32 partials [tile slot][TM*TN]
  int* counters;      // per split tile arrival counters (zero between launches)
  const WorkUnit* units;
  const int* wg_begin;
  const int* order;   // K-block schedule, K/G (+ kOrderPad) entries: g | is8 << 10 | (g + 8-bit blocks before g) << 11
  int n4;             // number of 4-bit blocks (they come first in `order`, except in natural order)
  const int* split_index;  // tile -> index into the partial/counter arrays (-1: not split)
  int M, N, K;
  int tiles_n;        // tiles along N
  int cus;            // compute units of the device
  int splits;         // split-K slots per column block (few-token kernel)
  int win_m0, win_m1, win_n0, win_n1;
  BlockMap map;
  // SwiGLU epilogue (tile and mid kernels): h of tile column block j goes,
  // quantized with out_map, to block j of out_A (block-major, M rows) and
  // out_sa [N/256][M]; nothing is written to `out`
  uint8_t* out_A;
  uint16_t* out_sa;
  BlockMap out_map;
};

// perm == nullptr: no channel permutation.
hipError_t launch_quantize_act(const uint16_t* X, const int32_t* perm, uint8_t* A, uint16_t* sa,
                               int M, int K, const BlockMap& map, hipStream_t stream);
hipError_t launch_pack_w4(const uint16_t* W, const int32_t* perm, uint8_t* Wp, uint16_t* sw,
                          int N, int K, hipStream_t stream);
hipError_t launch_channel_absmax(const uint16_t* X, float* absmax, int M, int K,
                                 hipStream_t stream);
// Host: calibration map and channel permutation from per-channel maxima.
// Returns nullptr on success, else a message.
const char* plan_channel_perm(const float* absmax, int K, int G, float ratio, float max_frac8,
                              int32_t* perm, uint8_t* prec, int* n_outliers);
// KV4 group quantizer; G in {32, 64, 128}.
hipError_t launch_kv4_quantize(const uint16_t* X, uint8_t* codes, uint16_t* params, int T, int C,
                               int G, hipStream_t stream);
hipError_t launch_kv4_dequantize(const uint8_t* codes, const uint16_t* params, uint16_t* out,
                                 int T, int C, int G, hipStream_t stream);

// Output tile of one GEMM workgroup: kTileN columns and kTileM or
// kTileMSmall rows (comet::choose_tile_m decides from the shape).
constexpr int kTileM = 256;
constexpr int kTileMSmall = 128;
constexpr int kTileN = 256;

// Persistent GEMM: `num_wgs` workgroups walk a.units (a.wg_begin per group);
// tile_m is the plan's tile height; swiglu selects the SwiGLU + quantize epilogue;
// natural: the plan's K order is the map's own (not precision-batched), which
// the SwiGLU epilogue does not support.
hipError_t launch_gemm(const GemmArgs& a, int num_wgs, bool diag, bool swiglu, bool natural,
                       int tile_m, hipStream_t stream);
// SwiGLU of an fp16 gate/up output GU [M][2I] (2G-wide gate/up column groups)
// and FMPQ quantization of h [M][I] with `map` into A / sa [I/G][M].
hipError_t launch_swiglu_quantize(const uint16_t* GU, uint8_t* A, uint16_t* sa, int M, int I,
                                  const BlockMap& map, hipStream_t stream);
// Few-token kernels.  When the 16-column panels divide evenly over the CUs
// (skinny_stream_eligible), persistent stream kernels whose workgroups own
// whole panels: for M <= 8 the waves stream contiguous runs of W_packed; for
// 8 < M <= 64 the K-blocks go in chunks whose activation fragments are staged
// in LDS.  Otherwise (M <= kSkinnyMaxM) one wave per (16 columns, split-K
// slot), or, for 8 < M <= 32 with at most two slots, four column blocks per
// workgroup sharing the activation operand through LDS.
constexpr int kSkinnyMaxM = 48;
constexpr int kStreamMaxLds = 160 * 1024;
bool skinny_stream_eligible(int M, int N, int K, int cus);
inline bool skinny_shared(int M, int splits) { return M > 8 && M <= 32 && splits <= 2; }
hipError_t launch_gemm_skinny(const GemmArgs& a, bool diag, hipStream_t stream);
// Allows the stream kernels' dynamic LDS size; once per process and device.
hipError_t set_skinny_attributes();
// Split-K slots (1, 2 or 4) for the few-token kernel: spread the (N/16 x
// slots) waves evenly over the device's SIMDs, keeping at least 4 K-blocks per
// slot.
int skinny_splits(int N, int K, int cus);

// Fixed per-device workspace of the no-allocation GEMM entry point:
// [fp32 split partials][split arrival counters][plan], in one static device
// array (noalloc.hip).  64 MiB of partials holds the split plans of the
// LLaMA-3 shapes (256 slots of a 256 x 256 tile); 2 MiB of plan holds about
// 87,000 tiles (six ints per tile).
constexpr size_t kNoallocPartialBytes = size_t(64) << 20;
constexpr size_t kNoallocCounterBytes = size_t(64) << 10;
constexpr size_t kNoallocPlanBytes = size_t(2) << 20;
constexpr size_t kNoallocBytes = kNoallocPartialBytes + kNoallocCounterBytes + kNoallocPlanBytes;
// Device address of the current device `dev`'s workspace (looked up once per
// device, with that device current).
hipError_t noalloc_scratch(int dev, uint8_t** ptr);
hipError_t launch_zero_ints(int* p, int n, hipStream_t stream);

// Allows the GEMM's dynamic LDS size; once per process and device.
hipError_t set_gemm_attributes();
int gemm_lds_bytes(int tile_m);

}  // namespace comet
