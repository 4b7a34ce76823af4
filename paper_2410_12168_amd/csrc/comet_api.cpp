// comet_api.cpp -- the C ABI of libcomet (include/comet.h): argument checks,
// device checks, plan cache and kernel launches.  Every step of the path runs
// in the HIP kernels; this file only validates, plans and enqueues.
#include <hip/hip_runtime.h>

#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <algorithm>
#include <cstring>
#include <map>
#include <mutex>
#include <string>
#include <tuple>
#include <vector>

#include "../../include/comet.h"
#include "kernels.h"
#include "scheduler.h"

#ifndef COMET_SOURCE_STAMP
#define COMET_SOURCE_STAMP "unstamped"
#endif

namespace {

// The build's source stamp, kept as one string so that a loader can find it
// in the library file without loading it.
const char kStamp[] = "COMET_SOURCE_STAMP=" COMET_SOURCE_STAMP;

thread_local std::string g_last_error;

comet_status_t fail(comet_status_t st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return st;
}

comet_status_t ok() {
  g_last_error.clear();
  return COMET_OK;
}

// Above this many rows the 128-row tile kernel takes over from the few-token
// kernel when its 256-column tiles cover at least 3/4 of the CUs (wide N).
constexpr int kSkinnyWideM = 32;

// The activation quantizer's grid has one row of workgroups per 32 tokens.
constexpr int kMaxQuantRows = 65535 * 32;

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// Checks shared by every entry point: G, K and the block map.
comet_status_t check_kg(int K, int G) {
  if (G != comet::kG) return fail(COMET_ERR_UNSUPPORTED, "G=%d: only G=128 is supported", G);
  if (K < G || K % G) return fail(COMET_ERR_INVALID_ARG, "K=%d must be a positive multiple of G", K);
  if (K / G > comet::kMaxBlocks)
    return fail(COMET_ERR_UNSUPPORTED, "K=%d exceeds %d", K, comet::kMaxBlocks * comet::kG);
  return COMET_OK;
}

comet_status_t make_map(const uint8_t* prec, int NG, comet::BlockMap* map) {
  if (!prec) return fail(COMET_ERR_INVALID_ARG, "group_prec_map is null");
  std::memset(map, 0, sizeof *map);
  for (int g = 0; g < NG; ++g) {
    if (prec[g] == 8)
      map->bits[g >> 6] |= 1ull << (g & 63);
    else if (prec[g] != 4)
      return fail(COMET_ERR_INVALID_ARG, "group_prec_map[%d]=%d is not 4 or 8", g, (int)prec[g]);
  }
  return COMET_OK;
}

struct DeviceInfo {
  bool gfx950 = false;
  int cus = 0;
};

std::mutex g_mu;
std::map<int, DeviceInfo> g_devices;

// Current device, checked to be gfx950.  COMET_TEST_FORCE_ARCH replaces the
// reported architecture name (used by the CPU tests of this check).
comet_status_t current_device(int* dev, DeviceInfo* info) {
  const char* forced = std::getenv("COMET_TEST_FORCE_ARCH");
  if (forced && *forced) {
    if (std::strncmp(forced, "gfx950", 6) != 0)
      return fail(COMET_ERR_UNSUPPORTED, "device architecture %s is not gfx950", forced);
  }
  hipError_t e = hipGetDevice(dev);
  if (e != hipSuccess) return fail(COMET_ERR_HIP, "hipGetDevice: %s", hipGetErrorString(e));
  std::lock_guard<std::mutex> lk(g_mu);
  auto it = g_devices.find(*dev);
  if (it == g_devices.end()) {
    hipDeviceProp_t prop;
    e = hipGetDeviceProperties(&prop, *dev);
    if (e != hipSuccess)
      return fail(COMET_ERR_HIP, "hipGetDeviceProperties: %s", hipGetErrorString(e));
    DeviceInfo di;
    di.gfx950 = std::strncmp(prop.gcnArchName, "gfx950", 6) == 0;
    di.cus = prop.multiProcessorCount;
    it = g_devices.emplace(*dev, di).first;
  }
  *info = it->second;
  if (!info->gfx950) return fail(COMET_ERR_UNSUPPORTED, "current device is not gfx950");
  return COMET_OK;
}

comet_status_t launched(hipError_t e, const char* what) {
  if (e != hipSuccess) return fail(COMET_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
  return ok();
}

comet_status_t gemm_common(const uint8_t* A, const uint8_t* prec, const uint16_t* sa,
                                  const uint8_t* W, const uint16_t* sw, void* out, int M, int N,
                                  int K, int G, comet::BlockMap* map) {
  if (!A || !sa || !W || !sw || !out) return fail(COMET_ERR_INVALID_ARG, "null pointer");
  if (M < 1 || N < 1) return fail(COMET_ERR_INVALID_ARG, "M=%d, N=%d must be >= 1", M, N);
  // the kernels address rows within one activation block with 32-bit offsets
  if (M > kMaxQuantRows)
    return fail(COMET_ERR_UNSUPPORTED, "M=%d exceeds %d rows per call", M, kMaxQuantRows);
  if (N % 16) return fail(COMET_ERR_INVALID_ARG, "N=%d must be a multiple of 16", N);
  comet_status_t st = check_kg(K, G);
  if (st) return st;
  if (!aligned16(A) || !aligned16(sa) || !aligned16(W) || !aligned16(sw) || !aligned16(out))
    return fail(COMET_ERR_INVALID_ARG, "device pointers must be 16-byte aligned");
  return make_map(prec, K / G, map);
}

// ---- plans and workspaces -------------------------------------------------

struct PlanKey {
  int dev, M, N, K, cus;
  std::string mode;
  comet::BlockMap map;
  bool operator<(const PlanKey& o) const {
    if (std::tie(dev, M, N, K, cus, mode) != std::tie(o.dev, o.M, o.N, o.K, o.cus, o.mode))
      return std::tie(dev, M, N, K, cus, mode) < std::tie(o.dev, o.M, o.N, o.K, o.cus, o.mode);
    return std::memcmp(map.bits, o.map.bits, sizeof map.bits) < 0;
  }
};

struct DevicePlan {
  comet::Plan host;
  std::vector<int> blob;  // the uploaded array, kept: the copy is asynchronous
  void* dmem = nullptr;  // units | wg_begin | order | split_index, one allocation
  const comet::WorkUnit* units = nullptr;
  const int* wg_begin = nullptr;
  const int* order = nullptr;
  const int* split_index = nullptr;
};

struct Workspace {
  float* partials = nullptr;
  size_t partial_floats = 0;
  int* counters = nullptr;
  size_t ncounters = 0;
  uint16_t* tmp = nullptr;  // fp16 gate/up output of the few-token SwiGLU path
  size_t tmp_bytes = 0;
};

std::map<PlanKey, DevicePlan> g_plans;
std::map<std::pair<int, hipStream_t>, Workspace> g_ws;
std::map<int, bool> g_attr_set;

std::string sched_mode() {
  const char* m = std::getenv("COMET_SCHED");
  return (m && *m) ? std::string(m) : std::string("cost");
}

// Which GEMM kernel runs for this shape on `cus` compute units.  The stream
// kernels take M <= 64 when the weight panels divide evenly over the CUs
// (and each wave gets enough of them).  Otherwise the few-token kernels take
// M <= 48, except that above 32 rows the 128-row tile kernel takes over when
// its 256-column tiles cover at least 3/4 of the CUs (wide N); the 128-row
// tile kernel runs up to M = 128; above, comet::choose_tile_m picks 128 or
// 256 rows from the shape.
int kernel_kind(int M, int N, int K, int cus) {
  if (comet::skinny_stream_eligible(M, N, K, cus)) return COMET_KERNEL_STREAM;
  const int col_tiles = (N + comet::kTileN - 1) / comet::kTileN;
  const bool wide = 4 * col_tiles >= 3 * cus;
  if (M <= comet::kSkinnyMaxM && !(M > kSkinnyWideM && wide))
    return comet::skinny_shared(M, comet::skinny_splits(N, K, cus))
               ? COMET_KERNEL_FEW_TOKEN_SHARED
               : COMET_KERNEL_FEW_TOKEN;
  return comet::choose_tile_m(M, N, K, comet::kG, cus) == comet::kTileMSmall ? COMET_KERNEL_MID
                                                                             : COMET_KERNEL_TILE;
}

comet::PlanOptions plan_options(int M, int N, int K, int cus, const std::string& mode) {
  comet::PlanOptions opt;
  opt.num_cus = cus;
  opt.tile_m = comet::choose_tile_m(M, N, K, comet::kG, cus);
  opt.tile_n = comet::kTileN;
  opt.mode = mode;
  return opt;
}

// A plan as the kernels read it, one int array: work units (5 ints each) |
// wg_begin | K-block schedule (block index, precision bit and the block's
// offset in A_packed in units of M*64 bytes, then kOrderPad repeats of the
// last entry, since kernels prefetch fixed-size batches past the end of a
// range) | split table.
struct PlanBlob {
  std::vector<int> v;
  size_t o_wgb = 0, o_order = 0, o_split = 0;
};

PlanBlob plan_blob(const comet::Plan& h, const uint8_t* prec) {
  PlanBlob b;
  for (const comet::PlanUnit& u : h.units) {
    b.v.push_back(u.tile);
    b.v.push_back(u.g_begin);
    b.v.push_back(u.g_end);
    b.v.push_back(u.slot);
    b.v.push_back(u.nslots);
  }
  b.o_wgb = b.v.size();
  b.v.insert(b.v.end(), h.wg_begin.begin(), h.wg_begin.end());
  b.o_order = b.v.size();
  std::vector<int> n8_before(h.order.size() + 1, 0);
  for (size_t g = 0; g < h.order.size(); ++g) n8_before[g + 1] = n8_before[g] + (prec[g] == 8);
  for (int g : h.order) b.v.push_back(g | (prec[g] == 8) << 10 | (g + n8_before[g]) << 11);
  const int last = b.v.back();
  b.v.insert(b.v.end(), comet::kOrderPad, last);
  b.o_split = b.v.size();
  b.v.insert(b.v.end(), h.split_base.begin(), h.split_base.end());
  return b;
}

// Plan for (device, shape, map, mode), built and uploaded on first use.
// Caller holds g_mu.
comet_status_t get_plan(int dev, int cus, int M, int N, int K, const uint8_t* prec,
                        const comet::BlockMap& map, const std::string& mode, hipStream_t stream,
                        const DevicePlan** out) {
  PlanKey key{dev, M, N, K, cus, mode, map};
  auto it = g_plans.find(key);
  if (it != g_plans.end()) {
    *out = &it->second;
    return COMET_OK;
  }
  DevicePlan dp;
  std::string err;
  if (!comet::build_plan(M, N, K, comet::kG, prec, plan_options(M, N, K, cus, mode), &dp.host, &err))
    return fail(COMET_ERR_INVALID_ARG, "%s", err.c_str());
  PlanBlob b = plan_blob(dp.host, prec);
  dp.blob = std::move(b.v);
  if (std::getenv("COMET_TEST_FAIL_ALLOC")) return fail(COMET_ERR_OOM, "plan allocation failed (forced)");
  hipError_t e = hipMalloc(&dp.dmem, dp.blob.size() * sizeof(int));
  if (e != hipSuccess) return fail(COMET_ERR_OOM, "plan allocation: %s", hipGetErrorString(e));
  // enqueued on the call's stream ahead of the kernel that reads it; the
  // host array lives in the cache entry, so nobody waits for the copy
  e = hipMemcpyAsync(dp.dmem, dp.blob.data(), dp.blob.size() * sizeof(int),
                     hipMemcpyHostToDevice, stream);
  if (e != hipSuccess) {
    (void)hipFree(dp.dmem);
    return fail(COMET_ERR_HIP, "plan upload: %s", hipGetErrorString(e));
  }
  int* d = static_cast<int*>(dp.dmem);
  dp.units = reinterpret_cast<const comet::WorkUnit*>(d);
  dp.wg_begin = d + b.o_wgb;
  dp.order = d + b.o_order;
  dp.split_index = d + b.o_split;
  const comet::Plan& h = dp.host;
  if (std::getenv("COMET_LOG"))
    std::fprintf(stderr,
                 "[comet] plan M=%d N=%d K=%d mode=%s tiles=%dx%d wgs=%d units=%zu split_tiles=%d "
                 "partial_slots=%d cost max/mean=%.3f\n",
                 M, N, K, mode.c_str(), h.tiles_m, h.tiles_n, h.num_wgs, h.units.size(),
                 h.split_tiles, h.partial_slots, h.mean_wg_cost > 0 ? h.max_wg_cost / h.mean_wg_cost : 0.0);
  *out = &g_plans.emplace(key, std::move(dp)).first->second;
  return COMET_OK;
}

// Split workspace of (device, stream): fp32 partials and arrival counters,
// grown on demand.  Counters start at zero and every launch leaves them at
// zero.  Caller holds g_mu.
comet_status_t get_workspace(int dev, hipStream_t stream, size_t partial_floats, size_t counters,
                             Workspace** out) {
  Workspace& ws = g_ws[{dev, stream}];
  if (partial_floats > ws.partial_floats || counters > ws.ncounters) {
    // only the split buffers are replaced; the stream's fp16 buffer (tmp)
    // stays as it is
    auto drop_split = [&ws] {
      ws.partials = nullptr;
      ws.counters = nullptr;
      ws.partial_floats = 0;
      ws.ncounters = 0;
    };
    if (ws.partials) {
      // the previous launch on this stream may still use them
      hipError_t e = hipStreamSynchronize(stream);
      if (e != hipSuccess) return fail(COMET_ERR_HIP, "workspace sync: %s", hipGetErrorString(e));
      (void)hipFree(ws.partials);
      (void)hipFree(ws.counters);
    }
    const size_t nf = std::max(partial_floats, ws.partial_floats);
    const size_t nc = std::max(counters, ws.ncounters);
    drop_split();
    if (std::getenv("COMET_TEST_FAIL_ALLOC")) return fail(COMET_ERR_OOM, "workspace allocation failed (forced)");
    hipError_t e = hipMalloc(&ws.partials, std::max<size_t>(nf, 1) * sizeof(float));
    if (e != hipSuccess) {
      drop_split();
      return fail(COMET_ERR_OOM, "workspace allocation: %s", hipGetErrorString(e));
    }
    e = hipMalloc(&ws.counters, std::max<size_t>(nc, 1) * sizeof(int));
    if (e == hipSuccess) e = hipMemsetAsync(ws.counters, 0, std::max<size_t>(nc, 1) * sizeof(int), stream);
    if (e != hipSuccess) {
      (void)hipFree(ws.partials);
      if (ws.counters) (void)hipFree(ws.counters);
      drop_split();
      return fail(COMET_ERR_OOM, "workspace counters: %s", hipGetErrorString(e));
    }
    ws.partial_floats = nf;
    ws.ncounters = nc;
  }
  *out = &ws;
  return COMET_OK;
}

// fp16 buffer of the few-token SwiGLU path on (device, stream), grown on
// demand.  Caller holds g_mu.
comet_status_t get_tmp(int dev, hipStream_t stream, size_t bytes, uint16_t** out) {
  Workspace& ws = g_ws[{dev, stream}];
  if (bytes > ws.tmp_bytes) {
    if (ws.tmp) {
      hipError_t e = hipStreamSynchronize(stream);
      if (e != hipSuccess) return fail(COMET_ERR_HIP, "workspace sync: %s", hipGetErrorString(e));
      (void)hipFree(ws.tmp);
      ws.tmp = nullptr;
      ws.tmp_bytes = 0;
    }
    if (std::getenv("COMET_TEST_FAIL_ALLOC")) return fail(COMET_ERR_OOM, "workspace allocation failed (forced)");
    hipError_t e = hipMalloc(&ws.tmp, bytes);
    if (e != hipSuccess) {
      ws.tmp = nullptr;
      return fail(COMET_ERR_OOM, "workspace allocation: %s", hipGetErrorString(e));
    }
    ws.tmp_bytes = bytes;
  }
  *out = ws.tmp;
  return COMET_OK;
}

// The GEMM.  With `swiglu` (non-null) the output is not stored: the tile
// kernels' epilogue quantizes h = SiLU(gate) * up straight into swiglu->A /
// swiglu->sa; the few-token kernel writes fp16 to a workspace that the SwiGLU
// quantizer then reads.
struct SwigluOut {
  uint8_t* A;
  uint16_t* sa;
  comet::BlockMap map;
};

comet_status_t run_gemm(const uint8_t* A, const uint8_t* prec, const uint16_t* sa,
                        const uint8_t* W, const uint16_t* sw, uint16_t* out, int32_t* acc, int M,
                        int N, int K, const comet::BlockMap& map, int m0, int m1, int n0, int n1,
                        hipStream_t stream, const SwigluOut* swiglu = nullptr) {
  int dev;
  DeviceInfo info;
  comet_status_t st = current_device(&dev, &info);
  if (st) return st;
  std::lock_guard<std::mutex> lk(g_mu);
  if (!g_attr_set[dev]) {
    hipError_t e = comet::set_gemm_attributes();
    if (e == hipSuccess) e = comet::set_skinny_attributes();
    if (e != hipSuccess) return fail(COMET_ERR_HIP, "kernel attributes: %s", hipGetErrorString(e));
    g_attr_set[dev] = true;
  }
  const bool diag = acc != nullptr;
  const int kind = kernel_kind(M, N, K, info.cus);
  const bool skinny = kind == COMET_KERNEL_FEW_TOKEN || kind == COMET_KERNEL_FEW_TOKEN_SHARED ||
                      kind == COMET_KERNEL_STREAM;
  // the few-token kernels walk the K-blocks in natural order and need no plan
  const DevicePlan* plan = nullptr;
  // the fused SwiGLU epilogue has no natural-order form: it takes "dp" instead
  std::string mode = sched_mode();
  if (swiglu && mode == "natural") mode = "dp";
  if (!skinny && (st = get_plan(dev, info.cus, M, N, K, prec, map, mode, stream, &plan)))
    return st;
  comet::GemmArgs a{};
  a.splits = skinny ? comet::skinny_splits(N, K, info.cus) : 1;
  Workspace* ws = nullptr;
  // the diagnostic form writes every unit's blocks straight to acc: no partials
  if (!skinny && !diag && plan->host.partial_slots > 0) {
    const size_t slots = (size_t)plan->host.partial_slots;
    if ((st = get_workspace(dev, stream, slots * plan->host.tile_m * plan->host.tile_n, slots,
                            &ws)))
      return st;
  }
  a.A = A;
  a.sa = sa;
  a.W = W;
  a.sw = sw;
  a.out = out;
  a.acc = acc;
  a.partials = ws ? ws->partials : nullptr;
  a.counters = ws ? ws->counters : nullptr;
  if (plan) {
    a.units = plan->units;
    a.wg_begin = plan->wg_begin;
    a.order = plan->order;
    a.split_index = plan->split_index;
    a.tiles_n = plan->host.tiles_n;
  }
  a.n4 = 0;
  for (int g = 0; g < K / comet::kG; ++g) a.n4 += prec[g] == 4;
  a.M = M;
  a.N = N;
  a.K = K;
  a.cus = info.cus;
  a.win_m0 = m0;
  a.win_m1 = m1;
  a.win_n0 = n0;
  a.win_n1 = n1;
  a.map = map;
  // The SwiGLU epilogue is fused into the 128-row tile kernel only.  With
  // the few-token kernels and the 256-row tile kernel, the GEMM plus the
  // standalone SwiGLU quantizer is faster (the epilogue's exp and division
  // then run on the whole chip at once, not on one tile's waves after its
  // K-loop), so the GEMM writes fp16 to the stream's workspace first.
  if (swiglu && kind != COMET_KERNEL_MID) {
    uint16_t* tmp;
    if ((st = get_tmp(dev, stream, (size_t)M * N * sizeof(uint16_t), &tmp))) return st;
    a.out = tmp;
    if (skinny)
      st = launched(comet::launch_gemm_skinny(a, false, stream), "gemm launch");
    else
      st = launched(comet::launch_gemm(a, plan->host.num_wgs, false, false, mode == "natural",
                                       plan->host.tile_m, stream),
                    "gemm launch");
    if (st) return st;
    return launched(comet::launch_swiglu_quantize(tmp, swiglu->A, swiglu->sa, M, N / 2,
                                                  swiglu->map, stream),
                    "swiglu_quantize launch");
  }
  if (swiglu) {
    a.out_A = swiglu->A;
    a.out_sa = swiglu->sa;
    a.out_map = swiglu->map;
  }
  if (skinny) return launched(comet::launch_gemm_skinny(a, diag, stream), "gemm launch");
  return launched(comet::launch_gemm(a, plan->host.num_wgs, diag, swiglu != nullptr,
                                     mode == "natural", plan->host.tile_m, stream),
                  "gemm launch");
}

// Per device: the plan last uploaded into the no-allocation workspace.
std::map<int, std::vector<int>> g_noalloc_plan;

// comet_w4ax_gemm over the fixed per-device workspace: no device allocation.
// The few-token kernels need no workspace.  The tile kernels' plan goes into
// the workspace's plan region (uploaded, with a wait, only when it differs
// from the plan already there); split partials and counters use the other
// regions, and a plan whose splits need more partials than fit is replaced
// by the same mode's whole-tile plan.
comet_status_t run_gemm_noalloc(const uint8_t* A, const uint8_t* prec, const uint16_t* sa,
                                const uint8_t* W, const uint16_t* sw, uint16_t* out, int M, int N,
                                int K, const comet::BlockMap& map, hipStream_t stream) {
  int dev;
  DeviceInfo info;
  comet_status_t st = current_device(&dev, &info);
  if (st) return st;
  std::lock_guard<std::mutex> lk(g_mu);
  if (!g_attr_set[dev]) {
    hipError_t e = comet::set_gemm_attributes();
    if (e == hipSuccess) e = comet::set_skinny_attributes();
    if (e != hipSuccess) return fail(COMET_ERR_HIP, "kernel attributes: %s", hipGetErrorString(e));
    g_attr_set[dev] = true;
  }
  const int kind = kernel_kind(M, N, K, info.cus);
  comet::GemmArgs a{};
  a.A = A;
  a.sa = sa;
  a.W = W;
  a.sw = sw;
  a.out = out;
  a.M = M;
  a.N = N;
  a.K = K;
  a.cus = info.cus;
  a.map = map;
  for (int g = 0; g < K / comet::kG; ++g) a.n4 += prec[g] == 4;
  if (kind == COMET_KERNEL_FEW_TOKEN || kind == COMET_KERNEL_FEW_TOKEN_SHARED ||
      kind == COMET_KERNEL_STREAM) {
    a.splits = comet::skinny_splits(N, K, info.cus);
    return launched(comet::launch_gemm_skinny(a, false, stream), "gemm launch");
  }
  uint8_t* ws = nullptr;
  hipError_t e = comet::noalloc_scratch(dev, &ws);
  if (e != hipSuccess)
    return fail(COMET_ERR_HIP, "workspace address (hipGetSymbolAddress): %s", hipGetErrorString(e));
  std::string mode = sched_mode();
  comet::Plan h;
  std::string err;
  if (!comet::build_plan(M, N, K, comet::kG, prec, plan_options(M, N, K, info.cus, mode), &h, &err))
    return fail(COMET_ERR_INVALID_ARG, "%s", err.c_str());
  const size_t tile_bytes = (size_t)h.tile_m * h.tile_n * sizeof(float);
  if ((size_t)h.partial_slots * tile_bytes > comet::kNoallocPartialBytes ||
      (size_t)h.partial_slots * sizeof(int) > comet::kNoallocCounterBytes) {
    mode = "dp";
    if (!comet::build_plan(M, N, K, comet::kG, prec, plan_options(M, N, K, info.cus, mode), &h, &err))
      return fail(COMET_ERR_INVALID_ARG, "%s", err.c_str());
  }
  const PlanBlob b = plan_blob(h, prec);
  const size_t plan_bytes = b.v.size() * sizeof(int);
  if (plan_bytes > comet::kNoallocPlanBytes)
    return fail(COMET_ERR_UNSUPPORTED,
                "M=%d, N=%d, K=%d: the schedule takes %zu bytes, more than the %zu of the "
                "no-allocation workspace (use comet_w4ax_gemm)",
                M, N, K, plan_bytes, comet::kNoallocPlanBytes);
  float* partials = reinterpret_cast<float*>(ws);
  int* counters = reinterpret_cast<int*>(ws + comet::kNoallocPartialBytes);
  int* plan = reinterpret_cast<int*>(ws + comet::kNoallocPartialBytes + comet::kNoallocCounterBytes);
  std::vector<int>& cur = g_noalloc_plan[dev];
  if (cur != b.v) {
    // the copy reads pageable host memory: wait for it before the vector can change
    e = hipMemcpyAsync(plan, b.v.data(), plan_bytes, hipMemcpyHostToDevice, stream);
    if (e == hipSuccess) e = hipStreamSynchronize(stream);
    if (e != hipSuccess) {
      cur.clear();
      return fail(COMET_ERR_HIP, "plan upload: %s", hipGetErrorString(e));
    }
    cur = b.v;
  }
  // split tiles count arrivals from zero (a fill kernel, not a memset, so the
  // call can be captured in a graph)
  if (h.partial_slots > 0 &&
      (st = launched(comet::launch_zero_ints(counters, h.partial_slots, stream), "counter reset")))
    return st;
  a.partials = partials;
  a.counters = counters;
  a.units = reinterpret_cast<const comet::WorkUnit*>(plan);
  a.wg_begin = plan + b.o_wgb;
  a.order = plan + b.o_order;
  a.split_index = plan + b.o_split;
  a.tiles_n = h.tiles_n;
  a.splits = 1;
  return launched(comet::launch_gemm(a, h.num_wgs, false, false, mode == "natural", h.tile_m,
                                     stream),
                  "gemm launch");
}

}  // namespace

extern "C" {

const char* comet_status_str(comet_status_t s) {
  switch (s) {
    case COMET_OK: return "COMET_OK";
    case COMET_ERR_INVALID_ARG: return "COMET_ERR_INVALID_ARG";
    case COMET_ERR_UNSUPPORTED: return "COMET_ERR_UNSUPPORTED";
    case COMET_ERR_HIP: return "COMET_ERR_HIP";
    case COMET_ERR_OOM: return "COMET_ERR_OOM";
  }
  return "COMET_ERR_UNKNOWN";
}

const char* comet_last_error(void) { return g_last_error.c_str(); }

const char* comet_build_stamp(void) { return kStamp + sizeof("COMET_SOURCE_STAMP=") - 1; }

size_t comet_act_packed_bytes(const uint8_t* prec, int M, int K, int G) {
  if (!prec || M < 1 || G < 1 || K < G || K % G) return 0;
  size_t units = 0;
  for (int g = 0; g < K / G; ++g) {
    if (prec[g] != 4 && prec[g] != 8) return 0;
    units += prec[g] == 8 ? (size_t)G : (size_t)G / 2;
  }
  return units * (size_t)M;
}

comet_status_t comet_fmpq_quantize_act_perm(const uint16_t* X, const int32_t* perm,
                                            const uint8_t* prec, uint8_t* A_packed,
                                            uint16_t* a_scales, int M, int K, int G,
                                            hipStream_t stream) {
  if (!X || !A_packed || !a_scales) return fail(COMET_ERR_INVALID_ARG, "null pointer");
  if (M < 1) return fail(COMET_ERR_INVALID_ARG, "M=%d must be >= 1", M);
  if (M > kMaxQuantRows)
    return fail(COMET_ERR_UNSUPPORTED, "M=%d exceeds %d rows per call", M, kMaxQuantRows);
  comet_status_t st = check_kg(K, G);
  if (st) return st;
  if (!aligned16(X) || !aligned16(A_packed) || !aligned16(a_scales) || !aligned16(perm))
    return fail(COMET_ERR_INVALID_ARG, "device pointers must be 16-byte aligned");
  comet::BlockMap map;
  if ((st = make_map(prec, K / G, &map))) return st;
  int dev;
  DeviceInfo info;
  if ((st = current_device(&dev, &info))) return st;
  return launched(comet::launch_quantize_act(X, perm, A_packed, a_scales, M, K, map, stream),
                  "quantize_act launch");
}

comet_status_t comet_fmpq_quantize_act(const uint16_t* X, const uint8_t* prec, uint8_t* A_packed,
                                       uint16_t* a_scales, int M, int K, int G,
                                       hipStream_t stream) {
  return comet_fmpq_quantize_act_perm(X, nullptr, prec, A_packed, a_scales, M, K, G, stream);
}

comet_status_t comet_pack_w4_perm(const uint16_t* W, const int32_t* perm, uint8_t* W_packed,
                                  uint16_t* w_scales, int N, int K, int G, hipStream_t stream) {
  if (!W || !W_packed || !w_scales) return fail(COMET_ERR_INVALID_ARG, "null pointer");
  if (N < 16 || N % 16)
    return fail(COMET_ERR_INVALID_ARG, "N=%d must be a positive multiple of 16", N);
  comet_status_t st = check_kg(K, G);
  if (st) return st;
  if (!aligned16(W) || !aligned16(W_packed) || !aligned16(w_scales) || !aligned16(perm))
    return fail(COMET_ERR_INVALID_ARG, "device pointers must be 16-byte aligned");
  int dev;
  DeviceInfo info;
  if ((st = current_device(&dev, &info))) return st;
  return launched(comet::launch_pack_w4(W, perm, W_packed, w_scales, N, K, stream),
                  "pack_w4 launch");
}

comet_status_t comet_pack_w4(const uint16_t* W, uint8_t* W_packed, uint16_t* w_scales, int N,
                             int K, int G, hipStream_t stream) {
  return comet_pack_w4_perm(W, nullptr, W_packed, w_scales, N, K, G, stream);
}

comet_status_t comet_channel_absmax(const uint16_t* X, float* absmax, int M, int K,
                                    hipStream_t stream) {
  if (!X || !absmax) return fail(COMET_ERR_INVALID_ARG, "null pointer");
  if (M < 1 || K < 8 || K % 8)
    return fail(COMET_ERR_INVALID_ARG, "M=%d must be >= 1 and K=%d a positive multiple of 8", M,
                K);
  if (!aligned16(X) || (reinterpret_cast<uintptr_t>(absmax) & 3u))
    return fail(COMET_ERR_INVALID_ARG, "X must be 16-byte and absmax 4-byte aligned");
  comet_status_t st;
  int dev;
  DeviceInfo info;
  if ((st = current_device(&dev, &info))) return st;
  return launched(comet::launch_channel_absmax(X, absmax, M, K, stream), "channel_absmax launch");
}

comet_status_t comet_plan_channel_perm(const float* absmax, int K, int G, float outlier_ratio,
                                       float max_frac_8bit, int32_t* perm,
                                       uint8_t* group_prec_map, int* n_outliers) {
  if (!absmax || !perm || !group_prec_map) return fail(COMET_ERR_INVALID_ARG, "null pointer");
  const char* why = comet::plan_channel_perm(absmax, K, G, outlier_ratio, max_frac_8bit, perm,
                                             group_prec_map, n_outliers);
  if (why) return fail(COMET_ERR_INVALID_ARG, "%s", why);
  return ok();
}

comet_status_t comet_kv4_quantize(const uint16_t* X, uint8_t* codes, uint16_t* params, int T,
                                  int C, int G, hipStream_t stream) {
  if (!X || !codes || !params) return fail(COMET_ERR_INVALID_ARG, "null pointer");
  if (G != 32 && G != 64 && G != 128)
    return fail(COMET_ERR_UNSUPPORTED, "G=%d: KV4 groups of 32, 64 or 128 channels", G);
  if (T < 1 || C < G || C % G)
    return fail(COMET_ERR_INVALID_ARG, "T=%d must be >= 1 and C=%d a positive multiple of G", T,
                C);
  if (!aligned16(X) || (reinterpret_cast<uintptr_t>(codes) & 3u) ||
      (reinterpret_cast<uintptr_t>(params) & 3u))
    return fail(COMET_ERR_INVALID_ARG, "X must be 16-byte, codes and params 4-byte aligned");
  comet_status_t st;
  int dev;
  DeviceInfo info;
  if ((st = current_device(&dev, &info))) return st;
  return launched(comet::launch_kv4_quantize(X, codes, params, T, C, G, stream),
                  "kv4_quantize launch");
}

comet_status_t comet_kv4_dequantize(const uint8_t* codes, const uint16_t* params, uint16_t* out,
                                    int T, int C, int G, hipStream_t stream) {
  if (!codes || !params || !out) return fail(COMET_ERR_INVALID_ARG, "null pointer");
  if (G != 32 && G != 64 && G != 128)
    return fail(COMET_ERR_UNSUPPORTED, "G=%d: KV4 groups of 32, 64 or 128 channels", G);
  if (T < 1 || C < G || C % G)
    return fail(COMET_ERR_INVALID_ARG, "T=%d must be >= 1 and C=%d a positive multiple of G", T,
                C);
  if (!aligned16(out) || (reinterpret_cast<uintptr_t>(codes) & 3u) ||
      (reinterpret_cast<uintptr_t>(params) & 3u))
    return fail(COMET_ERR_INVALID_ARG, "out must be 16-byte, codes and params 4-byte aligned");
  comet_status_t st;
  int dev;
  DeviceInfo info;
  if ((st = current_device(&dev, &info))) return st;
  return launched(comet::launch_kv4_dequantize(codes, params, out, T, C, G, stream),
                  "kv4_dequantize launch");
}

comet_status_t comet_w4ax_gemm(const uint8_t* A_packed, const uint8_t* prec,
                               const uint16_t* a_scales, const uint8_t* W_packed,
                               const uint16_t* w_scales, uint16_t* out, int M, int N, int K,
                               int G, hipStream_t stream) {
  comet::BlockMap map;
  comet_status_t st =
      gemm_common(A_packed, prec, a_scales, W_packed, w_scales, out, M, N, K, G, &map);
  if (st) return st;
  return run_gemm(A_packed, prec, a_scales, W_packed, w_scales, out, nullptr, M, N, K, map, 0, 0,
                  0, 0, stream);
}

comet_status_t comet_w4ax_gemm_noalloc(const uint8_t* A_packed, const uint8_t* prec,
                                       const uint16_t* a_scales, const uint8_t* W_packed,
                                       const uint16_t* w_scales, uint16_t* out, int M, int N,
                                       int K, int G, hipStream_t stream) {
  comet::BlockMap map;
  comet_status_t st =
      gemm_common(A_packed, prec, a_scales, W_packed, w_scales, out, M, N, K, G, &map);
  if (st) return st;
  return run_gemm_noalloc(A_packed, prec, a_scales, W_packed, w_scales, out, M, N, K, map, stream);
}

comet_status_t comet_w4ax_gemm_swiglu_quant(const uint8_t* A_packed, const uint8_t* prec,
                                            const uint16_t* a_scales, const uint8_t* W_packed,
                                            const uint16_t* w_scales, int M, int N, int K, int G,
                                            const uint8_t* out_prec, uint8_t* out_A_packed,
                                            uint16_t* out_a_scales, hipStream_t stream) {
  if (!out_A_packed || !out_a_scales) return fail(COMET_ERR_INVALID_ARG, "null pointer");
  if (N < 256 || N % 256)
    return fail(COMET_ERR_INVALID_ARG, "N=%d must be a positive multiple of 256 (2G-wide gate/up "
                "column groups)", N);
  if (!aligned16(out_A_packed) || !aligned16(out_a_scales))
    return fail(COMET_ERR_INVALID_ARG, "device pointers must be 16-byte aligned");
  comet::BlockMap map;
  // `out` is not written on this path; a non-null placeholder passes the common checks
  comet_status_t st = gemm_common(A_packed, prec, a_scales, W_packed, w_scales, out_A_packed, M,
                                  N, K, G, &map);
  if (st) return st;
  SwigluOut so{out_A_packed, out_a_scales, {}};
  if ((st = make_map(out_prec, N / 2 / G, &so.map))) return st;
  return run_gemm(A_packed, prec, a_scales, W_packed, w_scales, nullptr, nullptr, M, N, K, map, 0,
                  0, 0, 0, stream, &so);
}

comet_status_t comet_swiglu_quantize(const uint16_t* GU, const uint8_t* out_prec,
                                     uint8_t* out_A_packed, uint16_t* out_a_scales, int M, int I,
                                     int G, hipStream_t stream) {
  if (!GU || !out_A_packed || !out_a_scales) return fail(COMET_ERR_INVALID_ARG, "null pointer");
  if (M < 1) return fail(COMET_ERR_INVALID_ARG, "M=%d must be >= 1", M);
  if (M > kMaxQuantRows)
    return fail(COMET_ERR_UNSUPPORTED, "M=%d exceeds %d rows per call", M, kMaxQuantRows);
  comet_status_t st = check_kg(I, G);
  if (st) return st;
  if (!aligned16(GU) || !aligned16(out_A_packed) || !aligned16(out_a_scales))
    return fail(COMET_ERR_INVALID_ARG, "device pointers must be 16-byte aligned");
  comet::BlockMap map;
  if ((st = make_map(out_prec, I / G, &map))) return st;
  int dev;
  DeviceInfo info;
  if ((st = current_device(&dev, &info))) return st;
  return launched(comet::launch_swiglu_quantize(GU, out_A_packed, out_a_scales, M, I, map, stream),
                  "swiglu_quantize launch");
}

comet_status_t comet_w4ax_gemm_acc(const uint8_t* A_packed, const uint8_t* prec,
                                   const uint16_t* a_scales, const uint8_t* W_packed,
                                   const uint16_t* w_scales, int32_t* acc, int M, int N, int K,
                                   int G, int m0, int m1, int n0, int n1, hipStream_t stream) {
  comet::BlockMap map;
  comet_status_t st =
      gemm_common(A_packed, prec, a_scales, W_packed, w_scales, acc, M, N, K, G, &map);
  if (st) return st;
  if (m0 < 0 || m1 > M || m0 >= m1 || n0 < 0 || n1 > N || n0 >= n1)
    return fail(COMET_ERR_INVALID_ARG, "window [%d,%d)x[%d,%d) is empty or outside %dx%d", m0,
                m1, n0, n1, M, N);
  return run_gemm(A_packed, prec, a_scales, W_packed, w_scales, nullptr, acc, M, N, K, map, m0, m1,
                  n0, n1, stream);
}

comet_status_t comet_schedule_query(int M, int N, int K, int G, const uint8_t* prec, int num_cus,
                                    int* units, int max_units, int* n_units, int* wg_begin,
                                    int max_wgs, int* n_wgs, int* order, int* tile_m,
                                    int* tile_n) {
  if (M < 1 || N < 1 || num_cus < 1) return fail(COMET_ERR_INVALID_ARG, "bad shape or CU count");
  comet_status_t st = check_kg(K, G);
  if (st) return st;
  comet::BlockMap map;
  if ((st = make_map(prec, K / G, &map))) return st;
  comet::PlanOptions opt = plan_options(M, N, K, num_cus, sched_mode());
  comet::Plan plan;
  std::string err;
  if (!comet::build_plan(M, N, K, G, prec, opt, &plan, &err))
    return fail(COMET_ERR_INVALID_ARG, "%s", err.c_str());
  if (n_units) *n_units = (int)plan.units.size();
  if (n_wgs) *n_wgs = plan.num_wgs;
  if (tile_m) *tile_m = plan.tile_m;
  if (tile_n) *tile_n = plan.tile_n;
  if (units) {
    if (max_units < (int)plan.units.size())
      return fail(COMET_ERR_INVALID_ARG, "units buffer holds %d, need %d", max_units,
                  (int)plan.units.size());
    for (size_t i = 0; i < plan.units.size(); ++i) {
      const comet::PlanUnit& u = plan.units[i];
      int* o = units + 5 * i;
      o[0] = u.tile;
      o[1] = u.g_begin;
      o[2] = u.g_end;
      o[3] = u.slot;
      o[4] = u.nslots;
    }
  }
  if (wg_begin) {
    if (max_wgs < plan.num_wgs + 1)
      return fail(COMET_ERR_INVALID_ARG, "wg_begin buffer holds %d, need %d", max_wgs,
                  plan.num_wgs + 1);
    for (int i = 0; i <= plan.num_wgs; ++i) wg_begin[i] = plan.wg_begin[i];
  }
  if (order)
    for (int i = 0; i < K / G; ++i) order[i] = plan.order[i];
  return ok();
}

int comet_gemm_kernel(int M, int N, int K, int G, int num_cus) {
  if (M < 1 || N < 16 || N % 16 || num_cus < 1) {
    fail(COMET_ERR_INVALID_ARG, "M=%d, N=%d, num_cus=%d: bad shape or CU count", M, N, num_cus);
    return -1;
  }
  if (check_kg(K, G)) return -1;
  return kernel_kind(M, N, K, num_cus);
}

void comet_release_caches(void) {
  std::lock_guard<std::mutex> lk(g_mu);
  int cur = -1;
  (void)hipGetDevice(&cur);
  for (auto& kv : g_plans) {
    (void)hipSetDevice(kv.first.dev);
    (void)hipFree(kv.second.dmem);
  }
  for (auto& kv : g_ws) {
    (void)hipSetDevice(kv.first.first);
    (void)hipFree(kv.second.partials);
    (void)hipFree(kv.second.counters);
    (void)hipFree(kv.second.tmp);
  }
  if (cur >= 0) (void)hipSetDevice(cur);
  g_plans.clear();
  g_ws.clear();
  g_attr_set.clear();
  g_devices.clear();
}

}  // extern "C"
