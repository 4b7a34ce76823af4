// scheduler.h -- per-block-precision tile scheduler (host, pure C++).
//
// The paper's fine-grained SM scheduling (Sec. 4.4) has three parts:
// synchronisation only before write-back, tile remapping (spread 4-bit and
// 8-bit K-blocks evenly over the compute units) and tile decomposition (a
// tile may be shared by several compute units, Stream-K style).  On gfx950
// both precisions run on the same FP8 MFMA rate, but an 8-bit K-block costs
// more (two MFMAs per 16x16 block and a wider unpack), so a K-block of each
// precision carries its own cost.  The planner cuts the flattened
// (tile x K-block) cost space into equal shares, one per persistent
// workgroup, at K-block boundaries.  Full tiles go to workgroups directly
// (data-parallel waves); only the last, fractional wave of tiles is split.
#pragma once

#include <cstdint>
#include <string>
#include <vector>

namespace comet {

struct PlanUnit {
  int tile;
  int g_begin;  // position in `order`
  int g_end;
  int slot;
  int nslots;
};

struct Plan {
  int M = 0, N = 0, K = 0;
  int tile_m = 0, tile_n = 0;
  int tiles_m = 0, tiles_n = 0;
  int num_wgs = 0;             // persistent workgroups launched
  std::vector<int> order;      // K-block processing order (all 4-bit, then all 8-bit; natural: 0..NG-1)
  std::vector<PlanUnit> units; // grouped by workgroup
  std::vector<int> wg_begin;   // num_wgs + 1 offsets into units
  std::vector<int> split_base; // per tile: first partial slot index, or -1 if unsplit
  int partial_slots = 0;       // total fp32 partial tiles needed
  int split_tiles = 0;
  double max_wg_cost = 0, mean_wg_cost = 0;
  std::string mode;
};

struct PlanOptions {
  int num_cus = 256;
  int wgs_per_cu = 1;
  int tile_m = 128;
  int tile_n = 128;
  double cost4 = 1.0;   // relative cost of a 4-bit K-block of one tile
  double cost8 = 1.7;   // relative cost of an 8-bit K-block of one tile
  // "cost" mode splits the last wave of tiles only if leaving it unsplit
  // would idle more than this share of the workgroups
  double split_min_idle = 0.3;
  // "natural": the map's own K-block order, one whole tile per unit (no tile
  //            remapping, no tile decomposition);
  // "dp": precision-batched order, one whole tile per unit, tiles dealt
  //       round-robin;
  // "cost": precision-batched order, data-parallel full waves + cost-balanced
  //         split of the remainder.
  std::string mode = "cost";
};

// Builds the plan.  `prec` holds K/G entries in {4, 8}.  Returns false (and
// sets *err) on inconsistent arguments.
bool build_plan(int M, int N, int K, int G, const uint8_t* prec, const PlanOptions& opt,
                Plan* plan, std::string* err);

// Output tile height (rows) for an M x N x K GEMM on `cus` workgroups of
// 256-column tiles: 128 up to 128 rows, else 256 unless 128-row tiles are
// estimated clearly faster (see scheduler.cpp).
int choose_tile_m(int M, int N, int K, int G, int cus);

}  // namespace comet
