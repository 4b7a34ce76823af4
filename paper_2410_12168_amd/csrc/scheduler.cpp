// scheduler.cpp -- per-block-precision tile scheduler (see scheduler.h).
#include "scheduler.h"

#include <algorithm>
#include <cmath>

namespace comet {

namespace {

// Tile visiting sequence.  Workgroups are dispatched round-robin over the
// XCDs (workgroup w runs on XCD w % xcds), and each XCD has its own L2.  The
// sequence walks the tile grid in bands of `band` tile rows, column by column
// inside a band, and each XCD receives a contiguous run of it, so the tiles an
// XCD works on at the same time share activation rows and weight columns.
std::vector<int> tile_sequence(int tiles_m, int tiles_n) {
  const int band = 4;
  std::vector<int> seq;
  seq.reserve((size_t)tiles_m * tiles_n);
  for (int b0 = 0; b0 < tiles_m; b0 += band) {
    const int b1 = std::min(tiles_m, b0 + band);
    for (int tn = 0; tn < tiles_n; ++tn)
      for (int tm = b0; tm < b1; ++tm) seq.push_back(tm * tiles_n + tn);
  }
  return seq;
}

// Workgroup that takes position s of a wave of P workgroups, chosen so that
// each XCD's workgroups (w % xcds == x) own a contiguous run of positions:
// positions [x * P/xcds, (x+1) * P/xcds) go to XCD x.
int wg_for_slot(int s, int P, int xcds) {
  if (xcds <= 1 || P % xcds) return s;
  const int per_xcd = P / xcds;
  return (s % per_xcd) * xcds + s / per_xcd;
}

}  // namespace

bool build_plan(int M, int N, int K, int G, const uint8_t* prec, const PlanOptions& opt,
                Plan* plan, std::string* err) {
  if (M < 1 || N < 1 || K < G || G < 1 || K % G || !prec || opt.num_cus < 1 ||
      opt.wgs_per_cu < 1 || opt.tile_m < 1 || opt.tile_n < 1) {
    if (err) *err = "build_plan: bad arguments";
    return false;
  }
  const int NG = K / G;
  Plan p;
  p.M = M;
  p.N = N;
  p.K = K;
  p.tile_m = opt.tile_m;
  p.tile_n = opt.tile_n;
  p.tiles_m = (M + opt.tile_m - 1) / opt.tile_m;
  p.tiles_n = (N + opt.tile_n - 1) / opt.tile_n;
  p.mode = opt.mode;
  const int T = p.tiles_m * p.tiles_n;
  const int P = opt.num_cus * opt.wgs_per_cu;
  const int xcds = opt.num_cus % 32 == 0 ? opt.num_cus / 32 : 1;

  if (opt.mode != "dp" && opt.mode != "cost" && opt.mode != "natural") {
    if (err) *err = "build_plan: unknown mode " + opt.mode;
    return false;
  }
  // K-block order: precision-batched (all 4-bit blocks, then all 8-bit ones),
  // so every tile's loop has at most two uniform phases and a split unit
  // switches precision at most once.  "natural" keeps the map's own order
  // (the baseline without tile remapping).
  for (int g = 0; g < NG; ++g) {
    if (prec[g] != 4 && prec[g] != 8) {
      if (err) *err = "build_plan: map entry not 4 or 8";
      return false;
    }
    if (prec[g] == 4 || opt.mode == "natural") p.order.push_back(g);
  }
  if (opt.mode != "natural")
    for (int g = 0; g < NG; ++g)
      if (prec[g] == 8) p.order.push_back(g);
  std::vector<double> prefix(NG + 1, 0.0);
  for (int i = 0; i < NG; ++i)
    prefix[i + 1] = prefix[i] + (prec[p.order[i]] == 8 ? opt.cost8 : opt.cost4);
  const double Ct = prefix[NG];

  const std::vector<int> seq = tile_sequence(p.tiles_m, p.tiles_n);
  p.split_base.assign(T, -1);

  // How many tiles go to data-parallel waves, and how many are split.  A
  // split tile costs a fixup (fp32 partials, and a device-scope release and
  // acquire, each a whole-L2 write-back or invalidate on a multi-XCD part),
  // measured at about a quarter to a third of a wave of tiles.  So the last
  // wave is split only when, unsplit, it would leave a larger share of the
  // workgroups idle.
  int dp_tiles = T;
  if (opt.mode == "cost" && T % P != 0) {
    const double idle = (double)(P - T % P) / P;
    if (idle > opt.split_min_idle) {
      const int full = T / P;
      dp_tiles = full >= 1 ? (full - 1) * P : 0;
    }
  }
  const int sk_tiles = T - dp_tiles;
  // Number of workgroups: enough for the data-parallel waves; the split part
  // uses all P unless pieces would become shorter than 2 K-blocks.
  int nw = std::min(P, T);
  int sk_wgs = 0;
  if (sk_tiles > 0) {
    sk_wgs = P;
    const long long total_blocks = (long long)sk_tiles * NG;
    if (total_blocks < 2LL * sk_wgs) sk_wgs = (int)std::max(1LL, total_blocks / 2);
    nw = std::max(dp_tiles > 0 ? P : 0, sk_wgs);
  }
  p.num_wgs = nw;
  std::vector<std::vector<PlanUnit>> per(nw);

  // Data-parallel waves (fewer tiles than workgroups: one tile each, in order).
  for (int i = 0; i < dp_tiles; ++i) {
    const int w = dp_tiles < P ? i : wg_for_slot(i % P, P, xcds);
    per[w].push_back(PlanUnit{seq[i], 0, NG, 0, 1});
  }

  // Cost-balanced split of the remaining tiles over sk_wgs workgroups.
  if (sk_tiles > 0) {
    // cut[w] = flattened position (tile-major over the sk tiles, then block
    // position) where workgroup w's share starts.
    const double total = Ct * sk_tiles;
    std::vector<long long> cut(sk_wgs + 1);
    cut[0] = 0;
    cut[sk_wgs] = (long long)sk_tiles * NG;
    for (int w = 1; w < sk_wgs; ++w) {
      const double target = total * w / sk_wgs;
      int t = (int)std::floor(target / Ct);
      if (t >= sk_tiles) t = sk_tiles - 1;
      const double rem = target - t * Ct;
      // nearest block boundary inside tile t
      int b = (int)(std::lower_bound(prefix.begin(), prefix.end(), rem) - prefix.begin());
      if (b > 0 && rem - prefix[b - 1] < prefix[b] - rem) --b;
      long long c = (long long)t * NG + b;
      cut[w] = std::max(cut[w - 1], c);
    }
    // pieces per tile, to number the slots
    std::vector<int> nslots(sk_tiles, 0);
    for (int w = 0; w < sk_wgs; ++w) {
      long long a = cut[w], e = cut[w + 1];
      while (a < e) {
        const int t = (int)(a / NG);
        const long long tend = (long long)(t + 1) * NG;
        const long long stop = std::min(e, tend);
        ++nslots[t];
        a = stop;
      }
    }
    std::vector<int> next_slot(sk_tiles, 0);
    for (int t = 0; t < sk_tiles; ++t) {
      const int tile = seq[dp_tiles + t];
      if (nslots[t] > 1) {
        p.split_base[tile] = p.partial_slots;
        p.partial_slots += nslots[t];
        ++p.split_tiles;
      }
    }
    for (int w = 0; w < sk_wgs; ++w) {
      const int wg = sk_wgs == P ? wg_for_slot(w, P, xcds) : w;
      long long a = cut[w], e = cut[w + 1];
      while (a < e) {
        const int t = (int)(a / NG);
        const long long tend = (long long)(t + 1) * NG;
        const long long stop = std::min(e, tend);
        const int tile = seq[dp_tiles + t];
        per[wg].push_back(PlanUnit{tile, (int)(a - (long long)t * NG), (int)(stop - (long long)t * NG),
                                   next_slot[t]++, nslots[t]});
        a = stop;
      }
    }
  }

  // Within each workgroup: the split slots whose partial another slot will
  // add first, whole tiles next, and the slots that finish a split tile
  // last.  The early partials are then written while the chip still
  // computes, and a finishing slot usually finds the others arrived, so it
  // reads their partials and keeps its own in registers.
  for (std::vector<PlanUnit>& v : per) {
    auto rank = [](const PlanUnit& u) {
      return u.nslots == 1 ? 1 : (u.slot < u.nslots - 1 ? 0 : 2);
    };
    std::stable_sort(v.begin(), v.end(),
                     [&](const PlanUnit& a, const PlanUnit& b) { return rank(a) < rank(b); });
  }

  // Flatten, and record the cost balance.
  p.wg_begin.push_back(0);
  double sum = 0;
  for (int w = 0; w < nw; ++w) {
    double c = 0;
    for (const PlanUnit& u : per[w]) {
      p.units.push_back(u);
      c += prefix[u.g_end] - prefix[u.g_begin];
    }
    p.wg_begin.push_back((int)p.units.size());
    p.max_wg_cost = std::max(p.max_wg_cost, c);
    sum += c;
  }
  p.mean_wg_cost = nw ? sum / nw : 0;
  *plan = std::move(p);
  return true;
}

// Tile height.  Up to 128 rows a 128-row tile (a taller one would leave MFMA
// rows idle).  Above that, a 256-row tile does one K-block in about 2.1 us
// on MI355X against about 1.35 us for a 128-row tile, so per row it is the
// cheaper unit of work, but there are half as many tiles.  When that leaves a
// fractional last wave that the plan splits (build_plan, "cost" mode), the
// split costs a fixup of about 25 us: every split tile's fp32 partials are
// written and read back at the end of the launch, all at once.  The estimate
// below prices both heights that way (per workgroup: the K-blocks it runs,
// plus the fixup if any tile is split, plus ~4 us more prologue and epilogue
// for the smaller tile) and keeps 256 rows unless 128 is 3% faster: e.g.
// 2048 x 4096 x 4096 on 256 CUs has 128 tiles of 256 rows, each split in
// two, or 256 tiles of 128 rows, one per workgroup.
int choose_tile_m(int M, int N, int K, int G, int cus) {
  constexpr int kSmall = 128, kLarge = 256, kTileCols = 256;
  if (M <= kSmall || cus <= 0 || G <= 0) return M <= kSmall ? kSmall : kLarge;
  const PlanOptions defaults;
  const long long NG = K / G, P = cus;
  auto estimate = [&](int tm, double us_per_block, double extra_us) {
    const long long T = (long long)((M + tm - 1) / tm) * ((N + kTileCols - 1) / kTileCols);
    bool split = false;
    long long blocks = (T + P - 1) / P * NG;
    if (T % P != 0 && (double)(P - T % P) / P > defaults.split_min_idle) {
      split = true;
      blocks = (T * NG + P - 1) / P;
    }
    return blocks * us_per_block + (split ? 25.0 : 0.0) + extra_us;
  };
  const double t_large = estimate(kLarge, 2.1, 0.0);
  const double t_small = estimate(kSmall, 1.35, 4.0);
  return t_small < 0.97 * t_large ? kSmall : kLarge;
}

int skinny_splits(int N, int K, int cus) {
  // waves of (16 columns, slot) over 4 SIMDs per CU: pick the slot count whose
  // last round of waves is fullest, preferring fewer slots.  The slots of a
  // column block share one workgroup of four waves, so the count divides 4.
  const int simds = 4 * cus, cblocks = N / 16, NG = K / 128;
  int best = 1;
  double best_eff = 0;
  for (int s : {1, 2, 4}) {
    if (NG / s < 4) break;
    const long long units = (long long)cblocks * s;
    const long long rounds = (units + simds - 1) / simds;
    const double eff = (double)units / (double)(rounds * simds);
    if (eff > best_eff + 0.02) {
      best_eff = eff;
      best = s;
    }
  }
  return best;
}

}  // namespace comet
