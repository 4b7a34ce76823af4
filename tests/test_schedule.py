"""Properties of the per-block-precision tile scheduler (host only).

Tile remapping and tile decomposition (paper Sec. 4.4) must cover every
(tile, K-block) pair exactly once, number the partial slots of split tiles
consistently, keep every workgroup's cost within one K-block of the mean,
and be deterministic.
"""
import numpy as np
import pytest

import paper_2410_12168_amd as comet
import synth

COST4, COST8 = 1.0, 1.7


def check_plan(M, N, K, prec, num_cus=256):
    s = comet.comet_schedule_query(M, N, K, prec, num_cus)
    NG = K // 128
    tm, tn = s["tile_m"], s["tile_n"]
    T = -(-M // tm) * -(-N // tn)
    order = s["order"]
    assert sorted(order.tolist()) == list(range(NG))  # a permutation
    p = np.asarray(prec)[order]
    assert np.all(np.diff((p == 8).astype(int)) >= 0)  # 4-bit blocks first, then 8-bit
    cover = np.zeros((T, NG), np.int32)
    slots = {}
    units, wgb = s["units"], s["wg_begin"]
    assert wgb[0] == 0 and wgb[-1] == len(units) and np.all(np.diff(wgb) >= 0)
    assert s["num_wgs"] <= num_cus
    cost = np.where(p == 8, COST8, COST4)
    prefix = np.concatenate([[0], np.cumsum(cost)])
    wg_cost = []
    for w in range(s["num_wgs"]):
        c = 0.0
        for tile, g0, g1, slot, ns in units[wgb[w]:wgb[w + 1]]:
            assert 0 <= tile < T and 0 <= g0 < g1 <= NG and 0 <= slot < ns
            cover[tile, g0:g1] += 1
            slots.setdefault(tile, []).append((slot, ns, g0, g1))
            c += prefix[g1] - prefix[g0]
        wg_cost.append(c)
    assert np.all(cover == 1)  # every (tile, block) exactly once
    for tile, ss in slots.items():
        ns = ss[0][1]
        assert all(x[1] == ns for x in ss) and sorted(x[0] for x in ss) == list(range(ns))
        # slots follow the block order
        assert [x[2] for x in sorted(ss)] == sorted(x[2] for x in ss)
    wg_cost = np.array(wg_cost)
    return s, wg_cost, prefix[-1]


@pytest.mark.parametrize("M,N,K", [(2048, 6144, 4096), (2048, 4096, 4096), (2048, 28672, 4096),
                                   (2048, 4096, 14336), (4096, 10240, 8192), (4096, 8192, 8192),
                                   (4096, 57344, 8192), (4096, 8192, 28672), (16, 1024, 1024),
                                   (1, 57344, 8192), (128, 57344, 8192), (100, 272, 1152)])
def test_cover_and_balance(M, N, K):
    NG = K // 128
    prec = synth.prec_map(NG, max(1, NG // 16))
    s, wg_cost, Ct = check_plan(M, N, K, prec)
    T = -(-M // s["tile_m"]) * -(-N // s["tile_n"])
    if T > 256:
        # balanced: no workgroup above the mean by more than one 8-bit block
        assert wg_cost.max() <= wg_cost.mean() + COST8 + 1e-9


@pytest.mark.parametrize("frac", [0, 1 / 16, 1 / 4, 1 / 2])
@pytest.mark.parametrize("placement", ["contiguous", "random"])
def test_load_balance_sweep(frac, placement):
    K = 28672
    NG = K // 128
    prec = synth.prec_map(NG, int(NG * frac), placement, seed=1)
    s, wg_cost, Ct = check_plan(4096, 8192, K, prec)
    assert wg_cost.max() <= wg_cost.mean() + COST8 + 1e-9


def test_deterministic():
    prec = synth.prec_map(64, 4, "random", 3)
    a = comet.comet_schedule_query(4096, 10240, 8192, prec)
    b = comet.comet_schedule_query(4096, 10240, 8192, prec)
    assert all(np.array_equal(a[k], b[k]) for k in ("units", "wg_begin", "order"))


def test_small_cu_counts():
    prec = synth.prec_map(8, 1)
    for cus in (1, 3, 7, 64):
        check_plan(300, 1024, 1024, prec, num_cus=cus)


def test_tile_height_follows_m():
    # the tile kernel uses 128-row tiles up to M = 128 and 256-row tiles above
    prec = np.full(64, 4, np.uint8)
    for M, want in ((65, 128), (100, 128), (128, 128), (129, 256), (4096, 256)):
        s = comet.comet_schedule_query(M, 57344, 8192, prec)
        assert s["tile_m"] == want and s["tile_n"] == 256


@pytest.mark.parametrize("M,N,K,want", [
    (2048, 4096, 4096, 128),    # 128 tiles of 256 rows, all split; 256 of 128 rows: one each
    (2048, 4096, 14336, 256),   # the same tiles, but a long K amortizes the split
    (2048, 6144, 4096, 256),    # 192 tiles of 256 rows: a quarter idle, not split
    (2048, 28672, 4096, 256),
    (4096, 10240, 8192, 256),
    (256, 57344, 8192, 256)])
def test_tile_height_from_the_shape(M, N, K, want):
    # above 128 rows the plan prices both heights (K-blocks per workgroup,
    # plus the split fixup) and keeps 256 rows unless 128 is clearly faster
    prec = np.full(K // 128, 4, np.uint8)
    s = comet.comet_schedule_query(M, N, K, prec)
    assert s["tile_m"] == want
    kind = comet.KERNEL_NAMES[comet.comet_gemm_kernel(M, N, K, 256)]
    assert kind == ("mid" if want == 128 else "tile")
    # the 128-row plan splits nothing here: one tile per workgroup
    if want == 128:
        units = s["units"]
        assert (units[:, 4] == 1).all() and len(units) == 256


@pytest.mark.parametrize("M,N,K", [(4096, 10240, 8192), (2048, 28672, 4096), (512, 8192, 8192),
                                   (300, 1024, 1024)])
def test_split_slots_ordered_within_workgroup(M, N, K):
    # a workgroup runs the slots whose partial another slot adds first, whole
    # tiles next and the slots that finish a split tile last
    prec = synth.prec_map(K // 128, K // 128 // 16)
    s = comet.comet_schedule_query(M, N, K, prec)
    u, wgb = s["units"], s["wg_begin"]
    rank = np.where(u[:, 4] == 1, 1, np.where(u[:, 3] < u[:, 4] - 1, 0, 2))
    assert (rank != 1).any()
    for w in range(s["num_wgs"]):
        r = rank[wgb[w]:wgb[w + 1]]
        assert (np.diff(r) >= 0).all(), (w, r)


@pytest.mark.parametrize("M,N,split", [(128, 57344, False),   # 224 tiles: 12.5% of a wave idle
                                       (4096, 7936, False),   # 496 tiles: 6% idle
                                       (4096, 10240, True),   # 640 tiles: half a wave idle
                                       (2048, 28672, True)])  # 896 tiles
def test_last_wave_split_only_when_worth_it(M, N, split):
    # a split tile costs a cross-workgroup fixup; the last wave is split only
    # when leaving it whole would idle more than 30% of the workgroups
    K = 8192
    prec = synth.prec_map(K // 128, 4)
    s, wg_cost, Ct = check_plan(M, N, K, prec)
    assert bool((s["units"][:, 4] > 1).any()) == split
