"""Pins of the oracle's evaluation metrics (section "Selection Regret (The
Target Metric)": mean / median / 95th percentile / max regret, Top1, Top5
with minimum-rank ties, Within5%) and baselines (section "Final Fit and Test
Protocol": the uniform-random pick's expected regret, the best static
configuration over groups where it appears in at least 80% of them).

Hand-computed groups with ties and an infeasible (+inf) runtime, the numpy
percentile, the exact uniform-pick expectation (the mean regret over every
possible pick), and picks equal to the fastest runtime."""
import numpy as np
import pytest

import oracle
import synth


def groups():
    rt = np.array([3, 1, 2, 1,   5, 5, 5,   2, np.inf, 4,   1, 2], np.float32)
    seg = np.array([0, 4, 7, 10, 10, 12], np.int64)     # the fourth group is empty
    idx = np.array([[2], [1], [1], [-1], [0]], np.int32)
    return rt, seg, idx


def test_hand_computed_groups():
    rt, seg, idx = groups()
    agg, reg, rank, ybar = oracle.evaluate(rt, seg, idx)
    assert reg[0] == 0.5 and reg[1] == 0.0 and reg[2] == 1.0 and np.isnan(reg[3]) and reg[4] == 0.0
    assert rank.tolist() == [3, 1, 3, 0, 1]
    assert ybar[0] == pytest.approx((1 / 3 + 1 + 0.5 + 1) / 4, rel=1e-15)
    assert ybar[1] == 1.0 and ybar[2] == 0.5 and np.isnan(ybar[3]) and ybar[4] == 0.75
    assert agg["n_groups"] == 4
    assert agg["mean_regret"] == 0.375
    assert agg["median_regret"] == 0.25          # sorted (0, 0, 0.5, 1), position 1.5
    assert agg["p95_regret"] == pytest.approx(0.5 + 0.85 * 0.5, rel=1e-15)
    assert agg["max_regret"] == 1.0
    assert agg["top1"] == 0.5 and agg["top5"] == 1.0 and agg["within5"] == 0.5
    assert agg["random_regret"] == pytest.approx(((1 - ybar[0]) + 0 + 0.5 + 0.25) / 4, rel=1e-15)


def test_percentiles_match_numpy():
    rng = np.random.default_rng(5)
    seg = synth.ragged_segments(rng, 301, 30, empty_frac=0.0)
    rt = rng.lognormal(0, 0.5, int(seg[-1])).astype(np.float32)
    idx = np.zeros((301, 1), np.int32)
    agg, reg, _, _ = oracle.evaluate(rt, seg, idx)
    assert agg["median_regret"] == pytest.approx(np.percentile(reg, 50), rel=1e-13, abs=1e-15)
    assert agg["p95_regret"] == pytest.approx(np.percentile(reg, 95), rel=1e-13, abs=1e-15)
    assert agg["mean_regret"] == pytest.approx(reg.mean(), rel=1e-13)
    assert agg["max_regret"] == reg.max()


def test_fastest_pick_gives_zero_regret_and_top1():
    rng = np.random.default_rng(6)
    seg = synth.ragged_segments(rng, 50, 40, empty_frac=0.0)
    rt = rng.choice(np.array([1.0, 2.0, 3.0, np.inf], np.float32), int(seg[-1]))
    idx, _ = oracle.topk(-rt, seg, 5)
    agg, reg, rank, _ = oracle.evaluate(rt, seg, idx)
    finite = np.array([np.isfinite(rt[seg[p]:seg[p + 1]]).any() for p in range(50)])
    assert np.all(reg == 0.0) and np.all(rank == 1)
    assert agg["top1"] == 1.0 and agg["within5"] == 1.0 and agg["mean_regret"] == 0.0
    assert finite.any()


@pytest.mark.parametrize("seed", range(3))
def test_random_regret_is_mean_over_all_picks(seed):
    rng = np.random.default_rng(seed)
    n = 9
    rt = rng.choice(np.array([1.0, 1.5, 2.0, 4.0, np.inf], np.float32), n)
    rt[0] = 1.0
    seg = np.array([0, n], np.int64)
    regs = []
    for j in range(n):
        _, reg, _, _ = oracle.evaluate(rt, seg, np.array([[j]], np.int32))
        regs.append(reg[0])
    agg, _, _, _ = oracle.evaluate(rt, seg, np.array([[0]], np.int32))
    assert agg["random_regret"] == pytest.approx(np.mean(regs), rel=1e-14)


def test_rank_uses_minimum_rank_ties():
    rt = np.array([2, 1, 2, 2, 3], np.float32)
    seg = np.array([0, 5], np.int64)
    for pick, want in ((0, 2), (2, 2), (3, 2), (1, 1), (4, 5)):
        _, _, rank, _ = oracle.evaluate(rt, seg, np.array([[pick]], np.int32))
        assert rank[0] == want


def test_no_counted_group_gives_nan():
    agg, _, _, _ = oracle.evaluate(np.zeros(0, np.float32), np.array([0, 0], np.int64), np.array([[-1]], np.int32))
    assert agg["n_groups"] == 0 and np.isnan(agg["mean_regret"]) and np.isnan(agg["p95_regret"])


def test_static_config_hand_built():
    # five groups; config 9 is perfect but appears in 3/5 < 80% of groups;
    # config 3 appears in 4/5 (eligible), config 7 in all five.
    rows = [  # (config id, runtime) per group; the group's best runtime is 1
        [(7, 2.0), (3, 1.0), (9, 1.0)],
        [(7, 1.0), (3, 2.0), (9, 1.0)],
        [(7, 4.0), (3, 1.0), (9, 1.0), (7, 1.0)],   # a repeated id: its first row counts
        [(7, 1.0), (3, 1.0), (5, 1.0)],
        [(7, 2.0), (5, 1.0)],
    ]
    seg = np.cumsum([0] + [len(g) for g in rows]).astype(np.int64)
    cfg = np.array([c for g in rows for c, _ in g], np.int32)
    rt = np.array([t for g in rows for _, t in g], np.float32)
    best, cnt, mean_y = oracle.static_config(rt, seg, cfg, 16)
    y7 = (0.5 + 1.0 + 0.25 + 1.0 + 0.5) / 5
    y3 = (1.0 + 0.5 + 1.0 + 1.0) / 4
    assert y3 > y7
    assert (best, cnt) == (3, 4) and mean_y == pytest.approx(y3, rel=1e-15)
    # without config 3, config 7 wins; nothing qualifies when every id is rare
    cfg2 = np.where(cfg == 3, 11, cfg)
    cfg2[np.flatnonzero(cfg2 == 11)[0]] = 12
    best2, cnt2, my2 = oracle.static_config(rt, seg, cfg2, 16)
    assert (best2, cnt2) == (7, 5) and my2 == pytest.approx(y7, rel=1e-15)
    best3, _, my3 = oracle.static_config(rt, seg, np.arange(len(cfg), dtype=np.int32), len(cfg))
    assert best3 == -1 and np.isnan(my3)


def test_nan_runtime_reads_as_never_finishing():
    rt = np.array([1.0, np.nan, np.nan, np.nan], np.float32)
    seg = np.array([0, 2, 4], np.int64)
    agg, reg, rank, ybar = oracle.evaluate(rt, seg, np.array([[1], [0]], np.int32))
    assert reg.tolist() == [1.0, 1.0] and rank.tolist() == [2, 1]
    assert ybar.tolist() == [0.5, 0.0]
