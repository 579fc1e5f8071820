"""Pins of the oracle's selection (eq. (selection), generalised to top-k) and
regret (eq. (regret)): brute force with Python's sorted() on small inputs with
heavy ties, NaN and signed zeros; regret invariants; regret 0 when the scores
are the negated runtimes; the uniform-pick expectation."""
import math

import numpy as np
import pytest

import oracle
import synth


def brute_topk(scores, seg, k):
    out = []
    for p in range(len(seg) - 1):
        seg_s = [(float(scores[seg[p] + j]), j) for j in range(seg[p + 1] - seg[p])]
        key = lambda t: (0 if math.isnan(t[0]) else 1, -0.0 if math.isnan(t[0]) else t[0], -t[1])
        order = sorted(seg_s, key=key, reverse=True)
        idx = [j for _, j in order[:k]] + [-1] * max(0, k - len(order))
        out.append(idx)
    return np.array(out, np.int32)


@pytest.mark.parametrize("seed", range(6))
def test_topk_brute_force(seed):
    rng = np.random.default_rng(seed)
    seg = synth.ragged_segments(rng, 25, 40)
    s = synth.random_scores(rng, int(seg[-1]), tie_frac=0.5, n_levels=3)
    s[rng.random(len(s)) < 0.05] = np.nan
    s[rng.random(len(s)) < 0.05] = -0.0
    s[rng.random(len(s)) < 0.05] = 0.0
    s[rng.random(len(s)) < 0.02] = -np.inf
    for k in (1, 3, 16, 64):
        idx, vals = oracle.topk(s, seg, k)
        assert np.array_equal(idx, brute_topk(s, seg, k))
        pad = idx < 0
        assert np.all(np.isneginf(vals[pad]))


def test_topk_all_equal_gives_first_indices():
    seg = np.array([0, 100], np.int64)
    idx, _ = oracle.topk(np.ones(100, np.float32), seg, 7)
    assert idx[0].tolist() == list(range(7))


def test_regret_invariants_and_zero_at_oracle_choice():
    rng = np.random.default_rng(11)
    seg = synth.ragged_segments(rng, 40, 60, empty_frac=0.0)
    rt = np.exp(rng.standard_normal(int(seg[-1]))).astype(np.float32)
    rt[rng.random(len(rt)) < 0.05] = np.inf
    s = rng.standard_normal(len(rt)).astype(np.float32)
    idx, _ = oracle.topk(s, seg, 5)
    r1, rk, best = oracle.regret(rt, seg, idx)
    assert np.all(r1 >= 0) and np.all(r1 <= 1) and np.all(rk <= r1)
    for p in range(len(seg) - 1):
        seg_rt = rt[seg[p]:seg[p + 1]]
        assert best[p] == int(np.argmin(seg_rt))
    # scores = -runtimes selects a measured maximiser: regret exactly 0
    idx0, _ = oracle.topk(-rt, seg, 5)
    r1, rk, _ = oracle.regret(rt, seg, idx0)
    assert np.all(r1 == 0) and np.all(rk == 0)


def test_regret_uniform_pick_expectation():
    """Averaging R over every possible top-1 pick gives 1 - mean_c(t*/t_c),
    the expected regret of a uniform random pick."""
    rng = np.random.default_rng(2)
    n = 50
    rt = np.exp(rng.standard_normal(n)).astype(np.float32)
    seg = np.array([0, n], np.int64)
    rs = [oracle.regret(rt, seg, np.array([[c]], np.int32))[0][0] for c in range(n)]
    t = rt.astype(np.float64)
    assert abs(np.mean(rs) - (1 - np.mean(t.min() / t))) < 1e-6


def test_regret_edge_cases():
    seg = np.array([0, 0, 3], np.int64)
    rt = np.array([np.inf, np.inf, np.inf], np.float32)
    r1, rk, best = oracle.regret(rt, seg, np.array([[-1, -1], [2, 0]], np.int32))
    assert np.isnan(r1[0]) and np.isnan(rk[0]) and best[0] == -1
    # all candidates infeasible: equal (infinite) runtimes give regret 0
    assert r1[1] == 0 and rk[1] == 0 and best[1] == 0
    # a feasible best vs an infeasible pick: regret 1
    rt2 = np.array([1.0, np.inf], np.float32)
    r1, _, _ = oracle.regret(rt2, np.array([0, 2], np.int64), np.array([[1]], np.int32))
    assert r1[0] == 1.0


def test_nan_pick_reads_as_never_finishing():
    """One reading of eq. (regret) for a pick whose runtime is NaN: a kernel
    that never finishes has throughput 0, so R = 1 - 0 / T* = 1 -- in the
    regret call and in the evaluation metrics alike, also when every runtime
    of the group is NaN (no candidate finishes, none is matched)."""
    rt = np.array([1.0, np.nan, 2.0, np.nan, np.nan, 0.5, np.nan], np.float32)
    seg = np.array([0, 3, 5, 7], np.int64)
    idx = np.array([[1, 0], [0, 1], [1, 0]], np.int32)
    r1, rk, best = oracle.regret(rt, seg, idx)
    assert r1.tolist() == [1.0, 1.0, 1.0]
    # best of the two picks: {NaN, 1.0} -> 1.0 = t*; {NaN, NaN} -> 1; {NaN, 0.5} -> 0.5 = t*
    assert rk.tolist() == [0.0, 1.0, 0.0]
    assert best.tolist() == [0, 0, 0]
    _, reg, _, _ = oracle.evaluate(rt, seg, idx[:, :1])
    assert reg.tolist() == r1.astype(np.float64).tolist()
    # a NaN pick next to a finite best equals the regret of an infinitely slow pick
    inf_pick = oracle.regret(np.array([1.0, np.inf], np.float32), np.array([0, 2], np.int64),
                             np.array([[1]], np.int32))[0]
    assert inf_pick[0] == 1.0
