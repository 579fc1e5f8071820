"""Pins of the oracle's cheap scorers.

Linear ridge scorer (section "Linear Ridge Baseline", eq. ridge-loss):
special cases with known values (zero weights give the bias; one numeric
column gives bias + its standardised value; one-hot-only models give bias +
the level's weight; unseen levels encode to zeros; non-finite inputs read as
0 before scaling) and linearity in the weights.

Analytic sampling score (section "Candidate Sampling"): a hand-computed
value and its monotonicity in the stage count, through feature column 58.
"""
import math

import numpy as np
import pytest

import oracle
import synth

ONEHOT_COLS = {64: (0, 4), 73: (4, 3), 74: (7, 3), 75: (10, 2)}


def model(F, rng=None, zero=False):
    rng = rng or np.random.default_rng(0)
    m = {"n_features": F, "bias": 0.25,
         "mean": rng.normal(0, 1, F).astype(np.float32),
         "inv_std": rng.uniform(0.5, 2, F).astype(np.float32),
         "w": rng.normal(0, 1, F).astype(np.float32),
         "w_onehot": rng.normal(0, 1, 12).astype(np.float32)}
    if zero:
        m["w"][:] = 0
        m["w_onehot"][:] = 0
    return m


@pytest.mark.parametrize("F", [64, 96, 128])
def test_zero_weights_give_bias(F):
    X = np.random.default_rng(1).normal(0, 10, (50, F)).astype(np.float32)
    s, mag = oracle.linear(model(F, zero=True), X)
    assert np.all(s == np.float32(0.25))
    assert np.all(mag == 0.25)


@pytest.mark.parametrize("F", [64, 128])
def test_single_numeric_column(F):
    rng = np.random.default_rng(2)
    m = model(F, zero=True)
    j = 5
    m["w"][j] = 1.0
    m["mean"][j] = 0.0
    m["inv_std"][j] = 1.0
    X = rng.normal(0, 3, (100, F)).astype(np.float32)
    s, _ = oracle.linear(m, X)
    assert np.array_equal(s, (0.25 + X[:, j].astype(np.float64)).astype(np.float32))


def test_nonfinite_inputs_read_as_zero():
    m = model(128, zero=True)
    j = 7
    m["w"][j], m["mean"][j], m["inv_std"][j] = 2.0, 1.5, 0.5
    X = np.zeros((4, 128), np.float32)
    X[:, j] = [np.nan, np.inf, -np.inf, 0.0]
    s, _ = oracle.linear(m, X)
    assert np.all(s == np.float32(0.25 + 2.0 * (0.0 - 1.5) * 0.5))


def test_onehot_levels_and_unseen_values():
    m = model(96, zero=True)
    m["w_onehot"][:] = np.arange(1, 13, dtype=np.float32) * 10
    X = np.zeros((1, 96), np.float32)
    for col, (first, levels) in ONEHOT_COLS.items():
        for lv in range(levels):
            x = X.copy()
            x[0, col] = lv
            other = {c for c in ONEHOT_COLS if c != col}
            for c in other:
                x[0, c] = -1.0          # outside every level set: adds nothing
            s, _ = oracle.linear(m, x)
            assert s[0] == np.float32(0.25 + (first + lv + 1) * 10), (col, lv)
        for bad in (levels, 0.5, -1.0, np.nan):
            x = np.full((1, 96), -1.0, np.float32)
            x[0, col] = bad
            s, _ = oracle.linear(m, x)
            assert s[0] == np.float32(0.25), (col, bad)


def test_sixty_four_columns_have_no_categorical_part():
    m = model(64, zero=True)
    m["w_onehot"][:] = 100.0
    X = np.zeros((3, 64), np.float32)
    s, _ = oracle.linear(m, X)
    assert np.all(s == np.float32(0.25))


def test_linear_in_the_weights():
    rng = np.random.default_rng(3)
    X = rng.normal(0, 2, (200, 128)).astype(np.float32)
    X[:, 64] = rng.integers(0, 4, 200)
    X[:, 73] = rng.integers(0, 3, 200)
    a, b = model(128, rng), model(128, rng)
    for m in (a, b):
        m["mean"], m["inv_std"] = a["mean"], a["inv_std"]
        m["bias"] = 0.0
    ab = dict(a, w=(a["w"].astype(np.float64) + b["w"]).astype(np.float32),
              w_onehot=(a["w_onehot"].astype(np.float64) + b["w_onehot"]).astype(np.float32))
    sa, ma = oracle.linear(a, X)
    sb, mb = oracle.linear(b, X)
    sab, _ = oracle.linear(ab, X)
    tol = 2e-6 * (ma + mb) + 1e-30
    assert np.all(np.abs(sab.astype(np.float64) - (sa.astype(np.float64) + sb)) <= tol)


def test_sampling_score_hand_value():
    # 128 x 128 x 64 tile, 4 stages, 1 x 1 cluster on a 4096^3 problem, 132 SMs:
    # n_c = 32 * 32 = 1024 clusters, S_SM = 132 slots, W = ceil(1024/132) = 8,
    # s = 1024 / (8 * 132) * 4 * sqrt(128 * 128 * 64) = 1024 * 4 * 1024 / 1056.
    hw = synth.hardware()
    probs = np.zeros(1, synth.PROBLEM_DTYPE)
    probs["M"], probs["N"], probs["K"] = 4096, 4096, 4096
    c = {n: np.zeros(1, dt) for n, dt in synth.CAND_FIELDS}
    c["tile_m"][:], c["tile_n"][:], c["tile_k"][:], c["inst_n"][:] = 128, 128, 64, 128
    c["stages"][:], c["cluster_m"][:], c["cluster_n"][:], c["swizzle"][:] = 4, 1, 1, 1
    c["inst_m_div16"][:], c["inst_k"][:] = 4, 16
    X = oracle.features(hw, probs, np.array([0, 1]), c, 64)
    assert X[0, 58] == np.float32(1024 * 4 * 1024 / 1056)
    c["stages"][:] = 5
    X5 = oracle.features(hw, probs, np.array([0, 1]), c, 64)
    assert X5[0, 58] == np.float32(1024 * 5 * 1024 / 1056)
