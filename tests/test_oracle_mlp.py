"""Pins of the oracle's feed-forward ranker (section "Model B"): bf16 rounding
against its definition on hand-picked bit patterns, zero weights (output =
output bias), a one-hot network whose output has a closed form, and the
unrounded binary64 network within the bf16 error bound."""
import math

import numpy as np
import pytest

import oracle
import synth


def test_bf16_round_to_nearest_even():
    f = lambda u: np.array([u], np.uint32).view(np.float32)[0]
    # exactly half way between two bf16 values: ties go to the even mantissa
    assert oracle.bf16_round(f(0x3F808000)) == f(0x3F800000)
    assert oracle.bf16_round(f(0x3F818000)) == f(0x3F820000)
    assert oracle.bf16_round(f(0x3F808001)) == f(0x3F810000)
    assert oracle.bf16_round(f(0x3F807FFF)) == f(0x3F800000)
    assert oracle.bf16_round(1.0) == 1.0 and oracle.bf16_round(-2.5) == -2.5
    assert math.isinf(oracle.bf16_round(f(0x7F7FFFFF)))   # rounds up to +inf
    assert math.isnan(oracle.bf16_round(float("nan")))


def _zero_mlp():
    m = {}
    for l, (fi, fo) in enumerate(zip(synth.MLP_WIDTHS[:-1], synth.MLP_WIDTHS[1:])):
        m[f"W{l + 1}"] = np.zeros((fo, fi), np.uint16)
        m[f"b{l + 1}"] = np.zeros(fo, np.float32)
    m["mean"] = np.zeros(128, np.float32)
    m["inv_std"] = np.ones(128, np.float32)
    return m


def _bf16(x):
    return (np.asarray(x, np.float32).view(np.uint32) >> 16).astype(np.uint16)


def test_zero_weights_give_output_bias():
    m = _zero_mlp()
    m["b4"] = np.array([0.3125], np.float32)
    X = np.random.default_rng(0).standard_normal((9, 128)).astype(np.float32)
    assert np.all(oracle.mlp(m, X) == np.float32(0.3125))


def gelu(a):
    return 0.5 * a * (1 + math.erf(a / math.sqrt(2)))


def test_one_hot_chain_closed_form():
    """W1 row 0 picks input 0; W2 row 0 and W3 row 0 pick unit 0; W4 reads
    unit 0: s = G(G(G(z0 + b1) + b2) + b3) + b4 with bf16 rounding after each
    GELU (z0 exactly representable)."""
    m = _zero_mlp()
    for l in (1, 2, 3):
        m[f"W{l}"][0, 0] = _bf16(1.0)
    m["W4"][0] = _bf16(1.0)
    m["b1"][0], m["b2"][0], m["b3"][0], m["b4"][0] = 0.25, -0.5, 0.125, 1.0
    m["mean"][0], m["inv_std"][0] = 1.0, 2.0
    X = np.zeros((4, 128), np.float32)
    X[:, 0] = [1.0, 1.5, 0.0, np.inf]
    got = oracle.mlp(m, X)
    for r, x0 in enumerate([1.0, 1.5, 0.0, 0.0]):    # inf is read as 0
        z = (x0 - 1.0) * 2.0
        h = z
        for b in (0.25, -0.5, 0.125):
            h = oracle.bf16_round(np.float32(gelu(h + b)))
        assert got[r] == np.float32(h + 1.0)


def test_rounded_network_within_bf16_bound_of_exact():
    w = synth.workload("tiny", with_runtimes=False, with_model=False)
    cuts = synth.load_cuts("dataset")
    m = synth.mlp(synth.CONFIGS["mlp"], cuts)
    X = np.random.default_rng(1).standard_normal((256, 128)).astype(np.float32)
    X = X / np.where(m["inv_std"] > 0, m["inv_std"], 1.0) + m["mean"]
    a = oracle.mlp(m, X)
    e = oracle.mlp(m, X, exact=True)
    rms = float(np.sqrt(np.mean(e.astype(np.float64) ** 2)))
    # four bf16 roundings (input + 3 hidden layers), 2^-9 relative each
    assert np.all(np.abs(a - e) <= 4 * 2.0 ** -8 * np.maximum(np.abs(e), rms) + 1e-6)
    assert np.max(np.abs(a - e)) > 0   # the rounding is really applied
