"""The matrix-core MLP kernel's GELU, checked on the CPU.

The kernel evaluates GELU(a) = max(a, 0) - |a| 2^P(|a|), P a fitted cubic
standing in for log2 Phi(-x).  This test reads P's coefficients
from the kernel source, evaluates the same fp32 Horner steps (each FMA
rounded once) and compares with GELU(a) = a Phi(a) computed from erfc in
binary64.  It pins the error bound the source states, the behaviour past the
fitted range (P keeps falling and the result becomes exactly max(a, 0)) and
that the approximation moves no more bf16 roundings than its error bound
allows.  The bound, 8.2e-5, is a twentieth of the bf16 half-step at 1: the
kernel rounds every activation to bf16 right after GELU.
"""
import math
import pathlib
import re

import numpy as np

SRC = pathlib.Path(__file__).resolve().parents[1] / "paper_2609_35587_amd" / "csrc" / "mlp.hip"
BOUND = 8.2e-5      # |kernel GELU - GELU| for every finite argument


def coefficients():
    text = SRC.read_text()
    body = text[text.index("float gelu_fast(float a)"):]
    body = body[:body.index("}")]
    found = dict(re.findall(r"\b(c[0-9])\s*=\s*([-+0-9.eE]+)f", body))
    deg = len(found) - 1
    assert sorted(found) == [f"c{i}" for i in range(deg + 1)]
    return [np.float32(float(found[f"c{i}"])) for i in range(deg, -1, -1)]


def fma32(a, b, c):
    # fp32 FMA: the exact product-sum of fp32 inputs, rounded once (binary64
    # holds the product of two fp32 values exactly; the sum's double
    # rounding is harmless at this error scale)
    # (P overflows to -inf for huge |a|, as in fp32 on the GPU, and 2^-inf = 0)
    with np.errstate(over="ignore", invalid="ignore"):
        return (a.astype(np.float64) * b.astype(np.float64) + c.astype(np.float64)).astype(np.float32)


def kernel_gelu(a):
    a = np.asarray(a, dtype=np.float32)
    c = coefficients()
    x = np.abs(a)
    p = fma32(np.full_like(x, c[0]), x, np.full_like(x, c[1]))
    for ci in c[2:]:
        p = fma32(p, x, np.full_like(x, ci))
    with np.errstate(over="ignore", under="ignore"):
        e = np.exp2(p.astype(np.float64)).astype(np.float32)
    return fma32(-x, e, np.maximum(a, np.float32(0.0)))


def gelu_exact(a):
    a = np.asarray(a, dtype=np.float64)
    erfc = np.vectorize(math.erfc)
    return a * (1.0 - 0.5 * erfc(a / math.sqrt(2.0)))


def test_error_bound_over_the_working_range():
    a = np.linspace(-12.0, 12.0, 480001, dtype=np.float32)
    err = np.abs(kernel_gelu(a).astype(np.float64) - gelu_exact(a))
    assert err.max() <= BOUND, (float(err.max()), float(a[err.argmax()]))


def test_large_arguments_give_relu_exactly():
    a = np.concatenate([np.geomspace(12.0, 3e38, 2000), -np.geomspace(12.0, 3e38, 2000)]).astype(np.float32)
    g = kernel_gelu(a)
    assert np.all(np.isfinite(g))
    big = np.abs(a) >= 20.0
    assert np.array_equal(g[big], np.maximum(a[big], 0.0))
    err = np.abs(g.astype(np.float64) - gelu_exact(a))
    assert np.all(err <= BOUND * np.maximum(1.0, np.abs(a)))


def test_special_values():
    g = kernel_gelu(np.array([0.0, -0.0, 1.0, -1.0], dtype=np.float32))
    assert g[0] == 0.0 and g[1] == 0.0
    assert abs(float(g[2]) - 0.8413447460685429) <= BOUND     # Phi(1)
    assert abs(float(g[3]) + 0.15865525393145707) <= BOUND    # -Phi(-1)


def test_bf16_roundings_move_only_near_a_boundary():
    """Rounded to bf16 (as the kernel stores activations), the approximation
    and the exact GELU differ only where the exact value lies within the
    error bound of a rounding boundary, and then by at most the bound plus one
    bf16 step.  Where |GELU| is small the bf16 step is at or below the bound,
    so moves are common there (and worth at most the bound plus one small
    step); from |GELU| = 1 on, where a step is 2^-7 or more, at most a
    fraction 2 * bound / 2^-7 of the values can lie that close to a boundary."""
    rng = np.random.default_rng(7)
    a = (rng.standard_normal(400000) * 3).astype(np.float32)

    def bf16(v):
        u = np.asarray(v, dtype=np.float32).view(np.uint32).astype(np.uint64)
        u = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
        return u.astype(np.uint32).view(np.float32)

    g = kernel_gelu(a)
    exact = gelu_exact(a)
    moved = bf16(g) != bf16(exact.astype(np.float32))
    near = bf16((exact - BOUND).astype(np.float32)) != bf16((exact + BOUND).astype(np.float32))
    assert np.all(near[moved])
    step = np.abs(bf16(g)[moved].astype(np.float64) - bf16(exact.astype(np.float32))[moved])
    assert np.all(step <= BOUND + np.abs(exact[moved]) * 2.0 ** -7)
    large = np.abs(exact) >= 1.0
    assert moved[large].mean() <= 2 * BOUND / 2.0 ** -7, float(moved[large].mean())


def test_coefficients_come_from_the_committed_fit():
    """The kernel's coefficients are what csrc/gelu_fit.py produces (fp32),
    and the fit's own error check gives the bound the source states."""
    import importlib.util
    spec = importlib.util.spec_from_file_location("gelu_fit", SRC.parent / "gelu_fit.py")
    fit = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(fit)
    c = fit.fit()
    assert [np.float32(v) for v in c] == coefficients()
    err, _ = fit.max_error(c)
    assert err <= BOUND
