"""Runs in a subprocess of tests/test_sanitize.py with a sanitizer runtime
preloaded: argv[1] = "oracle" (oracle/ built with AddressSanitizer and
UBSan) or "library" (libhwsel.so with its host code built with both).
Exercises the code on small inputs and exits non-zero on any mismatch; a
sanitizer finding aborts the process by itself."""
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402


def run_oracle(lib_path: str) -> None:
    import oracle
    import synth
    oracle.LIB = lib_path
    w = synth.workload("tiny")
    X = oracle.features(w.hw, w.problems, w.seg, w.cands, 64)
    X96 = oracle.features(w.hw, w.problems, w.seg, w.cands, 96, rows=np.arange(0, w.cfg.rows, 7))
    X128 = oracle.features(w.hw, w.problems, w.seg, w.cands, 128, rows=np.arange(0, w.cfg.rows, 5))
    s, li, lh = oracle.forest(w.forest, X, leaves=True, leaf_hash=True)
    assert np.array_equal(oracle.forest_linked(w.forest, X), s)
    idx, vals = oracle.topk(s, w.seg, w.cfg.k)
    r1, rk, best = oracle.regret(w.runtimes, w.seg, idx)
    agg, reg, rank, ybar = oracle.evaluate(w.runtimes, w.seg, idx)
    ids = w.extra["config_id"]
    oracle.static_config(w.runtimes, w.seg, ids, int(ids.max()) + 1)
    m = synth.mlp(synth.CONFIGS["mlp"])
    sm = oracle.mlp(m, X128[:64])
    oracle.mlp(m, X128[:16], exact=True)
    mask, n_valid = oracle.catalogue_mask(w.hw, w.problems[:2], 1)
    oracle.catalogue_compact(mask)
    oracle.catalogue_decode(np.arange(0, 534600, 997), 0)
    lin = synth.linear(synth.CONFIGS["medium"])
    oracle.linear(lin, X96)
    print("oracle ok", float(s.sum()), int(lh[0]), float(r1.mean()), agg["mean_regret"], float(sm[0]), X.shape)


def run_library(lib_path: str) -> None:
    import ctypes as C
    from paper_2609_35587_amd import hwsel
    hwsel.LIB_PATH = lib_path
    L = hwsel.lib()
    # every host-side rejection path of the C ABI (nothing reaches the GPU)
    sys.path.insert(0, os.path.join(ROOT, "tests"))
    import test_abi
    import pytest  # noqa: F401
    names = [n for n in dir(test_abi) if n.startswith("test_") and "missing_library" not in n
             and "host_tensors" not in n and "exports" not in n]
    import inspect
    for n in names:
        fn = getattr(test_abi, n)
        params = inspect.signature(fn).parameters
        marks = getattr(fn, "pytestmark", [])
        cases = [m for m in marks if m.name == "parametrize"]
        if not cases:
            fn(L) if "L" in params else fn()
            continue
        argnames = [a.strip() for a in cases[0].args[0].split(",")]
        for vals in cases[0].args[1]:
            vals = vals if isinstance(vals, tuple) and len(argnames) > 1 else (vals,)
            kw = dict(zip(argnames, vals))
            fn(L, **kw) if "L" in params else fn(**kw)
    # the host forest packer on random forests of every packable depth
    rng = np.random.default_rng(3)
    for depth in range(1, 11):
        T, F = int(rng.integers(1, 70)), int(rng.integers(1, 129))
        n_int = (1 << depth) - 1
        f = dict(n_trees=T, depth=depth, n_features=F, flags=int(rng.integers(0, 2)), base_score=0.0,
                 node_feature=rng.integers(0, F, (T, n_int)).astype(np.uint8),
                 node_threshold=rng.integers(-120, 120, (T, n_int)).astype(np.float32) / 7,
                 leaf_value=rng.standard_normal((T, n_int + 1)).astype(np.float32))
        a, b = hwsel.hwsel_forest_pack_host(f), hwsel.hwsel_forest_pack_host(f)
        assert np.array_equal(a, b)
        hdr = a[:28].view(np.int32)
        assert hdr[0] == 0x48575346 and hdr[2] == T and hdr[3] == depth and hdr[4] == F
    bad = dict(f, node_feature=np.full_like(f["node_feature"], 200))
    try:
        hwsel.hwsel_forest_pack_host(dict(bad, n_features=100))
        raise AssertionError("a node feature past n_features was packed")
    except hwsel.HwselError as e:
        assert e.status == 1
    del C
    print("library ok")


if __name__ == "__main__":
    {"oracle": run_oracle, "library": run_library}[sys.argv[1]](sys.argv[2])
