"""Pins of the oracle's configuration catalogue (section "Configuration
Space", Table "Configuration knobs"; section "Validity Constraints", Table
"Static validity constraints").

The raw count is the printed 534,600 per layout and 2,138,400 over the four
layouts (tests/golden/printed_counts.txt).  Decoding is a bijection onto the
Table's value sets, first knob slowest.  Each validity predicate is checked
on hand-built boundary cases and against the feature map's validity columns
(86: shape guard, 87: the Table's predicates).  The paper's valid counts
(242,971 over the catalogue, 60,795 for one shape) rest on rules it does not
list: the valid counts are parity unpinned."""
import os

import numpy as np
import pytest

import oracle
import synth

HERE = os.path.dirname(os.path.abspath(__file__))
DOMAINS = {"tile_m": [64, 128, 192, 256], "tile_n": [16, 32, 48, 64, 80, 96, 128, 192, 256],
           "tile_k": [32, 64, 128, 256, 512], "stages": list(range(2, 13))}


def printed():
    out = {}
    for line in open(os.path.join(HERE, "golden", "printed_counts.txt")):
        if line.strip() and not line.startswith("#"):
            k, v = line.split()
            out[k] = float(v)
    return out


@pytest.fixture(scope="module")
def decoded():
    return oracle.catalogue_decode(np.arange(oracle.catalogue_size()), synth.DTYPE_BF16)


def test_raw_counts_match_the_printed_ones():
    p = printed()
    assert oracle.catalogue_size() == p["raw_per_layout"]
    assert 4 * oracle.catalogue_size() == p["raw_all_layouts"]


def test_decode_is_a_bijection_onto_the_table(decoded):
    d = decoded
    keys = np.stack([d[n].astype(np.int64) for n in ("tile_m", "tile_n", "tile_k", "stages", "cluster_m",
                                                     "cluster_n", "kernel_sched", "epi_sched", "tile_sched")], 1)
    assert len(np.unique(keys, axis=0)) == len(keys)
    n = len(keys)
    for f, dom in DOMAINS.items():
        vals, cnt = np.unique(d[f], return_counts=True)
        assert vals.tolist() == dom and np.all(cnt == n // len(dom))
    pairs = set(zip(d["cluster_m"].tolist(), d["cluster_n"].tolist()))
    assert pairs == {(a, b) for a in (1, 2, 4, 8, 16) for b in (1, 2, 4, 8, 16) if a * b <= 16}
    for f, k in (("kernel_sched", 3), ("epi_sched", 3), ("tile_sched", 2)):
        assert np.unique(d[f]).tolist() == list(range(k))
    # first knob slowest, last fastest
    assert np.all(d["tile_m"][: n // 4] == 64) and np.all(d["tile_m"][-n // 4:] == 256)
    assert d["tile_sched"][:4].tolist() == [0, 1, 0, 1]
    assert np.all(d["inst_n"] == d["tile_n"]) and np.all(d["inst_m_div16"] == 4) and np.all(d["swizzle"] == 1)
    assert np.all(d["inst_k"] == 16)
    assert np.all(oracle.catalogue_decode([0, 1000], synth.DTYPE_FP8)["inst_k"] == 32)


def one(M=4096, N=4096, K=4096, layout=0, dtype=0):
    pr = np.zeros(1, synth.PROBLEM_DTYPE)
    pr["M"], pr["N"], pr["K"], pr["layout"], pr["dtype"] = M, N, K, layout, dtype
    return pr


def find(d, **kv):
    m = np.ones(len(d["tile_m"]), bool)
    for k, v in kv.items():
        m &= d[k] == v
    return np.flatnonzero(m)


def valid(pr, i, flags=0):
    mask, _ = oracle.catalogue_mask(synth.hardware(), pr, flags)
    return bool(mask[0, i])


def test_predicates_on_boundary_cases(decoded):
    d = decoded
    base = dict(tile_m=128, tile_n=128, tile_k=64, cluster_m=1, cluster_n=1, epi_sched=0)
    # Stream-K needs the cooperative mainloop
    i = find(d, stages=4, kernel_sched=0, tile_sched=1, **base)[0]
    j = find(d, stages=4, kernel_sched=2, tile_sched=1, **base)[0]
    assert not valid(one(), i) and valid(one(), j)
    # cooperative needs T_M % 128 == 0
    for tm, ok in ((64, False), (192, False), (256, True)):
        k = find(d, stages=2, kernel_sched=2, tile_sched=0, **dict(base, tile_m=tm))[0]
        assert valid(one(), k) == ok, tm
    # shared memory: S (T_M + T_N) T_K 2 + 2048 <= 232,448: 7 stages of 32 KiB fit, 8 do not
    for st, ok in ((7, True), (8, False)):
        k = find(d, stages=st, kernel_sched=0, tile_sched=0, **base)[0]
        assert valid(one(), k) == ok, st
    # K-box limits: A column-major (NN, NT) needs T_K <= 256 C_N; B row-major (TT, NT) T_K <= 256 C_M
    big = dict(tile_m=64, tile_n=16, tile_k=512, stages=2, kernel_sched=0, epi_sched=0, tile_sched=0)
    k11 = find(d, cluster_m=1, cluster_n=1, **big)[0]
    k12 = find(d, cluster_m=1, cluster_n=2, **big)[0]
    k21 = find(d, cluster_m=2, cluster_n=1, **big)[0]
    assert valid(one(layout=0), k11)                              # TN: no limit
    assert not valid(one(layout=2), k11) and valid(one(layout=2), k12)   # NN
    assert not valid(one(layout=1), k11) and valid(one(layout=1), k21)   # TT
    assert not valid(one(layout=3), k12) and not valid(one(layout=3), k21)  # NT needs both
    # shape guard (flags bit 0): T_N <= 2M and T_N <= 2N
    k = find(d, stages=2, kernel_sched=0, tile_sched=0, **dict(base, tile_n=256))[0]
    assert valid(one(M=100), k) and not valid(one(M=100), k, flags=1) and valid(one(M=128), k, flags=1)


def test_mask_agrees_with_feature_validity_columns(decoded):
    rng = np.random.default_rng(9)
    hw = synth.hardware()
    for layout, dtype, M, N in ((0, 0, 4096, 4096), (2, 1, 96, 8192), (3, 2, 7000, 40), (1, 0, 512, 512)):
        pr = one(M=M, N=N, K=1000, layout=layout, dtype=dtype)
        mask, cnt = oracle.catalogue_mask(hw, pr, 0)
        mask_g, cnt_g = oracle.catalogue_mask(hw, pr, 1)
        assert cnt[0] == mask[0].sum() and cnt_g[0] == mask_g[0].sum() and cnt_g[0] <= cnt[0]
        sel = rng.choice(oracle.catalogue_size(), 4000, replace=False)
        c = oracle.catalogue_decode(sel, dtype)
        X = oracle.features(hw, pr, np.array([0, len(sel)]), c, 96)
        assert np.array_equal(mask[0, sel], X[:, 87] == 1)
        assert np.array_equal(mask_g[0, sel], (X[:, 87] == 1) & (X[:, 86] == 1))


def test_compaction_is_ordered_and_complete():
    hw = synth.hardware()
    pr = np.concatenate([one(M=64, N=4096), one(layout=3, dtype=2)])
    mask, cnt = oracle.catalogue_mask(hw, pr, 1)
    seg, idx = oracle.catalogue_compact(mask)
    assert seg.tolist() == [0, cnt[0], cnt[0] + cnt[1]]
    for p in range(2):
        part = idx[seg[p]:seg[p + 1]]
        assert np.all(np.diff(part) > 0) and np.all(mask[p, part] == 1)
