"""Oracle-matching selections on every problem of every workload: the HIP
path end to end at full size (features, then the packed forest as the
benchmark runs it or the matrix-core MLP, then the per-problem top-k of
eq. (selection) generalised to the k best) against the oracle's selections
stored in tests/golden/selections_<name>.npz by make_selections.py, which
calls the oracle alone.

Forest workloads (tiny, medium, full, dataset-scale):
  * leaf paths: the packed traversal's per-row leaf-path fingerprint, summed
    per problem, equals the oracle's for every problem -- every leaf of every
    tree on every row -- and its scores are bit-identical to
    hwsel_forest_score's; the leaf indices it reports for a window of rows
    equal the oracle's;
  * selections: top-k indices equal the oracle's for every problem.  A
    problem may differ only by a near tie, i.e. each differing pick's oracle
    score lies within the forest score bound (1e-5 of the larger of the
    score and the row's leaf L1 norm) of the oracle's k-th score; such
    problems are listed.
MLP workload: every pick of every problem is admissible (its oracle score
is at least the oracle's k-th score minus 4e-2 * max(|k-th|, rms of the
problem's oracle scores), the two-sided band of the 2e-2 score bound); the
number of problems whose top-1 and whole top-k match exactly is reported.
"""
import os
import sys

import numpy as np
import pytest
import torch

import oracle
import synth
from _gpu_util import Dev, path_l1, say
from paper_2609_35587_amd import hwsel

sys.path.insert(0, os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden"))
import make_selections  # noqa: E402

pytestmark = pytest.mark.gpu


def golden(name: str, w) -> dict:
    g = make_selections.load(name)
    assert str(g["fingerprint"]) == make_selections.fingerprint(w), \
        f"stored selections of {name} are stale: rerun tests/golden/make_selections.py {name}"
    return g


def per_problem_sums(h: np.ndarray, seg: np.ndarray) -> np.ndarray:
    return np.array([np.sum(h[seg[p]:seg[p + 1]], dtype=np.uint64) for p in range(len(seg) - 1)], np.uint64)


def explain_forest_mismatch(w, p: int, gpu_idx: np.ndarray, g: dict) -> str | None:
    """None if problem p's differing picks are near ties of the oracle's own
    scores, else a description of the first pick that is not."""
    lo, hi = int(w.seg[p]), int(w.seg[p + 1])
    rows = np.arange(lo, hi, dtype=np.int64)
    Xp = oracle.features(w.hw, w.problems, w.seg, w.cands, w.cfg.n_features, rows)
    s, li = oracle.forest(w.forest, Xp, leaves=True)
    l1 = path_l1(w.forest, li)
    kth = float(g["vals"][p, -1])
    for j in gpu_idx:
        if j in g["idx"][p]:
            continue
        band = 1e-5 * max(abs(float(s[j])), float(l1[j]), abs(kth))
        if float(s[j]) < kth - 2 * band:
            return f"pick {j}: oracle score {s[j]} vs k-th {kth} (band {band})"
    return None


@pytest.mark.parametrize("name", ["tiny", "medium", "full", "dataset"])
def test_forest_selection_every_problem(name):
    say(f"{name}: generate")
    w = synth.workload(name)
    cfg = w.cfg
    g = golden(name, w)
    d = Dev(w)
    say(f"{name}: features R={cfg.rows} F={cfg.n_features}")
    X = d.features(cfg.n_features)
    packed = hwsel.hwsel_forest_pack(d.forest)
    ws = torch.empty(hwsel.hwsel_forest_workspace_bytes(d.forest, cfg.rows), dtype=torch.uint8, device="cuda")
    say(f"{name}: packed forest {cfg.trees}x{cfg.depth} with leaf fingerprints")
    row0 = max(0, cfg.rows // 2 - 300)
    n_win = min(cfg.rows - row0, 777)
    s_chk, lh, li = hwsel.hwsel_forest_score_checked(d.forest, X, packed, leaf_rows=(row0, n_win), workspace=ws)
    s = hwsel.hwsel_forest_score(d.forest, X, packed=packed, workspace=ws)
    assert torch.equal(s_chk.view(torch.int32), s.view(torch.int32)), "checked traversal changed the scores"
    # every leaf of every tree on every row, per problem
    sums = per_problem_sums(lh.cpu().numpy().view(np.uint64), w.seg)
    bad = np.flatnonzero(sums != g["leaf_hash"])
    assert len(bad) == 0, f"leaf paths differ from the oracle's in problems {bad[:10].tolist()} ({len(bad)} in all)"
    say(f"  leaf paths equal the oracle's on all {cfg.n_problems} problems ({cfg.rows} rows x {cfg.trees} trees)")
    # the reported leaf indices of a window of rows (crossing row tiles)
    rows = np.arange(row0, row0 + n_win, dtype=np.int64)
    Xw = X[row0:row0 + n_win].cpu().numpy()
    _, oli = oracle.forest(w.forest, Xw, leaves=True)
    assert np.array_equal(li.cpu().numpy().view(np.uint16), oli), "leaf indices of the window differ"
    del rows
    say(f"{name}: top-{cfg.k} per problem")
    idx = hwsel.hwsel_topk_per_problem(s, d.seg, cfg.k, with_vals=False)[0].cpu().numpy()
    differ = [p for p in range(cfg.n_problems) if not np.array_equal(idx[p], g["idx"][p])]
    for p in differ:
        why = explain_forest_mismatch(w, p, idx[p], g)
        assert why is None, f"problem {p}: {why}"
        say(f"  problem {p}: differs from the oracle only by a near tie")
    say(f"  selections equal the oracle's on {cfg.n_problems - len(differ)} of {cfg.n_problems} problems"
        f" (the rest near ties)")


def test_mlp_selection_every_problem():
    say("mlp: generate")
    w = synth.workload("mlp")
    cfg = w.cfg
    g = golden("mlp", w)
    d = Dev(w)
    X = d.features(128)
    say("mlp: matrix-core path on all rows (as benchmarked)")
    s = hwsel.hwsel_mlp_score(d.mlp, X, packed=hwsel.hwsel_mlp_pack(d.mlp))
    idx = hwsel.hwsel_topk_per_problem(s, d.seg, cfg.k, with_vals=False)[0].cpu().numpy()
    # oracle scores of every GPU pick, from the oracle's own features
    rows = (w.seg[:-1, None] + idx).reshape(-1).astype(np.int64)
    Xo = oracle.features(w.hw, w.problems, w.seg, w.cands, 128, rows)
    o_pick = oracle.mlp(w.mlp, Xo).reshape(idx.shape).astype(np.float64)
    kth = g["vals"][:, -1].astype(np.float64)
    band = 4e-2 * np.maximum(np.abs(kth), g["rms"])
    ok = o_pick >= (kth - band)[:, None]
    bad = np.argwhere(~ok)
    assert len(bad) == 0, (f"inadmissible picks (problem, rank): {bad[:5].tolist()}; "
                           f"oracle score {o_pick[tuple(bad[0])]} vs k-th {kth[bad[0][0]]}")
    top1 = int(np.sum(idx[:, 0] == g["idx"][:, 0]))
    topk = int(sum(np.array_equal(idx[p], g["idx"][p]) for p in range(cfg.n_problems)))
    same_set = int(sum(set(idx[p]) == set(g["idx"][p]) for p in range(cfg.n_problems)))
    say(f"  all {idx.size} picks admissible; top-1 equal on {top1}/{cfg.n_problems} problems, "
        f"top-{cfg.k} equal on {topk}, same set on {same_set}")
