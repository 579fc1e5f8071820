"""Shared helpers of the GPU parity tests: upload a seeded workload, compare
with the oracle's acceptance rules."""
from __future__ import annotations

import sys

import numpy as np
import torch

import oracle
from paper_2609_35587_amd import hwsel

INT_COLS_T1 = [4, 5, 6, 7, 8, 9, 10, 11, 12, 13, 14, 15, 20, 22, 23, 24, 25, 26, 27, 29, 30, 31, 32, 33, 36,
               37, 38, 42, 48, 49, 56, 57, 59, 60, 61, 62, 63]
INT_COLS_T2 = [64, 65, 66, 67, 68, 69, 70, 71, 72, 73, 74, 75, 76, 77, 78, 79, 82, 83, 84, 85, 86, 87, 88, 89,
               93, 94, 95]
INT_COLS_T3 = [96, 97, 98, 99, 100, 101, 102, 103, 105, 106, 107, 108, 109, 110, 114, 116, 118, 125]


def int_cols(F: int) -> list[int]:
    return [c for c in INT_COLS_T1 + INT_COLS_T2 + INT_COLS_T3 if c < F]


def say(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


class Dev:
    """A workload's arrays in device memory."""

    def __init__(self, w, device="cuda"):
        self.w = w
        self.problems = hwsel.to_device(w.problems, device)
        self.seg = hwsel.to_device(w.seg, device)
        self.cands = {k: hwsel.to_device(v, device) for k, v in w.cands.items()}
        self.runtimes = hwsel.to_device(w.runtimes, device) if w.runtimes is not None else None
        self.forest = forest_to_device(w.forest, device) if w.forest is not None else None
        self.mlp = mlp_to_device(w.mlp, device) if w.mlp is not None else None

    def features(self, F: int) -> torch.Tensor:
        return hwsel.hwsel_features(self.w.hw, self.problems, self.seg, self.cands, F)


def forest_to_device(f: dict, device="cuda") -> dict:
    out = dict(f)
    for k in ("node_feature", "node_threshold", "leaf_value"):
        out[k] = hwsel.to_device(np.ascontiguousarray(f[k]), device)
    return out


def mlp_to_device(m: dict, device="cuda") -> dict:
    return {k: hwsel.to_device(np.ascontiguousarray(v), device) for k, v in m.items()}


def compare_features(gpu: np.ndarray, ref: np.ndarray, F: int) -> dict:
    """Integer columns bit-exact; the rest within 1e-6 relative.  Returns
    counts of rows that differ at all (for the report)."""
    ic = int_cols(F)
    g_i, r_i = gpu[:, ic], ref[:, ic]
    bad = np.argwhere(g_i.view(np.uint32) != r_i.view(np.uint32))
    assert len(bad) == 0, f"integer columns differ at (row, col) {[(int(a), ic[b]) for a, b in bad[:5]]}"
    rel = np.abs(gpu.astype(np.float64) - ref) / np.maximum(np.abs(ref.astype(np.float64)), 1e-30)
    worst = np.unravel_index(np.argmax(rel), rel.shape)
    assert rel.max() <= 1e-6, f"float column {worst[1]} row {worst[0]}: {gpu[worst]} vs {ref[worst]}"
    not_bitexact = int((gpu.view(np.uint32) != ref.view(np.uint32)).sum())
    return dict(max_rel=float(rel.max()), not_bitexact=not_bitexact)


def path_l1(forest: dict, leaves: np.ndarray) -> np.ndarray:
    """Sum over trees of |leaf value| along each row's path."""
    lv = np.abs(forest["leaf_value"].astype(np.float64))
    T = lv.shape[0]
    return lv[np.arange(T)[None, :], leaves.astype(np.int64)].sum(axis=1)


def assert_forest_scores(g: np.ndarray, o: np.ndarray, l1: np.ndarray, tol: float = 1e-5) -> float:
    bound = tol * np.maximum(np.abs(o.astype(np.float64)), l1)
    err = np.abs(g.astype(np.float64) - o)
    i = int(np.argmax(err - bound))
    assert np.all(err <= bound), f"row {i}: gpu {g[i]} oracle {o[i]} bound {bound[i]}"
    return float((err / np.maximum(bound, 1e-30)).max())


def check_selection(w, idx, problems):
    """The GPU's per-problem choice (idx [P][k], from the GPU's own scores)
    against the oracle's features -> forest -> top-k on every row of the given
    problems.  The forest's fp32 leaf sums may order two candidates whose
    oracle scores lie within the score tolerance differently: such a swap is
    accepted only when it is explained by that near-tie."""
    cfg = w.cfg
    for p in problems:
        rows = np.arange(w.seg[p], w.seg[p + 1], dtype=np.int64)
        Xp = oracle.features(w.hw, w.problems, w.seg, w.cands, cfg.n_features, rows)
        o, oli = oracle.forest(w.forest, Xp, leaves=True)
        oidx, _ = oracle.topk(o, np.array([0, len(rows)], np.int64), cfg.k)
        if np.array_equal(idx[p], oidx[0]):
            continue
        tol = 2e-5 * np.maximum(np.abs(o.astype(np.float64)), path_l1(w.forest, oli))
        for a, b in zip(idx[p], oidx[0]):
            if a != b:
                assert abs(float(o[a]) - float(o[b])) <= tol[a] + tol[b], f"problem {p}: {a} vs {b}"
        say(f"  problem {p}: order differs only on near-ties")
