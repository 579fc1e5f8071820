"""Write tests/golden/forest_cuts_<workload>.npz from the oracle alone.

For each forest workload (tiny, medium, full, dataset) a seeded sample of up
to 65,536 rows is featurised by the CPU oracle.  Per column it stores:

* ``cuts`` [F][255] float32 (NaN padded), ``n_cuts`` [F] int32: split
  candidates at the sample's quantiles j/256, j = 1..255.  Each candidate is
  the fp32 midpoint between the quantile value and the next distinct sample
  value above it (the gap below for the largest value); if the midpoint
  rounds down onto the lower value the upper value is used.  Candidates are
  de-duplicated, so a column has at most 255 distinct split values and none
  equals a sampled value unless two sampled values are adjacent floats.
* ``mean``, ``inv_std`` [F] float32: the sample's column mean and 1/std
  (population std; 1/std = 0 for a constant column) -- the standardisation
  statistics handed to the random MLP.

The random tree ensembles and MLPs of ``synth`` draw from these tables, so
their thresholds follow the feature distributions without the generator
computing any feature itself.

Run:  python tests/golden/make_forest_cuts.py
"""
from __future__ import annotations

import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

import oracle  # noqa: E402
import synth   # noqa: E402

N_SAMPLE = 65536
N_LEVELS = 255


def _split_between(a: np.float32, b: np.float32) -> np.float32:
    m = np.float32((np.float64(a) + np.float64(b)) / 2.0)
    return b if m <= a else m


def column_cuts(x: np.ndarray) -> np.ndarray:
    s = np.sort(x.astype(np.float32))
    u = np.unique(s)
    if len(u) < 2:
        return np.zeros(0, np.float32)
    n = len(s)
    out = []
    for j in range(1, N_LEVELS + 1):
        v = s[int(np.floor(j / (N_LEVELS + 1) * (n - 1)))]
        i = int(np.searchsorted(u, v))
        out.append(_split_between(u[i], u[i + 1]) if i + 1 < len(u) else _split_between(u[i - 1], u[i]))
    return np.unique(np.asarray(out, np.float32))


def make(name: str) -> str:
    cfg = synth.CONFIGS[name]
    probs = synth.problems(cfg)
    seg, cands = synth.candidates(cfg, probs)
    rows = synth.sample_rows(cfg, N_SAMPLE)
    X = oracle.features(synth.hardware(), probs, seg, cands, cfg.n_features, rows)
    F = cfg.n_features
    cuts = np.full((F, N_LEVELS), np.nan, np.float32)
    n_cuts = np.zeros(F, np.int32)
    for f in range(F):
        c = column_cuts(X[:, f])
        cuts[f, : len(c)] = c
        n_cuts[f] = len(c)
    X64 = X.astype(np.float64)
    mean = X64.mean(axis=0)
    std = X64.std(axis=0)
    inv_std = np.where(std > 0, 1.0 / np.where(std > 0, std, 1.0), 0.0)
    path = synth.cuts_path(name)
    np.savez_compressed(path, cuts=cuts, n_cuts=n_cuts, mean=mean.astype(np.float32),
                        inv_std=inv_std.astype(np.float32), rows=np.int64(len(rows)))
    return path


if __name__ == "__main__":
    for nm in (sys.argv[1:] or ["tiny", "medium", "full", "dataset"]):
        print(make(nm))
