"""Stored oracle selections for the full-size parity tests.

For every problem of a workload, the CPU oracle's whole scored path --
features phi(p, c, h), then the forest (Model A) or the MLP (Model B), then
the per-problem top-k of eq. (selection) generalised to the k best -- over
every row, stored per problem:

  idx       int32   [P][k]  local indices of the k best rows
  vals      float32 [P][k]  their scores
  next_val  float32 [P]     the (k+1)-th score (-inf if the segment has <= k
                            rows): the margin a pick can lose before a
                            different pick would be right
  leaf_hash uint64  [P]     forest workloads: wrapping sum over the segment's
                            rows of each row's leaf-path fingerprint
  rms       float64 [P]     MLP workload: RMS of the problem's oracle scores
                            (the scale of the MLP acceptance band)
  fingerprint               SHA-256 of the workload's inputs, so a test can
                            tell a stale file from a real mismatch

The inputs come from the seeded generators in synth/, every value from
oracle/ alone.  Run from the repository root (about 15 minutes on 8 cores):
    python tests/golden/make_selections.py [tiny medium full dataset mlp]
"""
from __future__ import annotations

import hashlib
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import oracle  # noqa: E402
import synth  # noqa: E402

NAMES = ("tiny", "medium", "full", "dataset", "mlp")
BLOCK_ROWS = 1 << 21          # rows per oracle pass (bounds host memory)


def path(name: str) -> str:
    return os.path.join(HERE, f"selections_{name}.npz")


def fingerprint(w) -> str:
    """SHA-256 over every input array of the workload that the scored path
    reads: problems, offsets, candidate fields, model parameters."""
    h = hashlib.sha256()
    arrays = [w.problems, w.seg] + [w.cands[n] for n in sorted(w.cands)]
    model = w.forest if w.forest is not None else w.mlp
    for n in sorted(model):
        v = model[n]
        arrays.append(v if isinstance(v, np.ndarray) else np.asarray(v))
    for a in arrays:
        a = np.ascontiguousarray(a)
        h.update(str(a.dtype).encode() + str(a.shape).encode())
        h.update(a.view(np.uint8).tobytes())
    return h.hexdigest()


def blocks(seg: np.ndarray):
    """Consecutive problem ranges [p0, p1) of about BLOCK_ROWS rows each."""
    P = len(seg) - 1
    p0 = 0
    while p0 < P:
        p1 = p0 + 1
        while p1 < P and seg[p1 + 1] - seg[p0] <= BLOCK_ROWS:
            p1 += 1
        yield p0, p1
        p0 = p1


def make(name: str) -> dict:
    w = synth.workload(name)
    cfg = w.cfg
    P, k, F = cfg.n_problems, cfg.k, cfg.n_features
    idx = np.empty((P, k), np.int32)
    vals = np.empty((P, k), np.float32)
    next_val = np.empty(P, np.float32)
    leaf_hash = np.zeros(P, np.uint64)
    rms = np.zeros(P, np.float64)
    for p0, p1 in blocks(w.seg):
        r0, r1 = int(w.seg[p0]), int(w.seg[p1])
        seg = w.seg[p0:p1 + 1] - r0
        cands = {n: v[r0:r1] for n, v in w.cands.items()}
        X = oracle.features(w.hw, w.problems[p0:p1], seg, cands, F)
        if w.forest is not None:
            s, h = oracle.forest(w.forest, X, leaf_hash=True)
            for p in range(p1 - p0):
                leaf_hash[p0 + p] = np.sum(h[seg[p]:seg[p + 1]], dtype=np.uint64)
        else:
            s = oracle.mlp(w.mlp, X)
            for p in range(p1 - p0):
                v = s[seg[p]:seg[p + 1]].astype(np.float64)
                rms[p0 + p] = np.sqrt(np.mean(v * v)) if len(v) else 0.0
        i, v = oracle.topk(s, seg, k + 1)
        idx[p0:p1], vals[p0:p1], next_val[p0:p1] = i[:, :k], v[:, :k], v[:, k]
        print(f"  {name}: problems {p0}..{p1 - 1} done", flush=True)
    out = dict(idx=idx, vals=vals, next_val=next_val, fingerprint=np.array(fingerprint(w)))
    if w.forest is not None:
        out["leaf_hash"] = leaf_hash
    else:
        out["rms"] = rms
    return out


def load(name: str) -> dict:
    with np.load(path(name), allow_pickle=False) as z:
        return {k: z[k] for k in z.files}


if __name__ == "__main__":
    for name in sys.argv[1:] or NAMES:
        t0 = time.time()
        np.savez_compressed(path(name), **make(name))
        print(f"{name}: wrote {path(name)} in {time.time() - t0:.0f} s", flush=True)
