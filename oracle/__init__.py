"""CPU oracle for batched candidate scoring -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The HIP library never depends on it.

The arithmetic lives in ``hwsel_oracle.c`` (plain C, binary64, OpenMP over
rows / problems); this module builds it with gcc and marshals numpy arrays.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "hwsel_oracle.c")
LIB = os.path.join(HERE, "_build", "liboracle.so")
CFLAGS = ["-O2", "-std=c11", "-fno-fast-math", "-ffp-contract=off", "-fopenmp", "-fPIC", "-shared"]


def build(force: bool = True) -> str:
    os.makedirs(os.path.dirname(LIB), exist_ok=True)
    if force or not os.path.exists(LIB) or os.path.getmtime(LIB) < os.path.getmtime(SRC):
        tmp = LIB + f".tmp{os.getpid()}"
        subprocess.run(["gcc", *CFLAGS, SRC, "-o", tmp, "-lm"], check=True)
        os.replace(tmp, LIB)
    return LIB


class _HW(C.Structure):
    _fields_ = [(n, C.c_int64) for n in (
        "n_sm", "smem_per_sm", "smem_per_block_max", "smem_reserved", "regs_per_sm",
        "max_regs_per_thread", "max_blocks_per_sm", "max_threads_per_sm", "arch_id",
        "llc_bytes", "hbm_bw_gbps")] + [("peak_gflops", C.c_int64 * 3)]


class _Problems(C.Structure):
    _fields_ = [("M", C.c_void_p), ("N", C.c_void_p), ("K", C.c_void_p),
                ("layout", C.c_void_p), ("dtype", C.c_void_p)]


_CAND = ("tile_m", "tile_n", "tile_k", "inst_n", "stages", "cluster_m", "cluster_n", "swizzle",
         "inst_m_div16", "inst_k", "kernel_sched", "epi_sched", "tile_sched")


class _Cands(C.Structure):
    _fields_ = [(n, C.c_void_p) for n in _CAND]


class _Forest(C.Structure):
    _fields_ = [("n_trees", C.c_int32), ("depth", C.c_int32), ("n_features", C.c_int32),
                ("flags", C.c_uint32), ("base_score", C.c_float), ("node_feature", C.c_void_p),
                ("node_threshold", C.c_void_p), ("leaf_value", C.c_void_p)]


class _MLP(C.Structure):
    _fields_ = [("n_in", C.c_int32), ("h1", C.c_int32), ("h2", C.c_int32), ("h3", C.c_int32),
                ("mean", C.c_void_p), ("inv_std", C.c_void_p), ("W1", C.c_void_p),
                ("W2", C.c_void_p), ("W3", C.c_void_p), ("W4", C.c_void_p), ("b1", C.c_void_p),
                ("b2", C.c_void_p), ("b3", C.c_void_p), ("b4", C.c_void_p)]


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB) or os.path.getmtime(LIB) < os.path.getmtime(SRC):
            build(force=True)
        _lib = C.CDLL(LIB)
        _lib.oracle_bf16_round.restype = C.c_float
        _lib.oracle_bf16_round.argtypes = [C.c_float]
    return _lib


def _p(a: np.ndarray | None):
    return None if a is None else C.c_void_p(a.ctypes.data)


def _c(a, dt):
    return np.ascontiguousarray(a, dtype=dt)


def hw_struct(hw: dict) -> _HW:
    s = _HW()
    for n, _ in _HW._fields_[:-1]:
        setattr(s, n, int(hw[n]))
    for i, v in enumerate(hw["peak_gflops"]):
        s.peak_gflops[i] = int(v)
    return s


def features(hw: dict, problems: np.ndarray, seg: np.ndarray, cands: dict, n_features: int,
             rows: np.ndarray | None = None) -> np.ndarray:
    """X[i] = phi(problem of row i, candidate row i, hw) for all rows, or for
    the listed ``rows`` (output row i is rows[i])."""
    keep = []
    pr = _Problems()
    for n, dt in (("M", np.int32), ("N", np.int32), ("K", np.int32), ("layout", np.uint8), ("dtype", np.uint8)):
        a = _c(problems[n], dt)
        keep.append(a)
        setattr(pr, n, a.ctypes.data)
    cs = _Cands()
    for n in _CAND:
        a = np.ascontiguousarray(cands[n])
        keep.append(a)
        setattr(cs, n, a.ctypes.data)
    seg = _c(seg, np.int64)
    P = len(seg) - 1
    if rows is None:
        n_out, rp = int(seg[-1]), None
    else:
        rows = _c(rows, np.int64)
        n_out, rp = len(rows), rows
    X = np.empty((n_out, n_features), np.float32)
    h = hw_struct(hw)
    rc = lib().oracle_features(C.byref(h), C.byref(pr), C.c_int64(P), _p(seg), C.byref(cs), _p(rp),
                               C.c_int64(n_out), C.c_int(n_features), _p(X), C.c_int64(n_features))
    if rc:
        raise ValueError(f"oracle_features: status {rc}")
    return X


def _forest_struct(f: dict, keep: list) -> _Forest:
    s = _Forest()
    s.n_trees, s.depth, s.n_features = int(f["n_trees"]), int(f["depth"]), int(f["n_features"])
    s.flags, s.base_score = int(f["flags"]), float(f["base_score"])
    for n, dt in (("node_feature", np.uint8), ("node_threshold", np.float32), ("leaf_value", np.float32)):
        a = _c(f[n], dt)
        keep.append(a)
        setattr(s, n, a.ctypes.data)
    return s


def forest(f: dict, X: np.ndarray, rows: np.ndarray | None = None, leaves: bool = False,
           leaf_hash: bool = False):
    """Scores of rows of X; with ``leaves`` also the leaf indices [n][T], with
    ``leaf_hash`` also each row's leaf-path fingerprint (uint64 [n]).  Returns
    the scores alone, or a tuple (scores, leaves?, hashes?) of what was asked."""
    X = _c(X, np.float32)
    keep = []
    s = _forest_struct(f, keep)
    if rows is not None:
        rows = _c(rows, np.int64)
    n = X.shape[0] if rows is None else len(rows)
    out = np.empty(n, np.float32)
    li = np.empty((n, s.n_trees), np.uint16) if leaves else None
    lh = np.empty(n, np.uint64) if leaf_hash else None
    lib().oracle_forest(C.byref(s), _p(X), C.c_int64(X.shape[1]), _p(rows), C.c_int64(n), _p(out), _p(li),
                        _p(lh))
    extra = tuple(a for a in (li, lh) if a is not None)
    return (out, *extra) if extra else out


def leaf_mix(z: int) -> int:
    """The 64-bit mixer of the leaf-path fingerprint."""
    lib().oracle_leaf_mix.restype = C.c_uint64
    lib().oracle_leaf_mix.argtypes = [C.c_uint64]
    return int(lib().oracle_leaf_mix(z))


def forest_linked(f: dict, X: np.ndarray) -> np.ndarray:
    X = _c(X, np.float32)
    keep = []
    s = _forest_struct(f, keep)
    out = np.empty(X.shape[0], np.float32)
    rc = lib().oracle_forest_linked(C.byref(s), _p(X), C.c_int64(X.shape[1]), C.c_int64(X.shape[0]), _p(out))
    if rc:
        raise MemoryError("oracle_forest_linked")
    return out


def mlp(m: dict, X: np.ndarray, rows: np.ndarray | None = None, exact: bool = False) -> np.ndarray:
    X = _c(X, np.float32)
    keep = []
    s = _MLP()
    s.n_in, s.h1, s.h2, s.h3 = 128, 512, 512, 256
    for n, dt in (("mean", np.float32), ("inv_std", np.float32), ("W1", np.uint16), ("W2", np.uint16),
                  ("W3", np.uint16), ("W4", np.uint16), ("b1", np.float32), ("b2", np.float32),
                  ("b3", np.float32), ("b4", np.float32)):
        a = _c(m[n], dt)
        keep.append(a)
        setattr(s, n, a.ctypes.data)
    if rows is not None:
        rows = _c(rows, np.int64)
    n = X.shape[0] if rows is None else len(rows)
    out = np.empty(n, np.float32)
    rc = lib().oracle_mlp(C.byref(s), _p(X), C.c_int64(X.shape[1]), _p(rows), C.c_int64(n), _p(out),
                          C.c_int(1 if exact else 0))
    if rc:
        raise ValueError(f"oracle_mlp: status {rc}")
    return out


def topk(scores: np.ndarray, seg: np.ndarray, k: int):
    scores = _c(scores, np.float32)
    seg = _c(seg, np.int64)
    P = len(seg) - 1
    idx = np.empty((P, k), np.int32)
    vals = np.empty((P, k), np.float32)
    lib().oracle_topk(_p(scores), _p(seg), C.c_int64(P), C.c_int32(k), _p(idx), _p(vals))
    return idx, vals


def regret(runtimes: np.ndarray, seg: np.ndarray, idx: np.ndarray):
    rt = _c(runtimes, np.float32)
    seg = _c(seg, np.int64)
    idx = _c(idx, np.int32)
    P, k = idx.shape
    r1 = np.empty(P, np.float32)
    rk = np.empty(P, np.float32)
    best = np.empty(P, np.int32)
    lib().oracle_regret(_p(rt), _p(seg), C.c_int64(P), _p(idx), C.c_int32(k), _p(r1), _p(rk), _p(best))
    return r1, rk, best


def bf16_round(x: float) -> float:
    return lib().oracle_bf16_round(float(x))


def num_threads() -> int:
    return int(lib().oracle_num_threads())


class _Linear(C.Structure):
    _fields_ = [("n_features", C.c_int32), ("bias", C.c_float), ("mean", C.c_void_p), ("inv_std", C.c_void_p),
                ("w", C.c_void_p), ("w_onehot", C.c_void_p)]


def linear(m: dict, X: np.ndarray):
    """Ridge scorer: (fp32 scores, binary64 sum of term magnitudes) per row."""
    X = _c(X, np.float32)
    keep = [_c(m[n], np.float32) for n in ("mean", "inv_std", "w", "w_onehot")]
    s = _Linear(int(m["n_features"]), float(m["bias"]), *[a.ctypes.data for a in keep])
    n = X.shape[0]
    out = np.empty(n, np.float32)
    mag = np.empty(n, np.float64)
    rc = lib().oracle_linear(C.byref(s), _p(X), C.c_int64(X.shape[1]), C.c_int64(n), _p(out), _p(mag))
    if rc:
        raise ValueError(f"oracle_linear: status {rc}")
    return out, mag


EVAL_FIELDS = ("mean_regret", "median_regret", "p95_regret", "max_regret", "top1", "top5", "within5",
               "random_regret", "n_groups")


def evaluate(runtimes: np.ndarray, seg: np.ndarray, idx: np.ndarray):
    """Aggregate selection metrics; returns (dict of EVAL_FIELDS, per-group
    regret float64, rank int32, ybar float64)."""
    rt = _c(runtimes, np.float32)
    seg = _c(seg, np.int64)
    idx = _c(idx, np.int32)
    P, k = idx.shape
    out = np.empty(9, np.float64)
    reg = np.empty(P, np.float64)
    rank = np.empty(P, np.int32)
    ybar = np.empty(P, np.float64)
    rc = lib().oracle_evaluate(_p(rt), _p(seg), C.c_int64(P), _p(idx), C.c_int32(k), _p(out), _p(reg), _p(rank),
                               _p(ybar))
    if rc:
        raise MemoryError("oracle_evaluate")
    return dict(zip(EVAL_FIELDS, out.tolist())), reg, rank, ybar


def static_config(runtimes: np.ndarray, seg: np.ndarray, config_id: np.ndarray, n_configs: int):
    """(best id or -1, its group count, its mean y)."""
    rt = _c(runtimes, np.float32)
    seg = _c(seg, np.int64)
    cfg = _c(config_id, np.int32)
    best, cnt, my = C.c_int32(0), C.c_int32(0), C.c_double(0.0)
    rc = lib().oracle_static_config(_p(rt), _p(seg), C.c_int64(len(seg) - 1), _p(cfg), C.c_int32(n_configs),
                                    C.byref(best), C.byref(cnt), C.byref(my))
    if rc:
        raise MemoryError("oracle_static_config")
    return int(best.value), int(cnt.value), float(my.value)


def catalogue_size() -> int:
    lib().oracle_catalogue_size.restype = C.c_int64
    return int(lib().oracle_catalogue_size())


def catalogue_decode(indices, dtype: int) -> dict:
    """Knob fields of catalogue points (candidate SoA with the library's
    field widths)."""
    indices = np.asarray(indices, np.int64)
    f = np.empty(13, np.int32)
    rows = np.empty((len(indices), 13), np.int32)
    for i, v in enumerate(indices):
        lib().oracle_catalogue_decode(C.c_int64(int(v)), C.c_int(int(dtype)), _p(f))
        rows[i] = f
    out = {}
    for j, n in enumerate(_CAND):
        out[n] = rows[:, j].astype(np.uint16 if n in ("tile_m", "tile_n", "tile_k", "inst_n") else np.uint8)
    return out


def catalogue_mask(hw: dict, problems: np.ndarray, flags: int = 0):
    """(mask uint8 [P][catalogue size], valid count int64 [P])."""
    keep = []
    pr = _Problems()
    for n, dt in (("M", np.int32), ("N", np.int32), ("K", np.int32), ("layout", np.uint8), ("dtype", np.uint8)):
        a = _c(problems[n], dt)
        keep.append(a)
        setattr(pr, n, a.ctypes.data)
    P = len(problems)
    n = catalogue_size()
    mask = np.empty((P, n), np.uint8)
    cnt = np.empty(P, np.int64)
    h = hw_struct(hw)
    lib().oracle_catalogue_mask(C.byref(h), C.byref(pr), C.c_int64(P), C.c_int(flags), _p(mask), _p(cnt))
    return mask, cnt


def catalogue_compact(mask: np.ndarray):
    """Group-contiguous list of valid points: (seg_offsets int64 [P+1],
    catalogue index int32 [total]) in problem order, ascending index."""
    seg = np.zeros(mask.shape[0] + 1, np.int64)
    parts = []
    for p in range(mask.shape[0]):
        nz = np.nonzero(mask[p])[0]
        parts.append(nz.astype(np.int32))
        seg[p + 1] = seg[p] + len(nz)
    return seg, (np.concatenate(parts) if parts else np.zeros(0, np.int32))
