"""Seeded synthetic workloads for batched (GEMM problem, candidate) scoring.

This module only *draws inputs*: GEMM problems, candidate configuration
records (struct-of-arrays), stand-in runtimes, and random model parameters
(a tree ensemble and an MLP).  It holds none of the scored path's arithmetic
-- no feature formula, no tree traversal, no MLP layer, no top-k, no regret.
Both the HIP library and the CPU oracle consume exactly the arrays returned
here, so a mistake in either of them cannot hide behind shared code.

Workload shapes follow the paper's description of its corpus: GEMM shapes
log-uniform over a [lo, hi]^3 box snapped to a lattice (Training the Selector,
"Shape Selection"), the searched CUTLASS knob grid (Table "Configuration knobs
exposed by the BF16 SM90 generator"), group-contiguous row order with one
segment per problem (Model A, group-id vector).  Runtimes are a stand-in for
measurements: a simple roofline time times lognormal noise; nothing in the
scored path depends on how they were made.

Every random draw comes from ``numpy.random.Generator(PCG64)`` streams spawned
from one ``SeedSequence`` per workload, so a workload is reproducible from its
name alone.
"""
from __future__ import annotations

import os
from dataclasses import dataclass, field

import numpy as np

# ----------------------------------------------------------------------------
# Integer codes shared by every consumer of a workload.
# ----------------------------------------------------------------------------
LAYOUT_TN, LAYOUT_TT, LAYOUT_NN, LAYOUT_NT = 0, 1, 2, 3
DTYPE_BF16, DTYPE_FP16, DTYPE_FP8 = 0, 1, 2
KS_WS, KS_PINGPONG, KS_COOP = 0, 1, 2
ES_NOSMEM, ES_TMA, ES_TMA_COOP = 0, 1, 2
TS_PERSISTENT, TS_STREAMK = 0, 1

#: Candidate struct-of-arrays fields, in the order of the C record of pointers.
CAND_FIELDS = (
    ("tile_m", np.uint16), ("tile_n", np.uint16), ("tile_k", np.uint16), ("inst_n", np.uint16),
    ("stages", np.uint8), ("cluster_m", np.uint8), ("cluster_n", np.uint8), ("swizzle", np.uint8),
    ("inst_m_div16", np.uint8), ("inst_k", np.uint8), ("kernel_sched", np.uint8),
    ("epi_sched", np.uint8), ("tile_sched", np.uint8),
)
PROBLEM_DTYPE = np.dtype([("M", "<i4"), ("N", "<i4"), ("K", "<i4"),
                          ("layout", "u1"), ("dtype", "u1"), ("pad", "u1", (2,))])


def hardware() -> dict:
    """Hardware descriptor of the *target* the ranked kernels run on.

    These are the GH200 figures the paper quotes (132 SMs, 228 KiB shared
    memory per SM, 227 KiB per block with a 2 KiB reserve, 50 MiB LLC,
    4 TB/s HBM, 989.5 TFLOP/s dense BF16), stored as exact integers in fixed
    units: bytes, GB/s (= bytes/ns), GFLOP/s (= flop/ns).  The FP8 peak is
    taken as twice BF16 (the paper gives BF16 only).
    """
    return dict(n_sm=132, smem_per_sm=233472, smem_per_block_max=232448, smem_reserved=2048,
                regs_per_sm=65536, max_regs_per_thread=255, max_blocks_per_sm=32,
                max_threads_per_sm=2048, arch_id=90, llc_bytes=52428800, hbm_bw_gbps=4000,
                peak_gflops=(989500, 989500, 1979000))


@dataclass(frozen=True)
class Config:
    name: str
    seed: int
    n_problems: int
    per_problem: int
    n_features: int
    trees: int
    depth: int
    k: int
    scorer: str = "forest"          # "forest" or "mlp"

    @property
    def rows(self) -> int:
        return self.n_problems * self.per_problem


CONFIGS = {
    "tiny": Config("tiny", 0, 16, 512, 64, 100, 6, 5),
    "medium": Config("medium", 1, 1024, 4096, 96, 500, 8, 10),
    "full": Config("full", 2, 256, 65536, 128, 1000, 8, 16),
    "dataset": Config("dataset", 3, 600, 8192, 128, 2000, 10, 10),
    # the neural ranker runs on the very rows of the dataset-scale workload
    "mlp": Config("mlp", 3, 600, 8192, 128, 0, 0, 10, scorer="mlp"),
}

MLP_WIDTHS = (128, 512, 512, 256, 1)

_STREAMS = ("problems", "candidates", "noise", "forest", "mlp", "sample", "linear")


def _streams(seed: int) -> dict:
    ss = np.random.SeedSequence(seed).spawn(len(_STREAMS))
    return {n: np.random.Generator(np.random.PCG64(s)) for n, s in zip(_STREAMS, ss)}


def _round8(x: np.ndarray, lo: int, hi: int) -> np.ndarray:
    return np.clip(8 * np.rint(x / 8.0), lo, hi).astype(np.int32)


def _loguniform(rng, lo, hi, n):
    return np.exp(rng.uniform(np.log(lo), np.log(hi), n))


# ----------------------------------------------------------------------------
# Problems
# ----------------------------------------------------------------------------
def problems(cfg: Config) -> np.ndarray:
    rng = _streams(cfg.seed)["problems"]
    P = cfg.n_problems
    out = np.zeros(P, PROBLEM_DTYPE)
    if cfg.name == "tiny":
        for f in ("M", "N", "K"):
            out[f] = _round8(_loguniform(rng, 64, 4096, P), 64, 4096)
        out["layout"] = LAYOUT_TN
        out["dtype"] = DTYPE_BF16
    elif cfg.name in ("medium", "full"):
        for f in ("M", "N", "K"):
            out[f] = _round8(_loguniform(rng, 64, 4096, P), 64, 4096)
        n_skinny = int(round(0.2 * P))
        skinny = rng.choice(P, n_skinny, replace=False)
        out["M"][skinny] = _round8(_loguniform(rng, 8, 64, n_skinny), 8, 64)
        out["layout"] = rng.integers(0, 4, P)
        out["dtype"] = rng.integers(0, 3, P)
    else:  # dataset / mlp
        for f in ("M", "N", "K"):
            out[f] = _round8(_loguniform(rng, 16, 16384, P), 16, 16384)
        n_deep = int(round(0.1 * P))
        deep = rng.choice(P, n_deep, replace=False)
        out["K"][deep] = _round8(_loguniform(rng, 32776, 131072, n_deep), 32776, 131072)
        out["layout"] = rng.integers(0, 4, P)
        out["dtype"] = DTYPE_BF16
    return out


# ----------------------------------------------------------------------------
# Candidate grids (each grid enumerated with its first field slowest)
# ----------------------------------------------------------------------------
def _product(**axes) -> dict:
    names = list(axes)
    vals = [np.asarray(axes[n]) for n in names]
    idx = np.indices([len(v) for v in vals]).reshape(len(vals), -1)
    return {n: v[i] for n, v, i in zip(names, vals, idx)}


def tiny_grid() -> dict:
    """864 points: T_M, T_N in {64,128,256}, T_K in {32,64}, stages 2-5,
    cluster (C_M, C_N) in {1,2}^2, swizzle in {1,2,4}."""
    return _product(tile_m=[64, 128, 256], tile_n=[64, 128, 256], tile_k=[32, 64],
                    stages=[2, 3, 4, 5], cluster_m=[1, 2], cluster_n=[1, 2], swizzle=[1, 2, 4])


CLUSTER_PAIRS = [(cm, cn) for cm in (1, 2, 4, 8, 16) for cn in (1, 2, 4, 8, 16) if cm * cn <= 16]


def paper_grid() -> dict:
    """The searched knob grid of the paper's BF16 generator: 4*9*5*11*15*3*3*2
    = 534,600 points per layout (Table "Configuration knobs")."""
    g = _product(tile_m=[64, 128, 192, 256], tile_n=[16, 32, 48, 64, 80, 96, 128, 192, 256],
                 tile_k=[32, 64, 128, 256, 512], stages=list(range(2, 13)),
                 cluster=list(range(len(CLUSTER_PAIRS))), kernel_sched=[0, 1, 2],
                 epi_sched=[0, 1, 2], tile_sched=[0, 1])
    cp = np.asarray(CLUSTER_PAIRS)
    g["cluster_m"] = cp[g["cluster"], 0]
    g["cluster_n"] = cp[g["cluster"], 1]
    del g["cluster"]
    return g


FULL_SCHED_PAIRS = [(KS_WS, ES_NOSMEM), (KS_WS, ES_TMA), (KS_PINGPONG, ES_TMA), (KS_COOP, ES_TMA_COOP)]


def full_grid() -> dict:
    """2^16-point cartesian grid: T_M(4) x T_N(8) x T_K(4) x I_N in {T_N, T_N/2}
    x stages 2-9 x (mainloop, epilogue) schedule pair(4) x cluster {1,2}^2
    x tile scheduler(2)."""
    g = _product(tile_m=[64, 128, 192, 256], tile_n=[16, 32, 48, 64, 96, 128, 192, 256],
                 tile_k=[32, 64, 128, 256], inst_half=[0, 1], stages=list(range(2, 10)),
                 sched=[0, 1, 2, 3], cluster_m=[1, 2], cluster_n=[1, 2], tile_sched=[0, 1])
    sp = np.asarray(FULL_SCHED_PAIRS)
    g["kernel_sched"] = sp[g["sched"], 0]
    g["epi_sched"] = sp[g["sched"], 1]
    g["inst_n"] = np.where(g["inst_half"] == 1, g["tile_n"] // 2, g["tile_n"])
    del g["sched"], g["inst_half"]
    return g


def catalogue_mask(g: dict, layout: int, dtype: int) -> np.ndarray:
    """Candidate-set construction: keep the grid points that pass the static
    legality rules of Table "Static validity constraints" (Stream-K needs the
    cooperative mainloop, cooperative needs T_M % 128 == 0, the K-box limits
    of transposed operands, and the per-block shared-memory capacity).

    This decides *which rows exist* in a workload; it is the catalogue the
    selector ranks, not part of the scored path.  The epilogue storage term is
    a plain size guess made here for filtering only.
    """
    b = 1 if dtype == DTYPE_FP8 else 2
    tm, tn, tk = (g[f].astype(np.int64) for f in ("tile_m", "tile_n", "tile_k"))
    st = g["stages"].astype(np.int64)
    ks, es, ts = g["kernel_sched"], g["epi_sched"], g["tile_sched"]
    cm, cn = g["cluster_m"].astype(np.int64), g["cluster_n"].astype(np.int64)
    epi = np.where(es == ES_NOSMEM, 0, np.where(es == ES_TMA, 2, 4)) * np.minimum(tm, 64) * np.minimum(tn, 32) * 2
    ok = (ts != TS_STREAMK) | (ks == KS_COOP)
    ok &= (ks != KS_COOP) | (tm % 128 == 0)
    ok &= st * (tm + tn) * tk * b + epi + 2048 <= 232448
    if layout in (LAYOUT_NN, LAYOUT_NT):      # A column-major
        ok &= tk <= 256 * cn
    if layout in (LAYOUT_TT, LAYOUT_NT):      # B row-major
        ok &= tk <= 256 * cm
    return ok


def _empty_cands(R: int) -> dict:
    return {f: np.zeros(R, dt) for f, dt in CAND_FIELDS}


def candidates(cfg: Config, probs: np.ndarray, with_ids: bool = False):
    """Return (seg_offsets int64 [P+1], candidate SoA dict of length R), and
    with ``with_ids`` also the grid index int32 [R] each row was drawn from
    (its configuration identity across problems)."""
    rng = _streams(cfg.seed)["candidates"]
    P, C = cfg.n_problems, cfg.per_problem
    R = P * C
    seg = np.arange(P + 1, dtype=np.int64) * C
    c = _empty_cands(R)
    in_bytes = np.where(probs["dtype"] == DTYPE_FP8, 1, 2)
    inst_k_row = np.repeat((32 // in_bytes).astype(np.uint8), C)
    if cfg.name == "tiny":
        g = tiny_grid()
        pick = np.concatenate([np.sort(rng.choice(len(g["tile_m"]), C, replace=False)) for _ in range(P)])
        for f in ("tile_m", "tile_n", "tile_k", "stages", "cluster_m", "cluster_n", "swizzle"):
            c[f][:] = g[f][pick]
        c["inst_n"][:] = c["tile_n"]
        c["kernel_sched"][:] = KS_WS
        c["epi_sched"][:] = ES_TMA
        c["tile_sched"][:] = TS_PERSISTENT
    elif cfg.name == "medium":
        g = paper_grid()
        masks = {}
        picks = []
        for p in range(P):
            key = (int(probs["layout"][p]), int(probs["dtype"][p]))
            if key not in masks:
                masks[key] = np.flatnonzero(catalogue_mask(g, *key))
            picks.append(np.sort(rng.choice(masks[key], C, replace=False)))
        pick = np.concatenate(picks)
        for f in ("tile_m", "tile_n", "tile_k", "stages", "cluster_m", "cluster_n",
                  "kernel_sched", "epi_sched", "tile_sched"):
            c[f][:] = g[f][pick]
        c["inst_n"][:] = c["tile_n"]
        c["swizzle"][:] = 1
    elif cfg.name == "full":
        g = full_grid()
        assert len(g["tile_m"]) == C
        for f in ("tile_m", "tile_n", "tile_k", "inst_n", "stages", "cluster_m", "cluster_n",
                  "kernel_sched", "epi_sched", "tile_sched"):
            c[f][:] = np.tile(g[f], P)
        c["swizzle"][:] = 1
    else:  # dataset / mlp: a draw from the legal part of the full grid
        g = full_grid()
        picks = []
        masks = {}
        for p in range(P):
            key = (int(probs["layout"][p]), int(probs["dtype"][p]))
            if key not in masks:
                masks[key] = np.flatnonzero(catalogue_mask(g, *key))
            picks.append(np.sort(rng.choice(masks[key], C, replace=False)))
        pick = np.concatenate(picks)
        for f in ("tile_m", "tile_n", "tile_k", "inst_n", "stages", "cluster_m", "cluster_n",
                  "kernel_sched", "epi_sched", "tile_sched"):
            c[f][:] = g[f][pick]
        c["swizzle"][:] = 1
    c["inst_m_div16"][:] = 4           # 64-row instruction tile
    c["inst_k"][:] = inst_k_row        # 32 bytes of K per instruction
    if with_ids:
        if cfg.name == "full":
            pick = np.tile(np.arange(C), P)
        return seg, c, pick.astype(np.int32)
    return seg, c


# ----------------------------------------------------------------------------
# Stand-in runtimes
# ----------------------------------------------------------------------------
def runtimes(cfg: Config, probs: np.ndarray, seg: np.ndarray, c: dict) -> np.ndarray:
    """Seconds, fp32.  A deliberately plain roofline stand-in for measured
    runtimes: waves-of-tiles compute time vs. re-streamed operand traffic, a
    mild stage-count efficiency, 2 us launch overhead, times exp(0.1 z),
    z ~ N(0, 1) per row.  Candidates whose pipeline buffers overflow the
    227 KiB per-block limit never run: +inf."""
    rng = _streams(cfg.seed)["noise"]
    hw = hardware()
    R = int(seg[-1])
    z = rng.standard_normal(R)
    out = np.empty(R, np.float32)
    pid = np.repeat(np.arange(len(probs)), np.diff(seg))
    peak_tab = np.asarray(hw["peak_gflops"], np.float64) * 1e9
    bw = hw["hbm_bw_gbps"] * 1e9
    sm = float(hw["n_sm"])
    step = 1 << 20
    for lo in range(0, R, step):
        hi = min(R, lo + step)
        pp = probs[pid[lo:hi]]
        M, N, K = (pp[f].astype(np.float64) for f in ("M", "N", "K"))
        b = np.where(pp["dtype"] == DTYPE_FP8, 1.0, 2.0)
        peak = peak_tab[pp["dtype"]]
        tm, tn, tk = (c[f][lo:hi].astype(np.float64) for f in ("tile_m", "tile_n", "tile_k"))
        st = c["stages"][lo:hi].astype(np.float64)
        gm, gn, gk = np.ceil(M / tm), np.ceil(N / tn), np.ceil(K / tk)
        t_comp = np.ceil(gm * gn / sm) * (2.0 * tm * tn * gk * tk) / (peak / sm)
        t_mem = (b * M * K * gn + b * K * N * gm + 4.0 * M * N) / bw
        eff = np.minimum(1.0, 0.55 + 0.1 * st)
        t = (np.maximum(t_comp, t_mem) / eff + 2e-6) * np.exp(0.1 * z[lo:hi])
        t[st * (tm + tn) * tk * b + 2048 > 232448] = np.inf
        out[lo:hi] = t
    return out


# ----------------------------------------------------------------------------
# Model parameters
# ----------------------------------------------------------------------------
GOLDEN = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "tests", "golden")


def cuts_path(name: str) -> str:
    base = "dataset" if name == "mlp" else name
    return os.path.join(GOLDEN, f"forest_cuts_{base}.npz")


def load_cuts(name: str) -> dict:
    """Per-column split candidates and column statistics of the workload's
    feature matrix, stored by ``tests/golden/make_forest_cuts.py``."""
    with np.load(cuts_path(name), allow_pickle=False) as z:
        return {k: z[k] for k in z.files}


def forest(cfg: Config, cuts: dict | None = None) -> dict:
    """Random GBDT-shaped ensemble: ``trees`` perfect trees of ``depth``.

    Node features are uniform over the non-constant columns; a node's threshold
    is uniform over that column's stored split candidates (quantile-placed
    midpoints between distinct values); leaves are fp32(N(0, 0.1^2)).  Nodes
    are stored breadth-first per tree (children of node i at 2i+1 / 2i+2).
    """
    if cuts is None:
        cuts = load_cuts(cfg.name)
    rng = _streams(cfg.seed)["forest"]
    T, d = cfg.trees, cfg.depth
    n_cut = cuts["n_cuts"][: cfg.n_features]
    cols = np.flatnonzero(n_cut > 0)
    n_int = (1 << d) - 1
    feat = rng.choice(cols, size=(T, n_int))
    j = np.floor(rng.random((T, n_int)) * n_cut[feat]).astype(np.int64)
    thr = cuts["cuts"][feat, j].astype(np.float32)
    leaves = rng.normal(0.0, 0.1, (T, 1 << d)).astype(np.float32)
    return dict(n_trees=T, depth=d, n_features=cfg.n_features, flags=1, base_score=0.0,
                node_feature=feat.astype(np.uint8), node_threshold=thr, leaf_value=leaves)


def _bf16_bits_rounded(w: np.ndarray) -> np.ndarray:
    """bf16 bit patterns of finite fp32 draws, rounded to nearest (ties to
    even); a plain encoding of the generator's parameters."""
    u = np.ascontiguousarray(w, np.float32).view(np.uint32).astype(np.uint64)
    return ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)


def mlp(cfg: Config, cuts: dict | None = None) -> dict:
    """Random MLP 128->512->512->256->1: Kaiming-normal weights (std
    sqrt(2/fan_in)) rounded to bf16, stored [out][in]; fp32 biases U(+-1/sqrt(fan_in));
    standardisation mean / 1/std taken from the stored column statistics
    (a column with zero spread gets 1/std = 0)."""
    if cuts is None:
        cuts = load_cuts(cfg.name)
    rng = _streams(cfg.seed)["mlp"]
    out = {}
    for l in range(4):
        fi, fo = MLP_WIDTHS[l], MLP_WIDTHS[l + 1]
        w = rng.normal(0.0, np.sqrt(2.0 / fi), (fo, fi)).astype(np.float32)
        out[f"W{l + 1}"] = _bf16_bits_rounded(w)
        out[f"b{l + 1}"] = rng.uniform(-1.0 / np.sqrt(fi), 1.0 / np.sqrt(fi), fo).astype(np.float32)
    out["mean"] = cuts["mean"][:128].astype(np.float32)
    out["inv_std"] = cuts["inv_std"][:128].astype(np.float32)
    return out


def linear(cfg: Config, cuts: dict | None = None) -> dict:
    """Random ridge-style linear scorer over cfg.n_features columns: weights
    N(0, 1/F), one-hot weights N(0, 0.1^2), bias U(-1, 1); standardisation
    from the stored column statistics (as for the MLP)."""
    if cuts is None:
        cuts = load_cuts(cfg.name)
    rng = _streams(cfg.seed)["linear"]
    F = cfg.n_features
    return {"n_features": F,
            "bias": float(np.float32(rng.uniform(-1.0, 1.0))),
            "mean": cuts["mean"][:F].astype(np.float32),
            "inv_std": cuts["inv_std"][:F].astype(np.float32),
            "w": rng.normal(0.0, 1.0 / np.sqrt(F), F).astype(np.float32),
            "w_onehot": rng.normal(0.0, 0.1, 12).astype(np.float32)}


def sample_rows(cfg: Config, n: int) -> np.ndarray:
    """Sorted distinct row indices, a seeded uniform sample (all rows if n >= R)."""
    R = cfg.rows
    if n >= R:
        return np.arange(R, dtype=np.int64)
    rng = _streams(cfg.seed)["sample"]
    return np.sort(rng.choice(R, n, replace=False)).astype(np.int64)


@dataclass
class Workload:
    cfg: Config
    hw: dict
    problems: np.ndarray
    seg: np.ndarray
    cands: dict
    runtimes: np.ndarray | None = None
    forest: dict | None = None
    mlp: dict | None = None
    extra: dict = field(default_factory=dict)


def workload(name: str, with_runtimes: bool = True, with_model: bool = True) -> Workload:
    cfg = CONFIGS[name]
    probs = problems(cfg)
    seg, cands, ids = candidates(cfg, probs, with_ids=True)
    w = Workload(cfg, hardware(), probs, seg, cands)
    w.extra["config_id"] = ids
    if with_runtimes:
        w.runtimes = runtimes(cfg, probs, seg, cands)
    if with_model:
        if cfg.scorer == "forest":
            w.forest = forest(cfg)
        else:
            w.mlp = mlp(cfg)
    return w


# ----------------------------------------------------------------------------
# Small generators for edge-case tests
# ----------------------------------------------------------------------------
def random_scores(rng, n: int, tie_frac: float = 0.0, n_levels: int = 4) -> np.ndarray:
    """fp32 scores; a fraction are drawn from a few repeated values (ties)."""
    s = rng.standard_normal(n).astype(np.float32)
    if tie_frac > 0:
        m = rng.random(n) < tie_frac
        s[m] = rng.integers(0, n_levels, int(m.sum())).astype(np.float32)
    return s


def ragged_segments(rng, P: int, max_len: int, empty_frac: float = 0.1) -> np.ndarray:
    lens = rng.integers(1, max_len + 1, P)
    lens[rng.random(P) < empty_frac] = 0
    return np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
