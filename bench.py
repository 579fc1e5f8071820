"""Benchmark of the batched candidate-scoring path on one MI355X.

Workload: the dataset-scale configuration -- 600 GEMM problems x 8,192
candidate configurations = 4,915,200 rows, 128 features, a random GBDT of
2,000 depth-10 trees and a random MLP 128->512->512->256->1 -- all synthetic
and seeded (see synth/).  One step is one pass of the whole path over that
batch, inputs already resident in HBM:

    features -> forest score -> top-10 per problem -> regret
             -> MLP score    -> top-10 per problem -> regret

Prints ONE JSON line (rank 0).  `value` = rows per second through the whole
step.  Per-stage times come from HIP events recorded on the launch stream
inside the timed region.  `roofline` is for the dominant kernel (forest
scoring); `cpu_baseline` times the CPU oracle on a bounded sample of the same
workload on the host cores.  `extras` times, each on its own after the timed
step, the entries around the path on the same workload: the fused
features -> forest -> top-k selection, the linear and sampling-score scorers,
the selection metrics and static-configuration baseline, and the
configuration catalogue (mask, compaction, candidate rows) for the same 600
problems.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "candidate rows scored/sec (features+forest+top-k) at 4.9M rows; % HBM roofline"
HBM_PEAK_GBS = 8000.0
BF16_PEAK_TFLOPS = 2500.0
# VALU issue: 256 CUs x 4 SIMDs x 16 lanes x 2.4 GHz
LANE_OPS_PER_S = 256 * 64 * 2.4e9
# the traversal's walk issues 5 VALU instructions per node visit (compare with
# borrow, child-code select, child index with carry, bin address, pair
# address: counted in its ISA) and 1.8 LDS gathers (bin, and the sibling pair
# on 7 of 10 levels); LDS serves 32 lanes per clock per CU
VALU_OPS_PER_VISIT = 5
LDS_LANES_PER_S = 256 * 32 * 2.4e9
LDS_OPS_PER_VISIT = 1.8


def forest_traffic_bytes():
    """HBM bytes per hwsel_forest_score call on this workload, from the two
    committed counter passes (FETCH_SIZE, WRITE_SIZE, scaled by the plain-copy
    calibration) -- or None once the forest kernels have changed since."""
    import hashlib
    path = os.path.join(ROOT, "profiles", "forest_score_dataset_traffic.json")
    try:
        rec = json.load(open(path))
        src = open(os.path.join(ROOT, rec["source"]), "rb").read()
    except (OSError, ValueError, KeyError):
        return None
    if hashlib.sha256(src).hexdigest() != rec["source_sha256"]:
        return None
    return 1024.0 * (rec["fetch_kib"] * rec["fetch_scale"] + rec["write_kib"] * rec["write_scale"])


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def ceilings(torch) -> dict:
    """Measured ceilings (libhwsel_ceilings.so): the traversal's own walk with
    every operand in LDS, back-to-back bf16 matrix-core products, a streaming
    copy and a streaming fill (the faster of a fill kernel and the runtime's
    own), each the best of 5 timings with HIP events on the current stream."""
    import ctypes as C
    path = os.path.join(ROOT, "paper_2609_35587_amd", "libhwsel_ceilings.so")
    L = C.CDLL(path)
    L.hwsel_ceiling_visits_per_launch.restype = C.c_int64
    L.hwsel_ceiling_mfma_flops_per_launch.restype = C.c_double
    L.hwsel_ceiling_visits.argtypes = [C.c_int, C.c_void_p, C.c_void_p]
    L.hwsel_ceiling_mfma.argtypes = [C.c_int, C.c_void_p, C.c_void_p]
    L.hwsel_ceiling_copy.argtypes = [C.c_void_p, C.c_void_p, C.c_int64, C.c_void_p]
    L.hwsel_ceiling_fill.argtypes = [C.c_void_p, C.c_int64, C.c_int, C.c_void_p]
    stream = torch.cuda.current_stream()
    sink = torch.zeros(16, dtype=torch.float32, device="cuda")
    h = stream.cuda_stream

    def best(fn, reps=5):
        fn()
        out = []
        for _ in range(reps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            fn()
            e1.record(stream)
            torch.cuda.synchronize()
            out.append(e0.elapsed_time(e1) / 1e3)
        return min(out)

    it_v, it_m = 2000, 20000
    t_v = best(lambda: L.hwsel_ceiling_visits(it_v, sink.data_ptr(), h))
    t_m = best(lambda: L.hwsel_ceiling_mfma(it_m, sink.data_ptr(), h))
    n16 = (1 << 30) // 16
    src = torch.ones(n16 * 4, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    t_c = best(lambda: L.hwsel_ceiling_copy(src.data_ptr(), dst.data_ptr(), n16, h))
    t_f = min(best(lambda: L.hwsel_ceiling_fill(dst.data_ptr(), n16, 0, h)),
              best(lambda: L.hwsel_ceiling_fill(dst.data_ptr(), n16, 1, h)))
    del src, dst
    return {"visits_per_s": L.hwsel_ceiling_visits_per_launch(it_v) / t_v,
            "bf16_flops_per_s": L.hwsel_ceiling_mfma_flops_per_launch(it_m) / t_m,
            "copy_GBps": 2 * (1 << 30) / t_c / 1e9, "fill_GBps": (1 << 30) / t_f / 1e9}


def per_config(hwsel, torch, dev, name: str) -> dict:
    """The scored path (features, packed forest, top-k, regret) on one of the
    other workloads, each stage timed on its own (median of 3)."""
    import synth
    w = synth.workload(name)
    cfg = w.cfg
    R, P, F, k = cfg.rows, cfg.n_problems, cfg.n_features, cfg.k
    probs, seg = hwsel.to_device(w.problems, dev), hwsel.to_device(w.seg, dev)
    cands = {n: hwsel.to_device(v, dev) for n, v in w.cands.items()}
    rt = hwsel.to_device(w.runtimes, dev)
    forest = dict(w.forest)
    for n in ("node_feature", "node_threshold", "leaf_value"):
        forest[n] = hwsel.to_device(w.forest[n], dev)
    packed = hwsel.hwsel_forest_pack(forest)
    ws = torch.empty(hwsel.hwsel_forest_workspace_bytes(forest, R), dtype=torch.uint8, device=dev)
    X = torch.empty((R, F), dtype=torch.float32, device=dev)
    s = torch.empty(R, dtype=torch.float32, device=dev)
    idx = torch.empty((P, k), dtype=torch.int32, device=dev)
    out = {"rows": R, "problems": P, "features": F, "trees": cfg.trees, "depth": cfg.depth, "k": k}
    out["features_ms"] = timed(torch, lambda: hwsel.hwsel_features(w.hw, probs, seg, cands, F, X=X))
    out["forest_ms"] = timed(torch, lambda: hwsel.hwsel_forest_score(forest, X, scores=s, packed=packed, workspace=ws))
    out["topk_ms"] = timed(torch, lambda: hwsel.hwsel_topk_per_problem(s, seg, k, idx=idx, with_vals=False))
    out["regret_ms"] = timed(torch, lambda: hwsel.hwsel_regret(rt, seg, idx))
    path_ms = out["features_ms"] + out["forest_ms"] + out["topk_ms"]
    out["rows_per_s"] = R / (path_ms / 1e3)
    out["visits_per_s"] = R * cfg.trees * cfg.depth / (out["forest_ms"] / 1e3)
    out["features_hbm_frac"] = R * (17 + 4 * F) / (out["features_ms"] / 1e3) / 1e9 / HBM_PEAK_GBS
    return out


def cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(w, n_problems: int, gpu_idx_forest: np.ndarray, gpu_idx_mlp: np.ndarray) -> tuple[dict, dict]:
    """Times the oracle on the first n_problems problems of the workload and
    compares its picks there with the library's from the timed step (problems
    whose forest top-k, MLP top-1 and MLP top-k equal the oracle's).  Returns
    the baseline record and the comparison."""
    import oracle
    cfg = w.cfg
    seg = w.seg[: n_problems + 1]
    R = int(seg[-1])
    probs = w.problems[:n_problems]
    cands = {k: v[:R] for k, v in w.cands.items()}
    import synth
    m = synth.mlp(synth.CONFIGS["mlp"])
    t0 = time.perf_counter()
    X = oracle.features(w.hw, probs, seg, cands, cfg.n_features)
    s = oracle.forest(w.forest, X)
    idx, _ = oracle.topk(s, seg, cfg.k)
    oracle.regret(w.runtimes[:R], seg, idx)
    sm = oracle.mlp(m, X)
    idx2, _ = oracle.topk(sm, seg, cfg.k)
    oracle.regret(w.runtimes[:R], seg, idx2)
    dt = time.perf_counter() - t0
    gf, gm = gpu_idx_forest[:n_problems], gpu_idx_mlp[:n_problems]
    parity = {"problems": n_problems,
              "forest_topk_equal": int(sum(np.array_equal(gf[p], idx[p]) for p in range(n_problems))),
              "mlp_top1_equal": int(np.sum(gm[:, 0] == idx2[:, 0])),
              "mlp_topk_equal": int(sum(np.array_equal(gm[p], idx2[p]) for p in range(n_problems)))}
    return {"value": R / dt, "unit": "rows/s", "cores": oracle.num_threads(), "kind": "oracle",
            "cpu": cpu_model(),
            "sample": f"first {n_problems} of {cfg.n_problems} problems ({R} rows), whole path "
                      f"(features, forest, MLP, top-{cfg.k}, regret), {dt:.1f} s"}, parity


def timed(torch, fn, reps: int = 3) -> float:
    """Median milliseconds of fn() over reps runs (HIP events on the current
    stream), after one untimed run."""
    fn()
    stream = torch.cuda.current_stream()
    out = []
    for _ in range(reps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        fn()
        e1.record(stream)
        torch.cuda.synchronize()
        out.append(e0.elapsed_time(e1))
    return float(np.median(out))


def extras(a, w, hwsel, torch, dev, probs, seg, cands, rt, forest, packed, X, idx, per_stage) -> dict:
    """Entries around the scored path on the same workload, each timed on its
    own (outside the timed step): the fused selection, the cheap scorers, the
    selection metrics and baselines, and the configuration catalogue."""
    import synth
    cfg = w.cfg
    R, P, F, k = cfg.rows, cfg.n_problems, cfg.n_features, cfg.k
    out = {}
    log("extras: fused selection")
    wsf = torch.empty(hwsel.hwsel_select_forest_workspace_bytes(forest, R), dtype=torch.uint8, device=dev)
    fidx = torch.empty((P, k), dtype=torch.int32, device=dev)
    ms = timed(torch, lambda: hwsel.hwsel_select_forest(w.hw, probs, seg, cands, F, forest, packed, k,
                                                        workspace=wsf, idx=fidx, with_vals=False))
    unfused = per_stage["features"] + per_stage["forest"] + per_stage["topk_forest"]
    out["fused_selection"] = {"ms": ms, "rows_per_s": R / (ms / 1e3), "unfused_ms": unfused,
                              "same_choice": bool(torch.equal(fidx, idx))}
    del wsf
    log("extras: linear and sampling scorers")
    lin = {kk: (hwsel.to_device(v, dev) if isinstance(v, np.ndarray) else v) for kk, v in synth.linear(cfg).items()}
    sl = torch.empty(R, dtype=torch.float32, device=dev)
    ms = timed(torch, lambda: hwsel.hwsel_linear_score(lin, X, scores=sl))
    gbs = R * (4 * F + 4) / (ms / 1e3) / 1e9
    out["linear_score"] = {"ms": ms, "rows_per_s": R / (ms / 1e3), "GBps": gbs, "hbm_frac": gbs / HBM_PEAK_GBS,
                           "bytes_per_row": 4 * F + 4}
    ms = timed(torch, lambda: hwsel.hwsel_sample_score(w.hw, probs, seg, cands, scores=sl))
    gbs = R * 21 / (ms / 1e3) / 1e9
    out["sample_score"] = {"ms": ms, "rows_per_s": R / (ms / 1e3), "GBps": gbs, "hbm_frac": gbs / HBM_PEAK_GBS,
                           "bytes_per_row": 21}
    log("extras: metrics and baselines")
    ms = timed(torch, lambda: hwsel.hwsel_evaluate(rt, seg, idx, per_group=False))
    gbs = R * 4 / (ms / 1e3) / 1e9
    out["evaluate"] = {"ms": ms, "GBps": gbs, "hbm_frac": gbs / HBM_PEAK_GBS, "problems": P}
    ids = hwsel.to_device(w.extra["config_id"], dev)
    n_cfg = int(w.extra["config_id"].max()) + 1
    ms = timed(torch, lambda: hwsel.hwsel_static_config(rt, seg, ids, n_cfg))
    out["static_config"] = {"ms": ms, "configs": n_cfg, "problems": P}
    log("extras: catalogue")
    mask = torch.empty((P, hwsel.HWSEL_CATALOGUE_SIZE), dtype=torch.uint8, device=dev)
    ms_mask = timed(torch, lambda: hwsel.hwsel_catalogue_mask(w.hw, probs, 1, mask=mask))
    _, n_valid = hwsel.hwsel_catalogue_mask(w.hw, probs, 1, mask=mask)
    total = int(n_valid.sum().item())
    pt = torch.empty(max(total, 1), dtype=torch.int32, device=dev)
    ms_comp = timed(torch, lambda: hwsel.hwsel_catalogue_compact(mask, n_valid, total, point=pt))
    cseg, _ = hwsel.hwsel_catalogue_compact(mask, n_valid, total, point=pt)
    ms_rows = timed(torch, lambda: hwsel.hwsel_catalogue_candidates(probs, cseg, total, point=pt))
    mbytes = P * hwsel.HWSEL_CATALOGUE_SIZE
    out["catalogue"] = {"problems": P, "points_per_problem": hwsel.HWSEL_CATALOGUE_SIZE, "valid_rows": total,
                        "mask_ms": ms_mask, "mask_points_per_s": mbytes / (ms_mask / 1e3),
                        "mask_hbm_frac": mbytes / (ms_mask / 1e3) / 1e9 / HBM_PEAK_GBS,
                        "compact_ms": ms_comp, "candidates_ms": ms_rows}
    del mask, pt
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--cpu-problems", type=int, default=64,
                    help="problems in the oracle's timed sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-extras", action="store_true",
                    help="skip the separately timed entries around the path (fused selection, cheap scorers, "
                         "metrics, catalogue)")
    ap.add_argument("--calibration-copy", action="store_true",
                    help="run one plain 1 GiB device-to-device copy before the timed region (a known-size "
                         "reference for the HBM byte counters)")
    a = ap.parse_args()
    if a.gpus != 1:
        print(f"bench.py: measures one GPU only (asked for --gpus {a.gpus}); "
              "the path shards by problem segment across GPUs, which is not built here.", file=sys.stderr)
        sys.exit(2)

    import torch
    import synth
    from paper_2609_35587_amd import hwsel

    torch.cuda.init()
    dev = torch.device("cuda:0")
    log("generate workload")
    w = synth.workload("dataset")
    mw = synth.mlp(synth.CONFIGS["mlp"])
    cfg = w.cfg
    R, P, F, k = cfg.rows, cfg.n_problems, cfg.n_features, cfg.k
    probs = hwsel.to_device(w.problems, dev)
    seg = hwsel.to_device(w.seg, dev)
    cands = {n: hwsel.to_device(v, dev) for n, v in w.cands.items()}
    rt = hwsel.to_device(w.runtimes, dev)
    forest = dict(w.forest)
    for n in ("node_feature", "node_threshold", "leaf_value"):
        forest[n] = hwsel.to_device(w.forest[n], dev)
    mlp = {n: hwsel.to_device(v, dev) for n, v in mw.items()}
    log("pack forest and MLP (once per model)")
    mlp_packed = hwsel.hwsel_mlp_pack(mlp)
    packed = hwsel.hwsel_forest_pack(forest)
    ws = torch.empty(hwsel.hwsel_forest_workspace_bytes(forest, R), dtype=torch.uint8, device=dev)
    X = torch.empty((R, F), dtype=torch.float32, device=dev)
    s_f = torch.empty(R, dtype=torch.float32, device=dev)
    s_m = torch.empty(R, dtype=torch.float32, device=dev)
    outs = [(torch.empty((P, k), dtype=torch.int32, device=dev), torch.empty((P, k), dtype=torch.float32, device=dev))
            for _ in range(2)]
    regs = [tuple(torch.empty(P, dtype=dt, device=dev) for dt in (torch.float32, torch.float32, torch.int32))
            for _ in range(2)]
    stream = torch.cuda.current_stream()
    stages = ["features", "forest", "topk_forest", "regret_forest", "mlp", "topk_mlp", "regret_mlp"]

    def step(ev=None):
        def mark(i):
            if ev is not None:
                ev[i].record(stream)
        mark(0)
        hwsel.hwsel_features(w.hw, probs, seg, cands, F, X=X)
        mark(1)
        hwsel.hwsel_forest_score(forest, X, scores=s_f, packed=packed, workspace=ws)
        mark(2)
        hwsel.hwsel_topk_per_problem(s_f, seg, k, idx=outs[0][0], vals=outs[0][1])
        mark(3)
        hwsel.hwsel_regret(rt, seg, outs[0][0], *regs[0])
        mark(4)
        hwsel.hwsel_mlp_score(mlp, X, scores=s_m, packed=mlp_packed)
        mark(5)
        hwsel.hwsel_topk_per_problem(s_m, seg, k, idx=outs[1][0], vals=outs[1][1])
        mark(6)
        hwsel.hwsel_regret(rt, seg, outs[1][0], *regs[1])
        mark(7)

    if a.calibration_copy:
        src = torch.ones(1 << 28, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        log("calibration copy: 1 GiB read + 1 GiB written")
        del src, dst
    log(f"warmup {a.warmup}")
    for _ in range(a.warmup):
        step()
    torch.cuda.synchronize()
    log(f"timed {a.steps}")
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(8)] for _ in range(a.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(a.steps):
        step(evs[i])
        log(f"  step {i + 1} enqueued")
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    per_stage = {name: float(np.mean([e[j].elapsed_time(e[j + 1]) for e in evs])) for j, name in enumerate(stages)}
    ms_step = float(np.mean([e[0].elapsed_time(e[7]) for e in evs]))
    log(f"stages ms {per_stage}  step {ms_step:.3f} ms  wall/step {1e3 * wall / a.steps:.3f} ms")

    # roofline of the dominant kernel (forest scoring): node visits per launch
    visits = R * cfg.trees * cfg.depth
    t_forest = per_stage["forest"] / 1e3
    visit_rate = visits / t_forest
    peak_visits = min(LANE_OPS_PER_S / VALU_OPS_PER_VISIT, LDS_LANES_PER_S / LDS_OPS_PER_VISIT)
    log("measured ceilings")
    ceil = ceilings(torch)
    mlp_flops = R * 918016 / (per_stage["mlp"] / 1e3)
    # algorithmic HBM bytes of the whole step: candidate records (17 B) + X write
    # (4F) + X read by forest and MLP (2 x 4F) + two score vectors written and
    # read (4 x 4 B) + runtimes read twice (2 x 4 B)
    step_bytes = R * (17 + 3 * 4 * F + 16 + 8)
    hbm_gbs = step_bytes / (ms_step / 1e3) / 1e9
    forest_bytes = R * (4 * F + 4)
    line = {
        "metric": METRIC, "value": R / (ms_step / 1e3), "unit": "rows/s", "n_gpus": 1, "steps": a.steps,
        "warmup": a.warmup, "ms_per_step": ms_step, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": {"workload": "dataset-scale: 600 problems x 8192 candidates = 4915200 rows, 128 features, "
                               "GBDT 2000 trees depth 10 + MLP 128-512-512-256-1 (bf16), top-10 + regret",
                   "rows": R, "problems": P, "features": F, "trees": cfg.trees, "depth": cfg.depth, "k": k},
        "stages_ms": per_stage,
        "hbm_roofline_step": {"achieved": hbm_gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                              "frac": hbm_gbs / HBM_PEAK_GBS, "bytes_per_row": step_bytes / R},
        "roofline": {"kernel": "hwsel_forest_score (k_bin + k_traverse<16,10> + k_reduce)", "bound": "alu",
                     "achieved": visit_rate / 1e9, "peak": peak_visits / 1e9, "unit": "Gvisits/s",
                     "frac": visit_rate / peak_visits, "traffic": forest_traffic_bytes(),
                     "visits_per_launch": visits,
                     "measured_ceiling": ceil["visits_per_s"] / 1e9,
                     "frac_of_measured_ceiling": visit_rate / ceil["visits_per_s"],
                     "hbm_frac": forest_bytes / t_forest / 1e9 / HBM_PEAK_GBS},
        "rooflines_other": {
            "mlp": {"kernel": "hwsel_mlp_score (k_mlp_mfma)", "bound": "mfma", "unit": "TFLOP/s",
                    "achieved": mlp_flops / 1e12, "peak": BF16_PEAK_TFLOPS,
                    "frac": mlp_flops / 1e12 / BF16_PEAK_TFLOPS,
                    "measured_ceiling": ceil["bf16_flops_per_s"] / 1e12,
                    "frac_of_measured_ceiling": mlp_flops / ceil["bf16_flops_per_s"]},
            "features": {"kernel": "hwsel_features (k_features<128>)", "bound": "hbm", "unit": "GB/s",
                         "achieved": R * (17 + 4 * F) / (per_stage["features"] / 1e3) / 1e9, "peak": HBM_PEAK_GBS,
                         "frac": R * (17 + 4 * F) / (per_stage["features"] / 1e3) / 1e9 / HBM_PEAK_GBS,
                         "measured_ceiling": ceil["fill_GBps"],
                         "frac_of_measured_ceiling": R * (17 + 4 * F) / (per_stage["features"] / 1e3) / 1e9
                         / ceil["fill_GBps"]},
        },
        "measured_ceilings": ceil,
    }
    picks = (outs[0][0].cpu().numpy(), outs[1][0].cpu().numpy())
    if not a.no_extras:
        line["extras"] = extras(a, w, hwsel, torch, dev, probs, seg, cands, rt, forest, packed, X, outs[0][0],
                                per_stage)
        del X, ws, s_f, s_m
        for name in ("tiny", "medium", "full"):
            log(f"extras: {name} workload")
            line["extras"][f"workload_{name}"] = per_config(hwsel, torch, dev, name)
            torch.cuda.empty_cache()
    if not a.no_cpu_baseline:
        log(f"cpu baseline: oracle on {a.cpu_problems} problems")
        line["cpu_baseline"], line["parity"] = cpu_baseline(w, a.cpu_problems, *picks)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
