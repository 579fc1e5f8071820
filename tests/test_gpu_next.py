"""GPU parity of the entries around the scored path: the cheap scorers (linear
ridge model, analytic sampling score), the selection metrics and baselines,
and the configuration catalogue -- the HIP library through its C ABI against
the CPU oracle, on identical inputs (inputs come from the generator or the
oracle, never from the library).

Acceptance:
  linear score   - |g - o| <= 1e-5 * (sum of the terms' magnitudes);
  sampling score - within 1e-6 relative (the same binary64 sequence; bit-exact
                   expected) -- it is feature column 58;
  evaluation     - regret, rank and every aggregate but the random-pick
                   regret bit-exact; ybar and the random-pick regret within
                   1e-12 relative (a different summation order);
  static config  - id, count and mean y bit-exact (same summation order);
  catalogue      - mask, counts, offsets, points and decoded knobs bit-exact.
"""
import numpy as np
import pytest
import torch

import oracle
import synth
from _gpu_util import Dev, say
from paper_2609_35587_amd import hwsel

pytestmark = pytest.mark.gpu


def up(a):
    return hwsel.to_device(np.ascontiguousarray(a))


def lin_dev(m):
    return {k: (up(v) if isinstance(v, np.ndarray) else v) for k, v in m.items()}


# ----------------------------------------------------------------------------
# linear ridge scorer
# ----------------------------------------------------------------------------
@pytest.mark.parametrize("F,R", [(64, 1), (64, 999), (96, 2048), (128, 4097)])
def test_linear_random_rows(F, R):
    say(f"linear F={F} R={R}")
    rng = np.random.default_rng(F + R)
    X = rng.normal(0, 3, (R, F)).astype(np.float32)
    X[rng.random((R, F)) < 0.01] = np.nan
    X[rng.random((R, F)) < 0.01] = np.inf
    if F > 64:
        for col, lv in ((64, 4), (73, 3), (74, 3), (75, 2)):
            X[:, col] = rng.integers(-1, lv + 1, R)          # includes unseen levels
        X[: R // 10, 73] = 0.5
    m = {"n_features": F, "bias": 0.375, "mean": rng.normal(0, 1, F).astype(np.float32),
         "inv_std": rng.uniform(0, 2, F).astype(np.float32), "w": rng.normal(0, 1, F).astype(np.float32),
         "w_onehot": rng.normal(0, 1, 12).astype(np.float32)}
    o, mag = oracle.linear(m, X)
    g = hwsel.hwsel_linear_score(lin_dev(m), up(X)).cpu().numpy()
    err = np.abs(g.astype(np.float64) - o)
    assert np.all(err <= 1e-5 * mag), f"worst row {int(np.argmax(err / mag))}"
    say(f"  max err/bound {float(np.max(err / (1e-5 * mag))):.3g}, bit-exact rows {int((g == o).sum())}/{R}")


def test_linear_dataset_rows_in_padded_matrix():
    say("linear dataset rows, ld 132")
    cfg = synth.CONFIGS["dataset"]
    w = synth.workload("dataset", with_runtimes=False, with_model=False)
    rows = synth.sample_rows(cfg, 20000)
    X = oracle.features(w.hw, w.problems, w.seg, w.cands, 128, rows=rows)
    Xp = np.zeros((len(X), 132), np.float32)
    Xp[:, :128] = X
    m = synth.linear(cfg)
    o, mag = oracle.linear(m, X)
    g = hwsel.hwsel_linear_score(lin_dev(m), up(Xp)[:, :].contiguous()).cpu().numpy()
    assert np.all(np.abs(g.astype(np.float64) - o) <= 1e-5 * mag)
    # top-k of the linear scores agrees with the oracle's on the same scores
    seg = np.arange(0, len(X) + 1, 1000, dtype=np.int64)
    gi, _ = hwsel.hwsel_topk_per_problem(up(o), up(seg), 10)
    oi, _ = oracle.topk(o, seg, 10)
    assert np.array_equal(gi.cpu().numpy(), oi)


# ----------------------------------------------------------------------------
# analytic sampling score
# ----------------------------------------------------------------------------
@pytest.mark.parametrize("name", ["tiny", "medium", "dataset"])
def test_sampling_score_is_column_58(name):
    say(f"sampling score {name}")
    w = synth.workload(name, with_runtimes=False, with_model=False)
    d = Dev(w)
    g = hwsel.hwsel_sample_score(w.hw, d.problems, d.seg, d.cands).cpu().numpy()
    rows = synth.sample_rows(w.cfg, 50000)
    o = oracle.features(w.hw, w.problems, w.seg, w.cands, 64, rows=rows)[:, 58]
    rel = np.abs(g[rows].astype(np.float64) - o) / np.maximum(np.abs(o), 1e-30)
    assert rel.max() <= 1e-6
    say(f"  max rel {rel.max():.3g}, not bit-exact {int((g[rows] != o).sum())}")


# ----------------------------------------------------------------------------
# evaluation metrics and baselines
# ----------------------------------------------------------------------------
def eval_compare(rt, seg, idx):
    o_agg, o_reg, o_rank, o_ybar = oracle.evaluate(rt, seg, idx)
    out, reg, rank, ybar = hwsel.hwsel_evaluate(up(rt), up(seg), up(idx))
    out, reg, rank, ybar = (t.cpu().numpy() for t in (out, reg, rank, ybar))
    o_out = np.array([o_agg[f] for f in oracle.EVAL_FIELDS])
    assert np.array_equal(rank, o_rank)
    assert np.array_equal(reg, o_reg, equal_nan=True)
    both_nan = np.isnan(ybar) & np.isnan(o_ybar)
    assert np.array_equal(np.isnan(ybar), np.isnan(o_ybar))
    assert np.all(np.abs(ybar[~both_nan] - o_ybar[~both_nan]) <= 1e-12 * np.abs(o_ybar[~both_nan]) + 1e-300)
    exact = [0, 1, 2, 3, 4, 5, 6, 8]
    assert np.array_equal(out[exact], o_out[exact], equal_nan=True), (out, o_out)
    if o_out[8] > 0:
        assert abs(out[7] - o_out[7]) <= 1e-12 * abs(o_out[7]) + 1e-300
    else:
        assert np.isnan(out[7])
    return o_agg


@pytest.mark.parametrize("seed,k", [(0, 1), (1, 5), (2, 10), (3, 64)])
def test_evaluate_ragged_with_edges(seed, k):
    say(f"evaluate ragged seed={seed} k={k}")
    rng = np.random.default_rng(seed)
    seg = synth.ragged_segments(rng, 97, 300)
    R = int(seg[-1])
    rt = rng.lognormal(0, 0.3, R).astype(np.float32)
    rt[rng.random(R) < 0.05] = np.inf
    rt[rng.random(R) < 0.01] = np.nan
    rt[rng.random(R) < 0.1] = 1.0                     # ties
    scores = synth.random_scores(rng, R, tie_frac=0.3)
    idx, _ = oracle.topk(scores, seg, k)
    eval_compare(rt, seg, idx)


def test_evaluate_all_nan_and_single_group():
    rt = np.array([np.nan, np.nan, 3.0, 1.0], np.float32)
    agg = eval_compare(rt, np.array([0, 2, 4], np.int64), np.array([[1], [0]], np.int32))
    assert agg["n_groups"] == 2 and agg["max_regret"] == 1.0
    eval_compare(np.array([2.0], np.float32), np.array([0, 1], np.int64), np.array([[0]], np.int32))
    # an empty segment (the runtime array is not read)
    eval_compare(np.ones(1, np.float32), np.array([0, 0], np.int64), np.array([[-1]], np.int32))


def test_evaluate_dataset_forest_selection():
    say("evaluate dataset-scale, oracle top-10 of random scores")
    w = synth.workload("dataset", with_model=False)
    rng = np.random.default_rng(7)
    scores = rng.standard_normal(len(w.runtimes)).astype(np.float32)
    idx, _ = oracle.topk(scores, w.seg, 10)
    agg = eval_compare(w.runtimes, w.seg, idx)
    idx2, _ = oracle.topk(-w.runtimes, w.seg, 10)
    agg2 = eval_compare(w.runtimes, w.seg, idx2)
    assert agg2["mean_regret"] == 0.0 and agg2["top1"] == 1.0
    say(f"  random scores: mean regret {agg['mean_regret']:.4f}, random-pick {agg['random_regret']:.4f}")


@pytest.mark.parametrize("name", ["medium", "dataset"])
def test_static_config(name):
    say(f"static config {name}")
    w = synth.workload(name, with_model=False)
    ids = w.extra["config_id"]
    n_cfg = int(ids.max()) + 1
    ob, oc, oy = oracle.static_config(w.runtimes, w.seg, ids, n_cfg)
    best, my = hwsel.hwsel_static_config(up(w.runtimes), up(w.seg), up(ids), n_cfg)
    best, my = best.cpu().numpy(), my.cpu().numpy()
    assert (int(best[0]), int(best[1])) == (ob, oc)
    assert (np.isnan(my[0]) and np.isnan(oy)) or my[0] == oy
    # a configuration present in every group: make the first row of every
    # segment the same id and the fastest
    ids2 = ids.copy()
    rt2 = w.runtimes.copy()
    ids2[w.seg[:-1]] = n_cfg
    rt2[w.seg[:-1]] = 1e-9
    ob2, oc2, oy2 = oracle.static_config(rt2, w.seg, ids2, n_cfg + 1)
    b2, my2 = hwsel.hwsel_static_config(up(rt2), up(w.seg), up(ids2), n_cfg + 1)
    assert (ob2, oc2, oy2) == (n_cfg, w.cfg.n_problems, 1.0)
    assert int(b2[0]) == ob2 and int(b2[1]) == oc2 and float(my2[0]) == 1.0
    say(f"  best id {ob} in {oc} groups, mean y {oy:.4f}")


# ----------------------------------------------------------------------------
# configuration catalogue
# ----------------------------------------------------------------------------
def catalogue_problems():
    pr = np.zeros(9, synth.PROBLEM_DTYPE)
    pr["M"] = [4096, 64, 100, 8192, 16, 2048, 333, 1, 12000]
    pr["N"] = [4096, 4096, 8192, 64, 16, 2048, 77, 1, 40]
    pr["K"] = [4096, 128, 256, 65536, 16, 2048, 999, 1, 300]
    pr["layout"] = [0, 1, 2, 3, 0, 3, 2, 1, 0]
    pr["dtype"] = [0, 1, 2, 0, 0, 2, 1, 0, 2]
    return pr


@pytest.mark.parametrize("flags", [0, 1])
def test_catalogue_mask_compact_and_rows(flags):
    say(f"catalogue flags={flags}")
    hw = synth.hardware()
    pr = catalogue_problems()
    om, on = oracle.catalogue_mask(hw, pr, flags)
    oseg, opoint = oracle.catalogue_compact(om)
    prd = up(pr)
    mask, n_valid = hwsel.hwsel_catalogue_mask(hw, prd, flags)
    assert np.array_equal(n_valid.cpu().numpy(), on)
    assert np.array_equal(mask.cpu().numpy(), om)
    cap = int(oseg[-1])
    seg, point = hwsel.hwsel_catalogue_compact(mask, n_valid, cap)
    assert np.array_equal(seg.cpu().numpy(), oseg)
    assert np.array_equal(point.cpu().numpy()[:cap], opoint)
    # a short capacity writes the prefix only
    seg2, point2 = hwsel.hwsel_catalogue_compact(mask, n_valid, 1000)
    assert np.array_equal(point2.cpu().numpy(), opoint[:1000])
    # decoded rows of the valid list, and the whole catalogue of one problem
    c = hwsel.hwsel_catalogue_candidates(prd, seg, cap, point=point)
    rows = np.random.default_rng(flags).choice(cap, 20000, replace=False)
    for p in range(len(pr)):
        sel = rows[(rows >= oseg[p]) & (rows < oseg[p + 1])]
        ref = oracle.catalogue_decode(opoint[sel], int(pr["dtype"][p]))
        for n in hwsel.CAND_FIELDS:
            got = c[n].cpu().numpy()[sel]
            assert np.array_equal(got.view(ref[n].dtype), ref[n]), (p, n)
    one = np.array([0, oracle.catalogue_size()], np.int64)
    c1 = hwsel.hwsel_catalogue_candidates(up(pr[5:6]), up(one), oracle.catalogue_size())
    ref = oracle.catalogue_decode(np.arange(oracle.catalogue_size()), int(pr["dtype"][5]))
    for n in hwsel.CAND_FIELDS:
        assert np.array_equal(c1[n].cpu().numpy().view(ref[n].dtype), ref[n]), n
    say(f"  valid per problem {on.tolist()}")


def test_catalogue_rows_feed_the_scored_path():
    """Valid catalogue -> features -> sampling score equals column 58."""
    say("catalogue -> features")
    hw = synth.hardware()
    pr = catalogue_problems()[:3]
    prd = up(pr)
    mask, n_valid = hwsel.hwsel_catalogue_mask(hw, prd, 1)
    cap = int(n_valid.sum().item())
    seg, point = hwsel.hwsel_catalogue_compact(mask, n_valid, cap)
    c = hwsel.hwsel_catalogue_candidates(prd, seg, cap, point=point)
    X = hwsel.hwsel_features(hw, prd, seg, c, 128).cpu().numpy()
    s = hwsel.hwsel_sample_score(hw, prd, seg, c).cpu().numpy()
    assert np.array_equal(s, X[:, 58])
    assert np.all(X[:, 87] == 1) and np.all(X[:, 86] == 1)


# ----------------------------------------------------------------------------
# fused selection: features -> bins -> forest -> top-k in one call
# ----------------------------------------------------------------------------
@pytest.mark.parametrize("name", ["tiny", "medium", "dataset"])
def test_fused_selection(name):
    from _gpu_util import check_selection
    say(f"fused selection {name}")
    w = synth.workload(name)
    cfg = w.cfg
    d = Dev(w)
    packed = hwsel.hwsel_forest_pack(d.forest)
    ws = torch.empty(hwsel.hwsel_forest_workspace_bytes(d.forest, cfg.rows), dtype=torch.uint8, device="cuda")
    X = d.features(cfg.n_features)
    s = hwsel.hwsel_forest_score(d.forest, X, packed=packed, workspace=ws)
    idx, vals = hwsel.hwsel_topk_per_problem(s, d.seg, cfg.k)
    del X
    fs = torch.empty(cfg.rows, dtype=torch.float32, device="cuda")
    fidx, fvals, _ = hwsel.hwsel_select_forest(w.hw, d.problems, d.seg, d.cands, cfg.n_features, d.forest, packed,
                                               cfg.k, scores=fs)
    assert bool((fs.view(torch.int32) == s.view(torch.int32)).all())
    assert np.array_equal(fidx.cpu().numpy(), idx.cpu().numpy())
    assert np.array_equal(fvals.cpu().numpy().view(np.uint32), vals.cpu().numpy().view(np.uint32))
    # no scores requested: the workspace holds them
    fidx2, _, _ = hwsel.hwsel_select_forest(w.hw, d.problems, d.seg, d.cands, cfg.n_features, d.forest, packed,
                                            cfg.k, with_vals=False)
    assert np.array_equal(fidx2.cpu().numpy(), idx.cpu().numpy())
    probs = np.arange(cfg.n_problems) if name == "tiny" else \
        np.random.default_rng(cfg.seed + 1).choice(cfg.n_problems, 2, replace=False)
    check_selection(w, fidx.cpu().numpy(), probs)


@pytest.mark.parametrize("P", [4096, 4097])
def test_evaluate_problem_count_boundary(P):
    """Both order-statistic paths (one workgroup up to 4,096 problems, radix selection above)."""
    say(f"evaluate {P} problems")
    rng = np.random.default_rng(P)
    seg = synth.ragged_segments(rng, P, 9, empty_frac=0.05)
    R = int(seg[-1])
    rt = rng.choice(np.array([1.0, 1.5, 2.0, 3.0, np.inf, np.nan], np.float32), R)
    idx, _ = oracle.topk(rng.standard_normal(R).astype(np.float32), seg, 2)
    eval_compare(rt, seg, idx)


def test_evaluate_many_problems():
    """Order statistics over many problems (radix selection, linear in P)."""
    say("evaluate 50,000 problems")
    rng = np.random.default_rng(11)
    seg = synth.ragged_segments(rng, 50000, 12, empty_frac=0.05)
    R = int(seg[-1])
    rt = rng.choice(np.array([1.0, 1.25, 1.5, 2.0, 4.0, np.inf], np.float32), R)
    idx, _ = oracle.topk(rng.standard_normal(R).astype(np.float32), seg, 1)
    eval_compare(rt, seg, idx)


def test_catalogue_rows_any_field_alignment():
    """Field arrays offset by one element (so no packed stores apply) give
    the oracle's rows too, with a row count that is not a multiple of four
    and segments that end inside a group of four rows."""
    say("catalogue rows, misaligned fields")
    pr = catalogue_problems()[[0, 2, 5]]
    seg = np.array([0, 1001, 2003, 2010], np.int64)
    R = int(seg[-1])
    wide = ("tile_m", "tile_n", "tile_k", "inst_n")
    bufs = {n: torch.zeros(R + 1, dtype=torch.int16 if n in wide else torch.uint8, device="cuda")
            for n in hwsel.CAND_FIELDS}
    prd = up(pr)
    for off in (0, 1):
        out = {n: t[off:off + R] for n, t in bufs.items()}
        c = hwsel.hwsel_catalogue_candidates(prd, up(seg), R, out=out)
        for p in range(len(pr)):
            ref = oracle.catalogue_decode(np.arange(seg[p + 1] - seg[p]), int(pr["dtype"][p]))
            for n in hwsel.CAND_FIELDS:
                got = c[n].cpu().numpy()[seg[p]:seg[p + 1]]
                assert np.array_equal(got.view(ref[n].dtype), ref[n]), (off, p, n)


# ----------------------------------------------------------------------------
# binding: short, mistyped or misplaced buffers are refused before any launch
# ----------------------------------------------------------------------------
def test_binding_rejects_bad_buffers():
    w = synth.workload("tiny")
    d = Dev(w)
    R = w.cfg.rows
    X = d.features(64)
    dev = X.device
    bad = [
        lambda: hwsel.hwsel_features(w.hw, d.problems, d.seg, d.cands, 64, X=torch.empty((R - 1, 64), device=dev)),
        lambda: hwsel.hwsel_features(w.hw, d.problems, d.seg, d.cands, 64, X=torch.empty((R, 64), device=dev,
                                                                                         dtype=torch.float64)),
        lambda: hwsel.hwsel_forest_score(d.forest, X, scores=torch.empty(R - 1, device=dev)),
        lambda: hwsel.hwsel_forest_score(d.forest, X[:, :32]),
        lambda: hwsel.hwsel_forest_score(d.forest, X, packed=torch.empty(100, dtype=torch.uint8, device=dev)),
        lambda: hwsel.hwsel_topk_per_problem(torch.zeros(R, device=dev), d.seg, 5,
                                             idx=torch.empty((w.cfg.n_problems, 4), dtype=torch.int32, device=dev)),
        lambda: hwsel.hwsel_topk_per_problem(torch.zeros(R, device=dev), d.seg, 5,
                                             idx=torch.empty((w.cfg.n_problems, 5), dtype=torch.int64, device=dev)),
        lambda: hwsel.hwsel_regret(d.runtimes, d.seg, torch.zeros((w.cfg.n_problems, 5), dtype=torch.int32,
                                                                  device=dev), r1=torch.empty(3, device=dev)),
        lambda: hwsel.hwsel_mlp_score(mlp_dev, torch.zeros((10, 128), device=dev), scores=torch.empty(9, device=dev)),
        lambda: hwsel.hwsel_catalogue_compact(torch.zeros((2, 10), dtype=torch.uint8, device=dev),
                                              torch.zeros(2, dtype=torch.int64, device=dev), 5),
    ]
    mlp_dev = {k: up(v) for k, v in synth.mlp(synth.CONFIGS["mlp"]).items()}
    for i, call in enumerate(bad):
        with pytest.raises(ValueError):
            call()
            say(f"  case {i} was not refused")
