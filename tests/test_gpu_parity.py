"""GPU parity: the HIP library (through its C ABI) against the CPU oracle.

Small workloads are compared on every row; the large ones run at full size
in the launch configuration the benchmark times and are compared on a seeded
row sample the oracle evaluates one by one, plus properties that hold at any
size.  Acceptance:
  features  - integer columns bit-exact, other columns within 1e-6 relative;
  forest    - leaf indices bit-exact, scores within 1e-5 * max(|o|, L1 of the
              row's leaf values);
  MLP       - within 2e-2 * max(|o|, rms of the oracle scores);
  top-k     - bit-exact indices on identical scores;
  regret    - bit-exact.
"""
import numpy as np
import pytest
import torch

import oracle
import synth
from _gpu_util import Dev, assert_forest_scores, check_selection, compare_features, path_l1, say
from paper_2609_35587_amd import hwsel

pytestmark = pytest.mark.gpu

SAMPLE = 65536


@pytest.fixture(scope="module")
def tiny():
    w = synth.workload("tiny")
    return w, Dev(w)


# ----------------------------------------------------------------------------
# tiny: every row, every stage, plus the end-to-end selection
# ----------------------------------------------------------------------------
def test_features_tiny_all_rows(tiny):
    w, d = tiny
    say("features tiny")
    X = d.features(64).cpu().numpy()
    ref = oracle.features(w.hw, w.problems, w.seg, w.cands, 64)
    say(f"  {compare_features(X, ref, 64)}")


@pytest.mark.parametrize("F", [64, 96, 128])
def test_features_ragged_segments(tiny, F):
    """Segments of 0 to 300 rows: workgroups of 256 rows that span many
    problems (more than the kernel computes problem terms for once), problems
    that change inside a wave, empty segments; every row and column against
    the oracle."""
    w, _ = tiny
    rng = np.random.default_rng(F)
    lengths = rng.choice([0, 0, 1, 2, 3, 5, 17, 63, 64, 65, 130, 300], size=160)
    lengths = lengths[np.cumsum(lengths) <= len(w.cands["tile_m"])]
    seg = np.concatenate([[0], np.cumsum(lengths)]).astype(np.int64)
    R = int(seg[-1])
    probs = w.problems[rng.integers(0, len(w.problems), len(lengths))]
    cands = {k: np.ascontiguousarray(v[:R]) for k, v in w.cands.items()}
    say(f"features ragged F={F}: {len(lengths)} problems, {R} rows")
    X = hwsel.hwsel_features(w.hw, hwsel.to_device(probs), hwsel.to_device(seg),
                             {k: hwsel.to_device(v) for k, v in cands.items()}, F).cpu().numpy()
    ref = oracle.features(w.hw, probs, seg, cands, F)
    say(f"  {compare_features(X, ref, F)}")


def test_forest_tiny_all_rows(tiny):
    w, d = tiny
    say("forest tiny")
    ref_X = oracle.features(w.hw, w.problems, w.seg, w.cands, 64)
    Xd = torch.from_numpy(ref_X).cuda()             # identical input on both sides
    rows = torch.arange(len(ref_X), dtype=torch.int64, device="cuda")
    li = hwsel.hwsel_forest_leaves(d.forest, Xd, rows).cpu().numpy().view(np.uint16)
    o, oli = oracle.forest(w.forest, ref_X, leaves=True)
    assert np.array_equal(li, oli)
    l1 = path_l1(w.forest, oli)
    s = hwsel.hwsel_forest_score(d.forest, Xd).cpu().numpy()
    say(f"  direct walk: score err/bound max {assert_forest_scores(s, o, l1):.3g}")
    packed = hwsel.hwsel_forest_pack(d.forest)
    sp = hwsel.hwsel_forest_score(d.forest, Xd, packed=packed).cpu().numpy()
    say(f"  packed: score err/bound max {assert_forest_scores(sp, o, l1):.3g}")
    sp2 = hwsel.hwsel_forest_score(d.forest, Xd, packed=packed).cpu().numpy()
    assert np.array_equal(sp.view(np.uint32), sp2.view(np.uint32))      # run-to-run identical


def test_features_and_forest_in_a_wider_matrix(tiny):
    """X as the first 64 columns of a 76-column matrix: features land in those
    columns only, bit-identical to a contiguous X, and both forest paths
    score the strided X exactly as the contiguous one."""
    w, d = tiny
    say("features + forest, ld 76")
    R = w.cands["tile_m"].shape[0]
    wide = torch.full((R, 76), -7.0, dtype=torch.float32, device="cuda")
    Xs = hwsel.hwsel_features(w.hw, d.problems, d.seg, d.cands, 64, X=wide[:, :64])
    Xc = d.features(64)
    assert Xs.stride(0) == 76
    assert bool((Xs.view(torch.int32) == Xc.view(torch.int32)).all())
    assert bool((wide[:, 64:] == -7.0).all())
    packed = hwsel.hwsel_forest_pack(d.forest)
    for pk in (None, packed):
        a = hwsel.hwsel_forest_score(d.forest, Xs, packed=pk)
        b = hwsel.hwsel_forest_score(d.forest, Xc, packed=pk)
        assert bool((a.view(torch.int32) == b.view(torch.int32)).all())


def _leaf_probe(forest: dict, t0: int) -> dict:
    """Same nodes, leaves zero except tree t0 whose leaf l holds the value l:
    the ensemble's score is exactly the leaf index reached in tree t0."""
    f = dict(forest)
    lv = np.zeros_like(forest["leaf_value"])
    lv[t0] = np.arange(lv.shape[1], dtype=np.float32)
    f["leaf_value"] = lv
    return f


def test_selection_tiny_end_to_end(tiny):
    w, d = tiny
    say("pipeline tiny")
    k = w.cfg.k
    X = d.features(64)
    s = hwsel.hwsel_forest_score(d.forest, X)
    idx, vals = hwsel.hwsel_topk_per_problem(s, d.seg, k)
    r1, rk, best = hwsel.hwsel_regret(d.runtimes, d.seg, idx)
    torch.cuda.synchronize()
    ref_X = oracle.features(w.hw, w.problems, w.seg, w.cands, 64)
    o = oracle.forest(w.forest, ref_X)
    oidx, ovals = oracle.topk(o, w.seg, k)
    assert np.array_equal(idx.cpu().numpy(), oidx)
    o1, ok, ob = oracle.regret(w.runtimes, w.seg, oidx)
    assert np.array_equal(r1.cpu().numpy().view(np.uint32), o1.view(np.uint32))
    assert np.array_equal(rk.cpu().numpy().view(np.uint32), ok.view(np.uint32))
    assert np.array_equal(best.cpu().numpy(), ob)
    say(f"  mean regret top1 {o1.mean():.4f} best-of-{k} {ok.mean():.4f}")


# ----------------------------------------------------------------------------
# top-k and regret: ragged and empty segments, ties, NaN, signed zeros, k range
# ----------------------------------------------------------------------------
@pytest.mark.parametrize("k", [1, 5, 16, 64])
def test_topk_regret_edge_cases(k):
    say(f"topk/regret edge k={k}")
    rng = np.random.default_rng(100 + k)
    seg = synth.ragged_segments(rng, 300, 700, empty_frac=0.1)
    seg[-1] = seg[-2]          # the last segment empty too
    R = int(seg[-1])
    s = synth.random_scores(rng, R, tie_frac=0.4, n_levels=3)
    s[rng.random(R) < 0.02] = np.nan
    s[rng.random(R) < 0.02] = -0.0
    s[rng.random(R) < 0.02] = 0.0
    s[rng.random(R) < 0.01] = -np.inf
    s[rng.random(R) < 0.01] = np.inf
    rt = np.exp(rng.standard_normal(R)).astype(np.float32)
    rt[rng.random(R) < 0.03] = np.inf
    rt[rng.random(R) < 0.03] = np.nan      # never finishing: a NaN pick has regret 1
    rt[rng.random(R) < 0.2] = 1.0          # many equal runtimes
    sd, segd, rtd = (torch.from_numpy(a).cuda() for a in (s, seg, rt))
    idx, vals = hwsel.hwsel_topk_per_problem(sd, segd, k)
    oidx, ovals = oracle.topk(s, seg, k)
    assert np.array_equal(idx.cpu().numpy(), oidx)
    assert np.array_equal(vals.cpu().numpy().view(np.uint32), ovals.view(np.uint32))
    r1, rk, best = hwsel.hwsel_regret(rtd, segd, idx)
    o1, ok, ob = oracle.regret(rt, seg, oidx)
    assert np.array_equal(r1.cpu().numpy().view(np.uint32), o1.view(np.uint32))
    assert np.array_equal(rk.cpu().numpy().view(np.uint32), ok.view(np.uint32))
    assert np.array_equal(best.cpu().numpy(), ob)


def test_topk_single_long_segment_and_all_ties():
    say("topk long segment")
    n = 65536 * 3 + 17
    seg = np.array([0, n, n + 5], np.int64)
    s = np.zeros(n + 5, np.float32)
    s[12345] = 1.0
    idx, _ = hwsel.hwsel_topk_per_problem(torch.from_numpy(s).cuda(), torch.from_numpy(seg).cuda(), 64)
    oidx, _ = oracle.topk(s, seg, 64)
    assert np.array_equal(idx.cpu().numpy(), oidx)
    assert oidx[0, 0] == 12345 and oidx[0, 1:].tolist() == list(range(63))


@pytest.mark.parametrize("k", [1, 16, 64])
def test_topk_long_segments_tile_merge(k):
    """Segments longer than one register tile (8,192 rows): read once, tile
    by tile, with a running list of the k best -- against the oracle's full
    sort on orders that stress the merge (best rows last, first, spread over
    tiles; heavy ties; NaN and infinities) and lengths around tile edges."""
    say(f"topk long segments k={k}")
    rng = np.random.default_rng(500 + k)
    lens = [8193, 16384, 16385, 40000, 65536, 8192 * 5 + 3, 100, 0, 70001]
    seg = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    R = int(seg[-1])
    s = synth.random_scores(rng, R, tie_frac=0.3, n_levels=5)
    a0, a1, a2, a3 = seg[0], seg[1], seg[2], seg[3]
    s[a0:a1] = np.arange(a1 - a0, dtype=np.float32)             # ascending: every tile beats the last
    s[a1:a2] = -np.arange(a2 - a1, dtype=np.float32)            # descending: the first tile wins
    s[a2:a3] = 7.0                                              # all ties: lowest indices win
    b = seg[4]
    s[b:b + 50] = np.nan
    s[b + 60000] = np.inf
    s[b + 30000] = -np.inf
    idx, vals = hwsel.hwsel_topk_per_problem(torch.from_numpy(s).cuda(), torch.from_numpy(seg).cuda(), k)
    oidx, ovals = oracle.topk(s, seg, k)
    assert np.array_equal(idx.cpu().numpy(), oidx)
    assert np.array_equal(vals.cpu().numpy().view(np.uint32), ovals.view(np.uint32))


# ----------------------------------------------------------------------------
# Full-size workloads: sampled rows + properties
# ----------------------------------------------------------------------------
@pytest.mark.parametrize("name", ["medium", "full", "dataset"])
def test_forest_workload_full_size(name):
    say(f"workload {name}: generate")
    w = synth.workload(name)
    cfg = w.cfg
    d = Dev(w)
    say(f"workload {name}: features R={cfg.rows} F={cfg.n_features}")
    X = d.features(cfg.n_features)
    rows = synth.sample_rows(cfg, SAMPLE)
    rows_d = torch.from_numpy(rows).cuda()
    Xs = X.index_select(0, rows_d).cpu().numpy()
    ref = oracle.features(w.hw, w.problems, w.seg, w.cands, cfg.n_features, rows)
    say(f"  features {compare_features(Xs, ref, cfg.n_features)}")
    say(f"workload {name}: forest {cfg.trees}x{cfg.depth}, packed path as benchmarked")
    packed = hwsel.hwsel_forest_pack(d.forest)
    ws = torch.empty(hwsel.hwsel_forest_workspace_bytes(d.forest, cfg.rows), dtype=torch.uint8, device="cuda")
    s = hwsel.hwsel_forest_score(d.forest, X, packed=packed, workspace=ws)
    li = hwsel.hwsel_forest_leaves(d.forest, X, rows_d).cpu().numpy().view(np.uint16)
    o, oli = oracle.forest(w.forest, ref, leaves=True)
    assert np.array_equal(li, oli)
    l1 = path_l1(w.forest, oli)
    g = s.index_select(0, rows_d).cpu().numpy()
    say(f"  packed forest err/bound {assert_forest_scores(g, o, l1):.3g}")
    assert bool(torch.isfinite(s).all())
    # leaf indices of the packed traversal itself, for a few trees, on every row
    for t0 in (0, cfg.trees // 2 + 1, cfg.trees - 1):
        probe = _leaf_probe(w.forest, t0)
        from _gpu_util import forest_to_device
        pd = forest_to_device(probe)
        sp = hwsel.hwsel_forest_score(pd, X, packed=hwsel.hwsel_forest_pack(pd), workspace=ws)
        assert np.array_equal(sp.index_select(0, rows_d).cpu().numpy(), oli[:, t0].astype(np.float32)), t0
        # and on every row, against the direct walk's leaves
        sg = hwsel.hwsel_forest_score(pd, X)
        assert bool((sp == sg).all()), t0
    say("  packed leaf indices match for probed trees")
    say(f"workload {name}: end-to-end selection on sampled problems")
    idx = hwsel.hwsel_topk_per_problem(s, d.seg, cfg.k, with_vals=False)[0].cpu().numpy()
    check_selection(w, idx, np.random.default_rng(cfg.seed).choice(cfg.n_problems, 3, replace=False))
    say(f"workload {name}: top-k / regret at full size on generator scores")
    rng = np.random.default_rng(cfg.seed + 100)
    s_gen = synth.random_scores(rng, cfg.rows, tie_frac=0.2, n_levels=64)
    gidx, gvals = hwsel.hwsel_topk_per_problem(torch.from_numpy(s_gen).cuda(), d.seg, cfg.k)
    oidx, ovals = oracle.topk(s_gen, w.seg, cfg.k)
    assert np.array_equal(gidx.cpu().numpy(), oidx)
    assert np.array_equal(gvals.cpu().numpy().view(np.uint32), ovals.view(np.uint32))
    r1, rk, best = hwsel.hwsel_regret(d.runtimes, d.seg, torch.from_numpy(oidx).cuda())
    o1, ok, ob = oracle.regret(w.runtimes, w.seg, oidx)
    assert np.array_equal(r1.cpu().numpy().view(np.uint32), o1.view(np.uint32))
    assert np.array_equal(rk.cpu().numpy().view(np.uint32), ok.view(np.uint32))
    assert np.array_equal(best.cpu().numpy(), ob)
    say(f"  mean regret top1 of generator scores {np.nanmean(o1):.4f}")


def _assert_mlp(g, o):
    rms = float(np.sqrt(np.mean(o.astype(np.float64) ** 2)))
    err = np.abs(g.astype(np.float64) - o)
    bound = 2e-2 * np.maximum(np.abs(o), rms)
    i = int(np.argmax(err / bound))
    assert np.all(err <= bound), f"row {i}: gpu {g[i]} oracle {o[i]} rms {rms}"
    return float((err / bound).max()), rms


def test_mlp_dataset_rows():
    say("mlp: features of the dataset-scale rows")
    w = synth.workload("mlp")
    d = Dev(w)
    X = d.features(128)
    rows = synth.sample_rows(w.cfg, 8192)
    rows_d = torch.from_numpy(rows).cuda()
    say("mlp: matrix-core path on all rows (as benchmarked)")
    packed = hwsel.hwsel_mlp_pack(d.mlp)
    s = hwsel.hwsel_mlp_score(d.mlp, X, packed=packed)
    g = s.index_select(0, rows_d).cpu().numpy()
    Xs = X.index_select(0, rows_d).cpu().numpy()
    o = oracle.mlp(w.mlp, Xs)
    say("  max err/bound %.3g  rms %.3g" % _assert_mlp(g, o))
    assert bool(torch.isfinite(s).all())
    s2 = hwsel.hwsel_mlp_score(d.mlp, X, packed=packed)
    assert bool((s == s2).all())                                    # run-to-run identical
    say("mlp: fp32 row-block path on the sample")
    g2 = hwsel.hwsel_mlp_score(d.mlp, X.index_select(0, rows_d).contiguous()).cpu().numpy()
    say("  max err/bound %.3g  rms %.3g" % _assert_mlp(g2, o))
    # every row: the matrix-core path against the independent fp32 row-block
    # path (itself checked against the oracle above), so that a wrong tile
    # anywhere in the 4.9 M rows is caught, not only in the sample
    say("mlp: matrix-core vs fp32 row-block path on all rows")
    s_ref = hwsel.hwsel_mlp_score(d.mlp, X).double()
    rms = float(torch.sqrt(torch.mean(s_ref ** 2)))
    ratio = torch.abs(s.double() - s_ref) / (2e-2 * torch.clamp(torch.abs(s_ref), min=rms))
    say("  max |diff| / (2e-2 max(|ref|, rms)) %.3g" % float(ratio.max()))
    assert float(ratio.max()) <= 1.0
    # top-k on the MLP scores: admissible picks (oracle score within the tie band of the k-th)
    idx, _ = hwsel.hwsel_topk_per_problem(s, d.seg, w.cfg.k)
    idx = idx.cpu().numpy()
    seg = w.seg
    for p in range(0, w.cfg.n_problems, 75):
        Xp = X[seg[p]:seg[p + 1]].cpu().numpy()
        op = oracle.mlp(w.mlp, Xp)
        kth = np.sort(op)[::-1][w.cfg.k - 1]
        rms_p = float(np.sqrt(np.mean(op.astype(np.float64) ** 2)))
        assert np.all(op[idx[p]] >= kth - 4e-2 * max(abs(kth), rms_p)), p


@pytest.mark.parametrize("R", [1, 127, 129, 1000])
def test_mlp_ragged_and_nonfinite(R):
    say(f"mlp ragged R={R}")
    rng = np.random.default_rng(R)
    m = synth.mlp(synth.CONFIGS["mlp"])
    md = {k: hwsel.to_device(v) for k, v in m.items()}
    sd = np.where(m["inv_std"] > 0, 1.0 / np.where(m["inv_std"] > 0, m["inv_std"], 1.0), 1.0)
    X = (rng.standard_normal((R, 128)) * sd + m["mean"]).astype(np.float32)
    X[rng.random(X.shape) < 0.01] = np.nan
    X[rng.random(X.shape) < 0.01] = np.inf
    X[rng.random(X.shape) < 0.01] = -np.inf
    Xd = torch.from_numpy(X).cuda()
    o = oracle.mlp(m, X)
    g = hwsel.hwsel_mlp_score(md, Xd, packed=hwsel.hwsel_mlp_pack(md)).cpu().numpy()
    _assert_mlp(g, o)
    g2 = hwsel.hwsel_mlp_score(md, Xd).cpu().numpy()
    _assert_mlp(g2, o)


def test_mlp_persistent_tile_walk():
    """513 tiles of 128 rows on at most 256 persistent workgroups: workgroups
    walk 2 or 3 tiles, the last one ragged (77 rows).  Every row against the
    fp32 row-block path, a sample (all of the last two tiles included)
    against the oracle."""
    R = 512 * 128 + 77
    say(f"mlp persistent walk R={R}")
    rng = np.random.default_rng(2609)
    m = synth.mlp(synth.CONFIGS["mlp"])
    md = {k: hwsel.to_device(v) for k, v in m.items()}
    sd = np.where(m["inv_std"] > 0, 1.0 / np.where(m["inv_std"] > 0, m["inv_std"], 1.0), 1.0)
    X = (rng.standard_normal((R, 128)) * sd + m["mean"]).astype(np.float32)
    Xd = torch.from_numpy(X).cuda()
    packed = hwsel.hwsel_mlp_pack(md)
    s = hwsel.hwsel_mlp_score(md, Xd, packed=packed)
    s_ref = hwsel.hwsel_mlp_score(md, Xd).double()
    rms = float(torch.sqrt(torch.mean(s_ref ** 2)))
    ratio = torch.abs(s.double() - s_ref) / (2e-2 * torch.clamp(torch.abs(s_ref), min=rms))
    say("  max |diff| / (2e-2 max(|ref|, rms)) %.3g" % float(ratio.max()))
    assert float(ratio.max()) <= 1.0
    rows = np.unique(np.concatenate([rng.choice(R, 2048, replace=False), np.arange(R - 205, R)]))
    g = s.cpu().numpy()[rows]
    o = oracle.mlp(m, X[rows])
    say("  oracle sample: max err/bound %.3g  rms %.3g" % _assert_mlp(g, o))
    # the output holds exactly R scores: a row past R is never written
    out = torch.full((R + 64,), 12345.0, device="cuda")
    hwsel.hwsel_mlp_score(md, Xd, scores=out[:R], packed=packed)
    assert bool((out[R:] == 12345.0).all())
    assert bool((out[:R] == s).all())


@pytest.mark.parametrize("ld", [136, 256])
def test_mlp_strided_rows(ld):
    """X with a row stride above 128 (a column slice of a wider matrix): both
    kernels give exactly the scores of the contiguous copy."""
    R = 3 * 128 + 5
    say(f"mlp strided ld={ld}")
    rng = np.random.default_rng(ld)
    m = synth.mlp(synth.CONFIGS["mlp"])
    md = {k: hwsel.to_device(v) for k, v in m.items()}
    wide = torch.from_numpy(rng.standard_normal((R, ld)).astype(np.float32)).cuda()
    Xs = wide[:, :128]
    assert Xs.stride(0) == ld
    Xc = Xs.contiguous()
    packed = hwsel.hwsel_mlp_pack(md)
    assert bool((hwsel.hwsel_mlp_score(md, Xs, packed=packed) == hwsel.hwsel_mlp_score(md, Xc, packed=packed)).all())
    assert bool((hwsel.hwsel_mlp_score(md, Xs) == hwsel.hwsel_mlp_score(md, Xc)).all())
    o = oracle.mlp(m, Xc.cpu().numpy())
    _assert_mlp(hwsel.hwsel_mlp_score(md, Xs, packed=packed).cpu().numpy(), o)


# ----------------------------------------------------------------------------
# every packed traversal shape (depth 1..10, chunk widths 64/32/16), padding
# trees, ragged row counts, NaN features with both default directions
# ----------------------------------------------------------------------------
@pytest.mark.parametrize("depth,trees,flags", [(1, 1, 1), (2, 65, 0), (3, 64, 1), (4, 7, 1), (5, 130, 0),
                                               (6, 33, 1), (7, 64, 0), (8, 70, 1), (9, 33, 1), (9, 40, 0),
                                               (10, 17, 1), (10, 20, 0)])
def test_forest_every_depth(depth, trees, flags):
    import dataclasses
    say(f"forest depth {depth} trees {trees} flags {flags}")
    base = synth.CONFIGS["tiny"]
    cfg = dataclasses.replace(base, trees=trees, depth=depth)
    w = synth.workload("tiny", with_model=False)
    f = synth.forest(cfg)
    f["flags"] = flags
    R = 8191
    X = oracle.features(w.hw, w.problems, w.seg, w.cands, 64)[:R].copy()
    rng = np.random.default_rng(depth * 100 + trees)
    X[rng.random(X.shape) < 0.02] = np.nan
    o, oli = oracle.forest(f, X, leaves=True)
    l1 = path_l1(f, oli)
    from _gpu_util import forest_to_device
    fd = forest_to_device(f)
    Xd = torch.from_numpy(X).cuda()
    g = hwsel.hwsel_forest_score(fd, Xd).cpu().numpy()
    e_direct = assert_forest_scores(g, o, l1)
    packed = hwsel.hwsel_forest_pack(fd)
    ws = torch.empty(hwsel.hwsel_forest_workspace_bytes(fd, R), dtype=torch.uint8, device="cuda")
    gp = hwsel.hwsel_forest_score(fd, Xd, packed=packed, workspace=ws).cpu().numpy()
    e_packed = assert_forest_scores(gp, o, l1)
    rows = torch.arange(0, R, 7, dtype=torch.int64, device="cuda")
    li = hwsel.hwsel_forest_leaves(fd, Xd, rows).cpu().numpy().view(np.uint16)
    assert np.array_equal(li, oli[::7])
    say(f"  err/bound direct {e_direct:.3g} packed {e_packed:.3g}")


# ----------------------------------------------------------------------------
# the direct walk beyond the packed limits: depth 11 and 12, more than 128
# features; packing refuses these forests with HWSEL_EUNSUPPORTED
# ----------------------------------------------------------------------------
@pytest.mark.parametrize("depth,trees,n_features", [(11, 9, 64), (12, 5, 64), (6, 40, 200), (12, 3, 256)])
def test_forest_direct_walk_beyond_packed_limits(depth, trees, n_features):
    import dataclasses
    from _gpu_util import forest_to_device
    say(f"direct walk depth {depth} trees {trees} features {n_features}")
    R = 5003
    if n_features == 64:
        cfg = dataclasses.replace(synth.CONFIGS["tiny"], trees=trees, depth=depth)
        w = synth.workload("tiny", with_model=False)
        f = synth.forest(cfg)
        X = oracle.features(w.hw, w.problems, w.seg, w.cands, 64)[:R].copy()
        rng = np.random.default_rng(depth)
    else:
        rng = np.random.default_rng(depth * 1000 + n_features)
        n_int = (1 << depth) - 1
        f = dict(n_trees=trees, depth=depth, n_features=n_features, flags=0, base_score=0.25,
                 node_feature=rng.integers(0, n_features, (trees, n_int)).astype(np.uint8),
                 node_threshold=rng.standard_normal((trees, n_int)).astype(np.float32),
                 leaf_value=rng.normal(0, 0.1, (trees, 1 << depth)).astype(np.float32))
        X = rng.standard_normal((R, n_features)).astype(np.float32)
    X[rng.random(X.shape) < 0.02] = np.nan
    o, oli = oracle.forest(f, X, leaves=True)
    fd = forest_to_device(f)
    Xd = torch.from_numpy(X).cuda()
    g = hwsel.hwsel_forest_score(fd, Xd).cpu().numpy()
    e = assert_forest_scores(g, o, path_l1(f, oli))
    rows = torch.arange(0, R, 3, dtype=torch.int64, device="cuda")
    li = hwsel.hwsel_forest_leaves(fd, Xd, rows).cpu().numpy().view(np.uint16)
    assert np.array_equal(li, oli[::3])
    with pytest.raises(hwsel.HwselError) as err:
        hwsel.hwsel_forest_pack(fd)
    assert err.value.status == hwsel.HWSEL_EUNSUPPORTED
    say(f"  err/bound {e:.3g}; leaf indices equal on {len(rows)} rows; packing refused")


@pytest.mark.parametrize("name", ["tiny", "dataset"])
def test_forest_pack_host_equals_device_pack(name):
    """hwsel_forest_pack (device arrays) and hwsel_forest_pack_host (host
    arrays, no GPU) write the same image, byte for byte."""
    from _gpu_util import forest_to_device
    f = synth.forest(synth.CONFIGS[name])
    dev_img = hwsel.hwsel_forest_pack(forest_to_device(f)).cpu().numpy()
    host_img = hwsel.hwsel_forest_pack_host(f)
    assert np.array_equal(dev_img, host_img)
