"""Pins of the oracle's feature map against the paper's definitions.

Each check derives the expected value by a route other than the oracle's own
formula: enumerating output tiles, K-steps and per-tile operand loads;
counting resident blocks upward until a resource runs out; simulating wave
and cluster-wave scheduling; the worked example of the printed kernel; the
paper's own identities between features (T_K cancels in I_mainloop,
r_pc = t_consumer / t_producer, streamK_applicability = max(0, 1 - eta_last),
S * f_smem); and invariants (eta in (0, 1], r_stream >= 1, ...).
"""
import math
import os

import numpy as np
import pytest

import oracle
import synth

HW = synth.hardware()
GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def feat(M, N, K, layout=0, dtype=0, tile_m=128, tile_n=128, tile_k=64, stages=4, cluster_m=1,
         cluster_n=1, swizzle=1, inst_n=None, inst_m_div16=4, inst_k=None, kernel_sched=0,
         epi_sched=1, tile_sched=0, F=128, hw=HW):
    probs = np.zeros(1, synth.PROBLEM_DTYPE)
    probs["M"], probs["N"], probs["K"], probs["layout"], probs["dtype"] = M, N, K, layout, dtype
    vals = dict(tile_m=tile_m, tile_n=tile_n, tile_k=tile_k, stages=stages, cluster_m=cluster_m,
                cluster_n=cluster_n, swizzle=swizzle, inst_n=tile_n if inst_n is None else inst_n,
                inst_m_div16=inst_m_div16,
                inst_k=(32 if dtype == 2 else 16) if inst_k is None else inst_k,
                kernel_sched=kernel_sched, epi_sched=epi_sched, tile_sched=tile_sched)
    cands = {f: np.array([vals[f]], dt) for f, dt in synth.CAND_FIELDS}
    return oracle.features(hw, probs, np.array([0, 1], np.int64), cands, F)[0]


def f32(x):
    return float(np.float32(x))


# ----------------------------------------------------------------------------
# Worked example (printed kernel) and printed constants
# ----------------------------------------------------------------------------
def test_generated_kernel_worked_example():
    lines = [l.split("#")[0].split() for l in open(os.path.join(GOLDEN, "generated_kernel.txt"))]
    lines = [l for l in lines if l]
    M, N, K, lay, dt = map(int, next(l for l in lines if l[0] == "problem")[1:])
    tm, tn, tk, st, cm, cn, ks, es, ts = map(int, next(l for l in lines if l[0] == "candidate")[1:])
    x = feat(M, N, K, lay, dt, tm, tn, tk, st, cm, cn, kernel_sched=ks, epi_sched=es, tile_sched=ts)
    for l in lines:
        if l[0] == "col":
            assert x[int(l[1])] == np.float32(float(l[3])), l
    # the printed ridge point ~247.3 flop/B
    assert abs(x[80] - 247.3) < 0.1


# ----------------------------------------------------------------------------
# Enumeration / simulation pins on random configurations
# ----------------------------------------------------------------------------
def _random_cases(n, seed=7):
    rng = np.random.default_rng(seed)
    for _ in range(n):
        d = dict(M=int(rng.integers(1, 3000)), N=int(rng.integers(1, 3000)), K=int(rng.integers(1, 5000)),
                 layout=int(rng.integers(0, 4)), dtype=int(rng.integers(0, 3)),
                 tile_m=int(rng.choice([64, 128, 192, 256])),
                 tile_n=int(rng.choice([16, 32, 48, 64, 80, 96, 128, 192, 256])),
                 tile_k=int(rng.choice([32, 64, 128, 256, 512])), stages=int(rng.integers(2, 13)),
                 kernel_sched=int(rng.integers(0, 3)), epi_sched=int(rng.integers(0, 3)),
                 tile_sched=int(rng.integers(0, 2)), swizzle=int(rng.choice([1, 2, 4, 8])))
        d["cluster_m"], d["cluster_n"] = synth.CLUSTER_PAIRS[int(rng.integers(0, 15))]
        d["inst_n"] = int(rng.choice([d["tile_n"], d["tile_n"] // 2]))
        yield d


def _count_up(fits):
    b = 0
    while fits(b + 1):
        b += 1
    return b


def _simulate_passes(work, slots):
    passes, left = 0, work
    while left > 0:
        left -= slots
        passes += 1
    return passes


@pytest.mark.parametrize("case", list(_random_cases(150)))
def test_columns_by_enumeration(case):
    c = case
    x = feat(**c)
    M, N, K = c["M"], c["N"], c["K"]
    TM, TN, TK, S = c["tile_m"], c["tile_n"], c["tile_k"], c["stages"]
    CM, CN = c["cluster_m"], c["cluster_n"]
    b = 1 if c["dtype"] == 2 else 2
    # output tiles and K-steps, by walking the tile origins
    row_tiles = [min(TM, M - i) for i in range(0, M, TM)]
    col_tiles = [min(TN, N - j) for j in range(0, N, TN)]
    ksteps = list(range(0, K, TK))
    assert x[12] == len(row_tiles) and x[13] == len(col_tiles) and x[14] == len(ksteps)
    tiles = len(row_tiles) * len(col_tiles)
    assert x[15] == tiles
    # edge waste: masked rows / columns of the padded grid
    assert x[16] == f32(sum(TM - r for r in row_tiles) / M)
    assert x[17] == f32(sum(TN - q for q in col_tiles) / N)
    assert x[18] == f32(sum(TK - min(TK, K - k) for k in ksteps) / K)
    assert x[19] == f32(tiles / HW["n_sm"])
    # per-stage buffers: one T_M x T_K slice of A and one T_K x T_N slice of B
    assert x[24] == TM * TK * b + TK * TN * b
    assert x[25] == S * x[24]
    # resident blocks: count up until a resource runs out
    T_block = x[20]
    assert T_block == (256 if c["kernel_sched"] == 0 else 384)
    B_smem = int(x[27])
    assert x[29] == _count_up(lambda k: k * B_smem <= HW["smem_per_sm"])
    regs = int(x[22])
    assert x[23] == _count_up(lambda k: k * regs * T_block <= HW["regs_per_sm"])
    assert x[30] == _count_up(lambda k: k <= HW["max_blocks_per_sm"] and k * T_block <= HW["max_threads_per_sm"])
    assert x[31] == min(x[29], x[23], x[30])
    assert x[31] <= x[29] and x[31] <= x[23] and x[31] <= x[30]
    # wave quantisation, simulated pass by pass over the resident slots
    slots = HW["n_sm"] * max(int(x[31]), 1)
    q = _simulate_passes(tiles, slots)
    assert x[33] == q
    assert x[34] == f32(tiles / (q * slots)) and 0 < x[34] <= 1
    # streamK_applicability = max(0, 1 - eta_last)
    assert abs(x[35] - max(0.0, 1.0 - x[34])) <= 1e-6
    assert (x[35] == 0) == (tiles % slots == 0)
    # clusters: walk the cluster grid, then pass by pass over cluster slots
    n_c = len(range(0, M, CM * TM)) * len(range(0, N, CN * TN))
    assert x[36] == n_c
    slots_c = max(1, HW["n_sm"] // (CM * CN))
    assert x[37] == slots_c
    W = _simulate_passes(n_c, slots_c)
    assert x[38] == W and x[39] == f32(n_c / (W * slots_c))
    assert x[42] == (CM > len(row_tiles) or CN > len(col_tiles))
    # operand traffic: sum of the A and B panels every output tile loads
    loads = sum(r * K * b + q_ * K * b for r in row_tiles for q_ in col_tiles)
    unique = M * K * b + K * N * b
    assert x[48] == np.float32(loads)
    assert x[45] == f32(loads / unique) and x[45] >= 1
    assert (x[45] == 1) == (tiles == 1)
    assert x[49] == 4 * M * N
    flops = 2 * M * N * K
    assert x[43] == f32(flops / (unique + 4 * M * N))
    # T_K cancels in I_mainloop: tile flops over tile operand bytes
    assert x[44] == f32((2 * TM * TN * TK) / (TM * TK * b + TN * TK * b))
    # pipeline balance: r_pc = t_consumer / t_producer
    assert abs(x[52] - x[51] / x[50]) <= 4e-7 * x[52]
    assert x[53] == f32(min(S, len(ksteps)) / S) and (x[53] == 1) == (len(ksteps) >= S)
    assert x[54] == f32(len(ksteps) / S)
    assert abs(x[55] - S * x[28]) <= 4e-7 * x[55]
    # sampling score = cluster-wave fill / (c_M c_N) * S * sqrt(T_M T_N T_K)
    assert abs(x[58] - x[39] / (CM * CN) * S * math.sqrt(TM * TN * TK)) <= 1e-6 * x[58]
    # log-scale columns
    for col, v in ((0, M), (1, N), (2, K), (3, flops), (127, tiles)):
        assert abs(2.0 ** float(x[col]) - v) <= 2e-6 * v * 30
    # padded work over useful work, by enumeration
    padded = sum(TM * TN for _ in row_tiles for _ in col_tiles) * len(ksteps) * TK
    assert x[92] == f32(padded / (M * N * K))
    # instruction count per K block by stepping the instruction tile
    IM, IN, IK = 64, c["inst_n"], (32 if b == 1 else 16)
    steps = len(range(0, TM, IM)) * len(range(0, TN, IN)) * len(range(0, TK, IK))
    assert x[99] == steps and x[100] == steps * len(ksteps)
    edge = sum(1 for r in row_tiles for q_ in col_tiles if r < TM or q_ < TN)
    assert x[125] == edge and x[126] == f32(edge / tiles)
    assert x[109] == min(S, len(ksteps)) and x[110] == max(0, len(ksteps) - S)
    # stage time = max(t_producer, t_consumer); mainloop = x n_K; wave = x q
    assert abs(x[111] - max(x[50], x[51])) <= 1e-7 * x[111]
    assert abs(x[112] - x[111] * len(ksteps)) <= 1e-6 * x[112]
    assert abs(x[113] - x[112] * q) <= 1e-6 * x[113]


def test_layout_decoding():
    # TN: A row-major, B column-major (the printed kernel's convention)
    want = {0: (0, 0), 1: (0, 1), 2: (1, 0), 3: (1, 1)}
    for lay, (a_col, b_row) in want.items():
        x = feat(512, 512, 512, layout=lay)
        assert (x[64], x[65], x[66]) == (lay, a_col, b_row)


def test_validity_predicates():
    base = dict(M=1024, N=1024, K=1024)
    # Stream-K needs the cooperative mainloop
    x = feat(**base, kernel_sched=0, tile_sched=1)
    assert x[85] == 0 and x[87] == 0
    x = feat(**base, tile_m=128, kernel_sched=2, epi_sched=2, tile_sched=1)
    assert x[85] == 1 and x[84] == 1 and x[87] == 1
    # cooperative needs T_M % 128 == 0
    x = feat(**base, tile_m=192, kernel_sched=2, epi_sched=2)
    assert x[84] == 0 and x[87] == 0
    # shared-memory capacity per block: 227 KiB including a 2 KiB reserve
    x = feat(**base, tile_m=256, tile_n=256, tile_k=128, stages=4)
    assert x[32] == 0 and x[87] == 0
    # K-box limits of transposed operands
    x = feat(**base, layout=2, tile_k=512, cluster_n=1, stages=1, tile_m=64, tile_n=16)
    assert x[82] == 0
    x = feat(**base, layout=2, tile_k=512, cluster_n=2, stages=1, tile_m=64, tile_n=16)
    assert x[82] == 1
    x = feat(**base, layout=1, tile_k=512, cluster_m=1, stages=1, tile_m=64, tile_n=16)
    assert x[83] == 0
    # the T_N guard is a feature only
    x = feat(M=8, N=1024, K=64, tile_n=32)
    assert x[86] == 0


def test_valid_count_on_full_grid_matches_catalogue_filter():
    """Two independent statements of the static legality rules -- the
    generator's catalogue filter and the oracle's validity column -- agree on
    every point of the 65,536-point grid, for each layout."""
    g = synth.full_grid()
    n = len(g["tile_m"])
    for lay in range(4):
        probs = np.zeros(1, synth.PROBLEM_DTYPE)
        probs["M"] = probs["N"] = probs["K"] = 4096
        probs["layout"] = lay
        cands = {f: np.zeros(n, dt) for f, dt in synth.CAND_FIELDS}
        for f in g:
            cands[f][:] = g[f]
        cands["swizzle"][:] = 1
        cands["inst_m_div16"][:] = 4
        cands["inst_k"][:] = 16
        X = oracle.features(HW, probs, np.array([0, n], np.int64), cands, 96)
        mask = synth.catalogue_mask(g, lay, 0)
        assert np.array_equal(X[:, 87] == 1, mask)
        assert mask.sum() == 16328


def test_ridge_and_hardware_columns():
    x = feat(4096, 4096, 4096)
    assert x[80] == np.float32(247.375)
    assert tuple(x[59:64]) == (132, 233472, 65536, 52428800, 4000)
    x8 = feat(4096, 4096, 4096, dtype=2)
    assert x8[79] == 1979000 and x8[70] == 1 and x8[88] == 4096 * 4096 * 2
    assert x8[89] == x8[48] + x8[49] + x8[88]


def test_degenerate_inputs_give_finite_features():
    # M, N, K below 1 are read as 1; zero knobs as 1; a block that cannot be
    # resident (b_res = 0) still yields finite wave features
    x = feat(0, 0, 0, tile_m=0, tile_n=0, tile_k=0, stages=0, cluster_m=0, cluster_n=0,
             inst_n=0, inst_m_div16=0, inst_k=0)
    assert np.all(np.isfinite(x))
    big = feat(64, 64, 64, tile_m=256, tile_n=256, tile_k=512, stages=12)
    assert big[31] == 0 and np.all(np.isfinite(big))


def test_feature_tiers_are_prefixes():
    full = feat(1000, 2000, 3000, F=128)
    for F in (64, 96):
        assert np.array_equal(feat(1000, 2000, 3000, F=F), full[:F])


# ----------------------------------------------------------------------------
# Hand-derived values of the columns no enumeration or identity above reaches
# ----------------------------------------------------------------------------
def _hand_cases():
    cases, order = {}, []
    for raw in open(os.path.join(GOLDEN, "hand_features.txt")):
        line = raw.split("#")[0].split()
        if not line:
            continue
        if line[0] == "case":
            name = line[1]
            M, N, K, lay, dt = map(int, line[2:7])
            assert line[7] == "|"
            tm, tn, tk, st, cm, cn, swz, im, in_, ik, ks, es, ts = map(int, line[8:21])
            cases[name] = dict(args=dict(M=M, N=N, K=K, layout=lay, dtype=dt, tile_m=tm, tile_n=tn, tile_k=tk,
                                         stages=st, cluster_m=cm, cluster_n=cn, swizzle=swz, inst_m_div16=im // 16,
                                         inst_n=in_, inst_k=ik, kernel_sched=ks, epi_sched=es, tile_sched=ts),
                               cols=[])
            order.append(name)
        else:
            cases[line[0]]["cols"].append((int(line[1]), line[2:]))
    return [(n, cases[n]) for n in order]


@pytest.mark.parametrize("name,case", _hand_cases(), ids=[n for n, _ in _hand_cases()])
def test_hand_derived_columns(name, case):
    """Columns 21, 26-28, 40-41, 46-47, 50-51, 55, 81, 90-91, 101-124 against
    values worked out by hand from the paper's definitions
    (tests/golden/hand_features.txt): an exact ratio must match bit for bit
    (one binary64 division rounded to fp32), a short binary64 sequence within
    1e-6 relative."""
    x = feat(**case["args"])
    assert len(case["cols"]) >= 30
    for col, spec in case["cols"]:
        if spec[0] == "sqrt":
            want = np.float32(math.sqrt(int(spec[1])))
            assert x[col] == want, (name, col, x[col], want)
        elif spec[0] == "q":
            num, den = map(int, spec[1].split("/"))
            want = num / den
            assert abs(float(x[col]) - want) <= 1e-6 * abs(want), (name, col, x[col], want)
        else:
            num, den = map(int, spec[0].split("/"))
            want = np.float32(float(num) / float(den))
            assert x[col] == want, (name, col, x[col], want)
