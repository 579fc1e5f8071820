"""Pins of the oracle's tree-ensemble scorer (additive ensemble of regression
trees, section "Model A").  Hand-built forests with known outputs, the closed
form of the leaf index (the path's right turns read as a binary number), an
independent pointer-chasing walk, and invariance of the sum under tree order."""
import numpy as np

import oracle


def forest(feat, thr, leaves, depth, flags=1, base=0.0, n_features=4):
    feat = np.asarray(feat, np.uint8).reshape(-1, (1 << depth) - 1)
    return dict(n_trees=feat.shape[0], depth=depth, n_features=n_features, flags=flags,
                base_score=base, node_feature=feat,
                node_threshold=np.asarray(thr, np.float32).reshape(feat.shape),
                leaf_value=np.asarray(leaves, np.float32).reshape(feat.shape[0], 1 << depth))


def test_one_stump():
    f = forest([0], [0.5], [-1.0, 1.0], depth=1)
    X = np.array([[0.49, 0, 0, 0], [0.5, 0, 0, 0], [0.51, 0, 0, 0], [np.nan, 0, 0, 0],
                  [-np.inf, 0, 0, 0], [np.inf, 0, 0, 0]], np.float32)
    s, li = oracle.forest(f, X, leaves=True)
    # below goes left; a tie goes right; NaN follows the default (left)
    assert s.tolist() == [-1.0, 1.0, 1.0, -1.0, -1.0, 1.0]
    assert li[:, 0].tolist() == [0, 1, 1, 0, 0, 1]
    f_right = forest([0], [0.5], [-1.0, 1.0], depth=1, flags=0)
    assert oracle.forest(f_right, X[3:4])[0] == 1.0


def test_two_trees_depth_two_hand_sum():
    # tree 0: root x0<1 ; left x1<2 ; right x2<3 ; leaves 1,2,3,4
    # tree 1: root x3<0 ; left x0<0 ; right x1<0 ; leaves 10,20,30,40
    f = forest([0, 1, 2, 3, 0, 1], [1, 2, 3, 0, 0, 0], [1, 2, 3, 4, 10, 20, 30, 40], depth=2, base=0.5)
    X = np.array([[0, 0, 0, 0],      # t0: L,L ->1 ; t1: x3=0 not<0 -> R, x1=0 not<0 -> R ->40
                  [5, 5, 0, -1],     # t0: R, x2=0<3 L ->3 ; t1: L, x0=5 R ->20
                  [0, 9, 9, 1]],     # t0: L, x1=9 R ->2 ; t1: R, x1=9 R ->40
                 np.float32)
    s, li = oracle.forest(f, X, leaves=True)
    assert s.tolist() == [0.5 + 1 + 40, 0.5 + 3 + 20, 0.5 + 2 + 40]
    assert li.tolist() == [[0, 3], [2, 1], [1, 3]]


def test_leaf_index_is_path_bits_and_linked_walk_agrees():
    rng = np.random.default_rng(3)
    for depth in (1, 3, 6, 8):
        T, F = 7, 9
        n_int = (1 << depth) - 1
        feat = rng.integers(0, F, (T, n_int))
        thr = rng.standard_normal((T, n_int)).astype(np.float32)
        leaves = rng.standard_normal((T, 1 << depth)).astype(np.float32)
        f = forest(feat, thr, leaves, depth, n_features=F)
        X = rng.standard_normal((300, F)).astype(np.float32)
        X[rng.random(X.shape) < 0.05] = np.nan
        s, li = oracle.forest(f, X, leaves=True)
        # closed form: leaf = sum over levels of (went right) * 2^(depth-1-level)
        for r in range(0, 300, 37):
            for t in range(T):
                node, bits = 0, 0
                for lev in range(depth):
                    v = X[r, feat[t, node]]
                    right = not (v < thr[t, node] or np.isnan(v))
                    bits = 2 * bits + right
                    node = 2 * node + 1 + right
                assert li[r, t] == bits
        assert np.array_equal(oracle.forest_linked(f, X), s)


def test_tree_order_changes_sum_only_by_rounding():
    rng = np.random.default_rng(5)
    depth, T, F = 5, 40, 6
    n_int = (1 << depth) - 1
    feat = rng.integers(0, F, (T, n_int))
    thr = rng.standard_normal((T, n_int)).astype(np.float32)
    leaves = rng.normal(0, 0.1, (T, 1 << depth)).astype(np.float32)
    X = rng.standard_normal((200, F)).astype(np.float32)
    a = oracle.forest(forest(feat, thr, leaves, depth, n_features=F), X)
    perm = rng.permutation(T)
    b = oracle.forest(forest(feat[perm], thr[perm], leaves[perm], depth, n_features=F), X)
    assert np.allclose(a, b, rtol=0, atol=1e-6)


def test_row_subset_matches_full():
    rng = np.random.default_rng(9)
    f = forest(rng.integers(0, 4, (3, 7)), rng.standard_normal(21), rng.standard_normal(24), depth=3)
    X = rng.standard_normal((50, 4)).astype(np.float32)
    rows = np.array([49, 3, 17, 17], np.int64)
    assert np.array_equal(oracle.forest(f, X, rows=rows), oracle.forest(f, X)[rows])


def test_leaf_mix_is_splitmix64_finaliser():
    # SplitMix64 seeded with 0 returns mix(g), mix(2g), ... with the golden
    # gamma g = 0x9E3779B97F4A7C15; its first two published outputs
    g = 0x9E3779B97F4A7C15
    assert oracle.leaf_mix(g) == 0xE220A8397B1DCDAF
    assert oracle.leaf_mix(2 * g) == 0x6E789E6AA1B965F4
    assert oracle.leaf_mix(0) == 0


def test_leaf_hash_is_sum_of_mixed_tree_leaf_pairs():
    rng = np.random.default_rng(21)
    depth, T, F = 4, 9, 5
    n_int = (1 << depth) - 1
    f = forest(rng.integers(0, F, (T, n_int)), rng.standard_normal(T * n_int), rng.standard_normal(T << depth),
               depth, n_features=F)
    X = rng.standard_normal((40, F)).astype(np.float32)
    s, li, h = oracle.forest(f, X, leaves=True, leaf_hash=True)
    assert np.array_equal(s, oracle.forest(f, X))
    for r in range(40):
        want = sum(oracle.leaf_mix((t << 32) | int(li[r, t])) for t in range(T)) % (1 << 64)
        assert int(h[r]) == want
    # one changed leaf changes the fingerprint; the tree order does not matter
    # for it, only which leaf each tree reaches
    alt = (int(h[0]) - oracle.leaf_mix((3 << 32) | int(li[0, 3]))
           + oracle.leaf_mix((3 << 32) | (int(li[0, 3]) ^ 1))) % (1 << 64)
    assert alt != int(h[0])
    # the same leaf reached in another tree is another term: the fingerprint
    # tells which tree reached which leaf
    assert oracle.leaf_mix((3 << 32) | 5) != oracle.leaf_mix((4 << 32) | 5)
