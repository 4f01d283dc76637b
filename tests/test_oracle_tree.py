"""Oracle pins for Alg. 1 (BuildHistograms, EvaluateSplit with Eq. 8,
RepartitionInstances), Eq. 6 leaves and Eq. 1 prediction.  CPU only."""
from fractions import Fraction
import json
import os

import numpy as np
import pytest

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_eq8_worked_example(orc):
    g = json.load(open(os.path.join(GOLDEN, "eq8_worked_example.json")))
    gp = np.stack([g["g"], g["h"]], 1)
    q, eg, eh = orc.fixed_point(gp)
    nb = np.array([4], np.int32)
    hist = np.zeros((4, 2), np.int64)
    for b, row in zip(g["bins"], q):
        hist[b] += row
    P = orc.Params(lambda_=g["lambda"], gamma=g["gamma"], eta=g["eta"],
                   min_child_weight=g["min_child_weight"])
    s = orc.eval_node(hist, q.sum(0), nb, P, eg, eh)
    assert s.valid and s.feature == 0 and s.split_bin == g["best_split_bin"]
    assert s.gain == g["best_gain"] and s.default_left == 0
    # every candidate's gain, by forcing the others out via a single-cut histogram
    for sb, want in g["gains_by_s"].items():
        sb = int(sb)
        h2 = np.array([hist[:sb].sum(0), hist[sb:].sum(0)])
        s2 = orc.eval_node(h2, q.sum(0), np.array([2], np.int32), P, eg, eh)
        assert s2.gain == want
    lv = orc.leaf_value(s.left_g, s.left_h, eg, eh, g["lambda"], g["eta"])
    rv = orc.leaf_value(s.right_g, s.right_h, eg, eh, g["lambda"], g["eta"])
    assert lv == np.float32(g["left_leaf"]) and rv == np.float32(g["right_leaf"])


def _small_data(orc, seed, n, m, missing=0.2, B=256):
    rng = np.random.default_rng(seed)
    X = rng.normal(size=(n, m)).astype(np.float32)
    X[rng.random(X.shape) < missing] = np.nan
    cuts = orc.sketch_cuts_dense(X, B)
    return X, orc.bin_dense(X, cuts), rng


def test_histogram_equals_add_at(orc):
    X, b, rng = _small_data(orc, 1, 500, 7)
    q = rng.integers(-2**40, 2**40, size=(500, 2)).astype(np.int64)
    rows = np.sort(rng.choice(500, 200, replace=False))
    hist = orc.build_hist(b, rows, q)
    off = np.concatenate([[0], np.cumsum(b.cuts.nbins)])
    ref = np.zeros_like(hist)
    for j in range(7):
        ok = b.dense[rows, j] != orc.MISSING
        np.add.at(ref, off[j] + b.dense[rows[ok], j].astype(np.int64), q[rows[ok]])
    assert np.array_equal(hist, ref)
    # per feature: sum over bins + missing rows = node sum
    tot = q[rows].sum(0)
    for j in range(7):
        miss = q[rows[b.dense[rows, j] == orc.MISSING]].sum(0)
        assert np.array_equal(hist[off[j]:off[j + 1]].sum(0) + miss, tot)


def test_left_plus_right_is_parent(orc):
    X, b, rng = _small_data(orc, 2, 800, 5)
    q = rng.integers(-2**30, 2**30, size=(800, 2)).astype(np.int64)
    rows = np.arange(800)
    left, right = orc.partition(b, rows, 3, 100, True)
    assert len(left) + len(right) == 800
    assert np.array_equal(orc.build_hist(b, left, q) + orc.build_hist(b, right, q),
                          orc.build_hist(b, rows, q))


def test_partition_agrees_with_raw_threshold_and_is_stable(orc):
    X, b, rng = _small_data(orc, 3, 1000, 4)
    rows = np.sort(rng.choice(1000, 600, replace=False))
    for j, s, dl in [(0, 10, False), (2, 128, True), (3, 1, True)]:
        t = b.cuts.cut_values[b.cuts.cut_ptr[j] + s - 1]
        left, right = orc.partition(b, rows, j, s, dl)
        x = X[rows, j]
        goes_left = np.where(np.isnan(x), dl, x <= t)
        assert np.array_equal(left, rows[goes_left])
        assert np.array_equal(right, rows[~goes_left])


def _exact_gain(GL, HL, GR, HR, G, H, lam, gam):
    return Fraction(1, 2) * (GL * GL / (HL + lam) + GR * GR / (HR + lam) - G * G / (H + lam)) - gam


def brute_tree(X, q, eg, eh, cutvals, D, lam, gam, mcw):
    """Greedy tree by exhaustive enumeration of raw-value partitions with
    exact rational gains.  Returns {heap id: record}."""
    lam, gam, mcw = Fraction(lam), Fraction(gam), Fraction(mcw)
    sg = 2 ** eg
    sh = 2 ** eh
    out = {}

    def grow(node, rows, depth):
        Qg = sum(int(q[r, 0]) for r in rows)
        Qh = sum(int(q[r, 1]) for r in rows)
        rec = {"rows": len(rows), "sum": (Qg, Qh)}
        out[node] = rec
        if depth >= D:
            return
        G, H = Fraction(Qg, sg), Fraction(Qh, sh)
        best = None
        for j in range(X.shape[1]):
            for s, t in enumerate(cutvals[j], start=1):
                for dl in (False, True):
                    left = [r for r in rows if (dl if np.isnan(X[r, j]) else X[r, j] <= t)]
                    lset = set(left)
                    right = [r for r in rows if r not in lset]
                    QLg = sum(int(q[r, 0]) for r in left)
                    QLh = sum(int(q[r, 1]) for r in left)
                    HL, HR = Fraction(QLh, sh), Fraction(Qh - QLh, sh)
                    if HL < mcw or HR < mcw:
                        continue
                    gain = _exact_gain(Fraction(QLg, sg), HL, Fraction(Qg - QLg, sg), HR, G, H,
                                       lam, gam)
                    if best is None or gain > best[0]:
                        best = (gain, j, s, dl, left, right)
        if best is not None and best[0] > 0:
            rec.update(gain=best[0], feature=best[1], split_bin=best[2], default_left=best[3])
            grow(2 * node + 1, best[4], depth + 1)
            grow(2 * node + 2, best[5], depth + 1)

    grow(0, list(range(X.shape[0])), 0)
    return out


@pytest.mark.parametrize("seed", range(6))
def test_tree_matches_exhaustive_search_tiny(orc, seed):
    rng = np.random.default_rng(100 + seed)
    n, m, D = int(rng.integers(5, 13)), 3, 3
    X = rng.normal(size=(n, m)).astype(np.float32)
    X[rng.random(X.shape) < 0.25] = np.nan
    y = (rng.random(n) < 0.5).astype(np.float32)
    cuts = orc.sketch_cuts_dense(X, 256)
    b = orc.bin_dense(X, cuts)
    # with n < max_bin every distinct value but the largest is a cut
    cutvals = []
    for j in range(m):
        u = np.unique(X[~np.isnan(X[:, j]), j])
        cutvals.append(u[:-1])
        assert np.array_equal(u[:-1], cuts.cut_values[cuts.cut_ptr[j]:cuts.cut_ptr[j + 1]])
    lam, gam, mcw = 1.0, 0.0, 0.05
    P = orc.Params(loss=orc.LOSS_LOGISTIC, max_depth=D, eta=0.3, lambda_=lam, gamma=gam,
                   min_child_weight=mcw)
    margin = (rng.normal(size=n) * 0.5).astype(np.float32)
    m0 = margin.copy()
    res = orc.train_tree(b, y, margin, P, want_detail=True)
    q = res.q
    ref = brute_tree(X, q, res.info.e_g, res.info.e_h, cutvals, D, lam, gam, mcw)
    nodes = res.nodes
    present = {i for i in range(len(nodes)) if nodes[i]["flags"] & orc.NODE_PRESENT}
    assert present == set(ref)
    for i, rec in ref.items():
        nd = nodes[i]
        assert nd["n_rows"] == rec["rows"]
        assert (int(nd["sum_g"]), int(nd["sum_h"])) == rec["sum"]
        if "feature" in rec:
            assert not nd["flags"] & orc.NODE_LEAF
            assert (nd["feature"], nd["split_bin"]) == (rec["feature"], rec["split_bin"])
            assert bool(nd["flags"] & orc.NODE_DEFAULT_LEFT) == rec["default_left"]
            assert abs(nd["gain"] - float(rec["gain"])) <= 1e-12 * max(1.0, abs(float(rec["gain"])))
        else:
            assert nd["flags"] & orc.NODE_LEAF
            G = Fraction(rec["sum"][0], 2 ** res.info.e_g)
            H = Fraction(rec["sum"][1], 2 ** res.info.e_h)
            want = np.float32(float(-G / (H + Fraction(lam)) * Fraction(0.3)))
            assert abs(int(np.float32(nd["leaf_value"]).view(np.int32)) - int(want.view(np.int32))) <= 1
    # margins moved by the reached leaf
    assert np.array_equal(margin, m0 + orc.predict_binned(b, [res.nodes], 0.0))


def test_squared_error_special_case_is_cart(orc):
    """Squared error, lambda=0, gamma=0, eta=1, no sampling, no missing
    values: the greedy tree is a CART regression tree on the bin indices."""
    from sklearn.tree import DecisionTreeRegressor
    rng = np.random.default_rng(7)
    n, m, D = 400, 5, 4
    X = rng.normal(size=(n, m)).astype(np.float32)
    y = (X[:, 0] > 0.3).astype(np.float32) * 2 + X[:, 1] * X[:, 2] + \
        rng.normal(size=n).astype(np.float32) * 0.1
    y = y.astype(np.float32)
    cuts = orc.sketch_cuts_dense(X, 16)
    b = orc.bin_dense(X, cuts)
    P = orc.Params(loss=orc.LOSS_SQUARED, max_depth=D, eta=1.0, lambda_=0.0, gamma=0.0,
                   min_child_weight=1.0)
    margin = np.zeros(n, np.float32)
    res = orc.train_tree(b, y, margin, P)
    sk = DecisionTreeRegressor(max_depth=D, random_state=0).fit(b.dense.astype(np.float32),
                                                                y.astype(np.float64))
    # root split: sklearn threshold k + 0.5 on bin indices <=> split_bin k + 1
    root = res.nodes[0]
    assert root["feature"] == sk.tree_.feature[0]
    assert root["split_bin"] == int(np.floor(sk.tree_.threshold[0])) + 1
    np.testing.assert_allclose(margin, sk.predict(b.dense.astype(np.float32)), rtol=0, atol=2e-6)
    assert len(np.unique(margin)) == sk.get_n_leaves()


def test_depth_zero_tree_is_closed_form_leaf(orc):
    rng = np.random.default_rng(9)
    X = rng.normal(size=(300, 3)).astype(np.float32)
    y = (rng.random(300) < 0.3).astype(np.float32)
    b = orc.bin_dense(X, orc.sketch_cuts_dense(X, 32))
    margin = np.zeros(300, np.float32)
    P = orc.Params(max_depth=0, eta=0.3, lambda_=1.0)
    res = orc.train_tree(b, y, margin, P)
    g = 0.5 - y.astype(np.float64)
    want = np.float32(-0.3 * g.sum() / (0.25 * 300 + 1.0))
    assert abs(int(np.float32(res.nodes[0]["leaf_value"]).view(np.int32)) - int(want.view(np.int32))) <= 1
    assert (margin == res.nodes[0]["leaf_value"]).all()


def test_predict_raw_equals_binned_and_margin_trajectory(orc):
    X, b, rng = _small_data(orc, 4, 3000, 6, missing=0.15, B=64)
    y = (rng.random(3000) < 0.5).astype(np.float32)
    P = orc.Params(max_depth=4, eta=0.3)
    trees, margin = orc.train(b, y, P, 4, 0.0)
    assert np.array_equal(orc.predict_binned(b, trees, 0.0), margin)
    assert np.array_equal(orc.predict_raw_dense(X, trees, 0.0), margin)


def test_predict_raw_csr(orc):
    rng = np.random.default_rng(5)
    n, m = 1500, 30
    X = rng.lognormal(size=(n, m)).astype(np.float32)
    X[rng.random(X.shape) < 0.85] = np.nan
    rows, cols = np.nonzero(~np.isnan(X))
    indptr = np.concatenate([[0], np.cumsum(np.bincount(rows, minlength=n))])
    vals = X[rows, cols]
    cuts = orc.sketch_cuts_csr(indptr, cols, vals, m, 64)
    b = orc.bin_csr(indptr, cols, vals, m, cuts)
    y = (rng.random(n) < 0.5).astype(np.float32)
    P = orc.Params(max_depth=5, eta=0.3, gamma=0.1)
    trees, margin = orc.train(b, y, P, 3, 0.0)
    assert np.array_equal(orc.predict_raw_csr(indptr, cols, vals, trees, 0.0), margin)
    # the same matrix given densely (absent = NaN) trains the same trees
    bd = orc.bin_dense(X, orc.sketch_cuts_dense(X, 64))
    trees2, margin2 = orc.train(bd, y, P, 3, 0.0)
    assert np.array_equal(margin, margin2)
    for t1, t2 in zip(trees, trees2):
        assert np.array_equal(t1.nodes, t2.nodes)


def test_training_loss_decreases_without_sampling(orc):
    X, b, rng = _small_data(orc, 6, 2000, 8, missing=0.0)
    y = (X[:, 0] + X[:, 1] * X[:, 2] > 0).astype(np.float32)
    P = orc.Params(max_depth=3, eta=0.3)
    margin = np.zeros(2000, np.float32)
    losses = []
    for t in range(6):
        orc.train_tree(b, y, margin, P, iteration=t)
        p = 1 / (1 + np.exp(-margin.astype(np.float64)))
        losses.append(-np.mean(y * np.log(p) + (1 - y) * np.log(1 - p)))
    assert all(b2 < a for a, b2 in zip(losses, losses[1:]))


def test_sampled_tree_uses_only_sampled_rows(orc):
    X, b, rng = _small_data(orc, 8, 5000, 6, missing=0.1, B=64)
    y = rng.normal(size=5000).astype(np.float32)
    P = orc.Params(loss=orc.LOSS_SQUARED, max_depth=4, eta=0.1, f=0.2)
    margin = np.full(5000, 0.5, np.float32)
    res = orc.train_tree(b, y, margin, P, iteration=3, want_detail=True)
    R = res.info.n_sampled
    assert abs(R - 1000) < 150 and res.nodes[0]["n_rows"] == R
    assert np.all(np.diff(res.sel) > 0)
    # selection reproduces through the step functions
    keys, e = orc.mvs_keys(res.gpair, 1.0)
    T = orc.mvs_threshold(keys, orc.mvs_target(0.2, 5000))
    assert T == res.info.T and e == res.info.e_key
    keep = orc.mvs_select(keys, T, 0, 3)
    assert np.array_equal(np.nonzero(keep)[0], res.sel)
    # root sums = sum of the reweighted fixed-point gradients
    assert int(res.nodes[0]["sum_g"]) == int(res.q[:, 0].sum())


def test_min_child_weight_and_gamma_block_splits(orc):
    X, b, rng = _small_data(orc, 10, 200, 3, missing=0.0)
    y = (rng.random(200) < 0.5).astype(np.float32)
    margin = np.zeros(200, np.float32)
    res = orc.train_tree(b, y, margin, orc.Params(max_depth=3, min_child_weight=1e9))
    assert res.nodes[0]["flags"] & orc.NODE_LEAF
    res = orc.train_tree(b, y, np.zeros(200, np.float32), orc.Params(max_depth=3, gamma=1e9))
    assert res.nodes[0]["flags"] & orc.NODE_LEAF
