"""Pins of the oracle's batch-merged quantile sketch (Sec. 3.1, Alg. 3).

Each batch's column summary is folded into one running summary per feature.
What fixes it, other than the oracle itself:
  * lossless case: when no summary ever holds more than S distinct values
    every count is exact, so the cuts equal the exact rule over the whole
    sketch sample, computed here directly with numpy (sorted sample,
    candidate k at sorted position ceil(kN/B) - 1, duplicates and the
    maximum dropped), for any batching;
  * brute force: every summary count is at most the true number of sample
    values at or below its value (merging and pruning can only lose mass),
    exactly that number in one batch, and the last entry is the maximum
    with count N;
  * the rank error of every cut, counted by brute force on continuous data,
    stays within the bound that the prune rule allows (each prune of a
    summary over N' values loses less than N'/S + 2 values at any point,
    and merges add the losses of their inputs);
  * special cases: constant and all-missing features have no cuts; CSR input
    gives the cuts of the same data made dense with NaN for absent entries.
"""
import numpy as np
import pytest


def exact_cuts_numpy(col, B):
    """The exact rule over all (non-missing) values of one column."""
    s = np.sort(col[~np.isnan(col)].astype(np.float32))
    s[s == 0] = 0.0
    N = len(s)
    if N == 0:
        return np.zeros(0, np.float32)
    out = []
    for k in range(1, B):
        t = s[(k * N + B - 1) // B - 1]
        if t >= s[-1] or (out and t == out[-1]):
            continue
        out.append(t)
    return np.array(out, np.float32)


def cuts_of(cuts, j):
    return cuts.cut_values[cuts.cut_ptr[j]:cuts.cut_ptr[j + 1]]


def low_cardinality(seed, n, m):
    rng = np.random.default_rng(seed)
    X = rng.integers(-3, 4, size=(n, m)).astype(np.float32) * np.float32(0.5)
    X[:, 0] = 2.0                      # constant
    X[:, 1] = np.nan                   # all missing
    X[rng.random((n, m)) < 0.1] = np.nan
    X[::5, 2] = -0.0                   # -0 counts as +0
    X[:, 3] = rng.choice(np.array([0.25, 1e9, -7.0], np.float32), size=n, p=[0.98, 0.01, 0.01])
    return X


@pytest.mark.parametrize("batch_rows", [7_000, 1_001, 50_000, 333])
@pytest.mark.parametrize("B", [2, 4, 16, 256])
def test_lossless_merge_equals_the_exact_rule(orc, batch_rows, B):
    X = low_cardinality(1, 50_000, 6)
    cuts, ent = orc.sketch_cuts_merge_dense(X, B, 64, batch_rows, sketch_max_rows=1 << 30)
    assert (ent <= 64).all() and ent[1] == 0 and ent[0] == 1
    for j in range(X.shape[1]):
        assert cuts_of(cuts, j).tobytes() == exact_cuts_numpy(X[:, j], B).tobytes(), j
    # and the exact rule of the oracle itself on the same sample
    ex = orc.sketch_cuts_dense(X, B, sketch_max_rows=1 << 30)
    assert np.array_equal(cuts.cut_ptr, ex.cut_ptr) and cuts.cut_values.tobytes() == ex.cut_values.tobytes()


def test_lossless_merge_on_the_strided_sample(orc):
    # more rows than the sketch sample: the merged sketch sees every
    # ceil(n / sketch_max_rows)-th row, like the exact rule
    X = low_cardinality(2, 30_001, 5)
    cuts, _ = orc.sketch_cuts_merge_dense(X, 16, 64, 4_096, sketch_max_rows=10_000)
    for j in range(5):
        assert cuts_of(cuts, j).tobytes() == exact_cuts_numpy(X[::4, j], 16).tobytes()


def brute_count_le(sample, v):
    return int(np.count_nonzero(sample <= v))


def test_single_batch_summary_counts_are_exact(orc):
    rng = np.random.default_rng(3)
    n, S = 40_000, 300
    X = rng.normal(size=(n, 2)).astype(np.float32)
    X[:, 1] = np.round(X[:, 1] * 20) / 20  # ties
    for j in range(2):
        v, c = orc.sketch_summary_dense(X, j, S, n)
        col = X[:, j]
        assert len(v) <= S and np.all(np.diff(v) > 0)
        assert v[-1] == col.max() and c[-1] == n
        for vi, ci in zip(v, c):
            assert ci == brute_count_le(col, vi)


@pytest.mark.parametrize("n,S", [(40_000, 256), (99_999, 1024), (1_000, 512)])
def test_single_batch_prune_is_inverted_cdf_quantiles(orc, n, S):
    # one batch of more distinct values than S entries: the entries are the
    # values at ranks ceil(tN/S), which for a power-of-two S are numpy's
    # inverted-CDF quantiles at t/S (the library routine, not a retyping)
    rng = np.random.default_rng(n)
    X = rng.normal(size=(n, 1)).astype(np.float32)
    v, c = orc.sketch_summary_dense(X, 0, S, n)
    s = np.sort(X[:, 0])
    if n <= S:
        assert np.array_equal(v, s) and np.array_equal(c, np.arange(1, n + 1))
        return
    # (in float64: on a float32 array numpy forms the index n q in float32)
    s64 = s.astype(np.float64)
    want = np.unique(np.array([np.quantile(s64, t / S, method="inverted_cdf") for t in range(1, S + 1)],
                              np.float32))
    assert v.tobytes() == want.tobytes()
    assert np.array_equal(c, np.searchsorted(s, v, side="right"))


@pytest.mark.parametrize("B", [16, 64, 256])
def test_lossless_continuous_cuts_at_exact_ranks(orc, B):
    # 4096 distinct values (N divisible by B) in batches of 512, with room
    # for all of them: the cuts are the sorted values at ranks k N / B
    rng = np.random.default_rng(B)
    X = rng.normal(size=(4096, 1)).astype(np.float32)
    cuts, ent = orc.sketch_cuts_merge_dense(X, B, 8192, 512)
    assert ent[0] == 4096
    s = np.sort(X[:, 0])
    assert cuts.cut_values.tobytes() == s[np.arange(1, B) * (4096 // B) - 1].tobytes()


@pytest.mark.parametrize("S,batch_rows", [(512, 20_000), (128, 7_777), (2048, 3_000)])
def test_merged_counts_never_exceed_the_truth(orc, S, batch_rows):
    rng = np.random.default_rng(4)
    n = 120_000
    X = np.stack([rng.normal(size=n), rng.lognormal(size=n), rng.integers(0, 900, n) * 0.1], 1).astype(np.float32)
    for j in range(3):
        v, c = orc.sketch_summary_dense(X, j, S, batch_rows)
        col = np.sort(X[:, j])
        assert len(v) <= S and np.all(np.diff(v) > 0) and np.all(np.diff(c) > 0)
        assert v[-1] == col[-1] and c[-1] == n
        true = np.searchsorted(col, v, side="right")
        assert np.all(c <= true)
        assert (true - c).max() < error_bound(n, S, batch_rows)


def error_bound(n, S, batch_rows):
    """Values a summary may lose at one point: each prune of a summary over
    N' values loses less than N'/S + 2 (the mass between two kept entries);
    every batch is pruned once alone and once merged."""
    e, seen = 0.0, 0
    for b0 in range(0, n, batch_rows):
        nb = min(batch_rows, n - b0)
        seen += nb
        e += nb / S + 2 + seen / S + 2
    return e


@pytest.mark.parametrize("S,batch_rows,B", [(512, 20_000, 256), (256, 25_000, 64), (4096, 40_000, 256)])
def test_cut_ranks_within_the_bound(orc, S, batch_rows, B):
    rng = np.random.default_rng(5)
    n = 200_000
    X = np.stack([rng.normal(size=n), rng.uniform(size=n) ** 3], 1).astype(np.float32)
    cuts, ent = orc.sketch_cuts_merge_dense(X, B, S, batch_rows)
    assert (ent <= S).all()
    bound = error_bound(n, S, batch_rows) + n / S + 2  # plus the jump of one final entry
    for j in range(2):
        col = np.sort(X[:, j])
        t = cuts_of(cuts, j)
        assert len(t) == B - 1 and np.all(np.diff(t) > 0)
        ranks = np.searchsorted(col, t, side="right")
        target = np.ceil(np.arange(1, B) * n / B)
        assert np.all(ranks >= target)                # counts only ever fall short
        assert np.max(ranks - target) < bound, (np.max(ranks - target), bound)
    # a plausible mistake: merging by taking the batch's counts alone would
    # put the cuts of the last batch; check we are far from that failure
    assert bound < n / 20


def test_csr_equals_dense_with_missing(orc):
    rng = np.random.default_rng(6)
    n, m = 9_000, 40
    X = rng.lognormal(size=(n, m)).astype(np.float32)
    X[rng.random((n, m)) > 0.15] = np.nan
    rows, cols = np.nonzero(~np.isnan(X))
    indptr = np.concatenate([[0], np.cumsum(np.bincount(rows, minlength=n))]).astype(np.int64)
    for S, br in [(64, 2_000), (4096, 9_000), (16, 777)]:
        a, ea = orc.sketch_cuts_merge_csr(indptr, cols.astype(np.int32), X[rows, cols], m, 32, S, br)
        b, eb = orc.sketch_cuts_merge_dense(X, 32, S, br)
        assert np.array_equal(a.cut_ptr, b.cut_ptr) and a.cut_values.tobytes() == b.cut_values.tobytes()
        assert np.array_equal(ea, eb)


def test_rejects_bad_arguments(orc):
    X = np.zeros((10, 2), np.float32)
    for S, br in [(1, 5), (8, 0)]:
        with pytest.raises(ValueError):
            orc.sketch_cuts_merge_dense(X, 8, S, br)
    X[3, 1] = np.inf
    with pytest.raises(ValueError):
        orc.sketch_cuts_merge_dense(X, 8, 8, 4)
