"""Oracle pins for Sec. 3.1 (quantile cuts, Alg. 2/3) and Sec. 3.2 (ELLPACK
rows, Alg. 4/5).  CPU only."""
import json
import os

import numpy as np
import pytest

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def numpy_cuts(vals, B):
    """Cuts from numpy's inverted-CDF quantiles at k/B, then the dedupe/drop
    rule: keep distinct values strictly below the maximum."""
    s = np.sort(vals[~np.isnan(vals)])
    if len(s) == 0:
        return np.zeros(0, np.float32)
    qs = [np.quantile(s, k / B, method="inverted_cdf") for k in range(1, B)]
    out = []
    for t in qs:
        if t >= s[-1]:
            continue
        if out and t == out[-1]:
            continue
        out.append(t)
    return np.array(out, np.float32)


@pytest.mark.parametrize("B", [2, 4, 16, 64, 256])
@pytest.mark.parametrize("n", [1, 7, 100, 1001])
def test_cuts_match_numpy_inverted_cdf(orc, B, n):
    rng = np.random.default_rng(B * 1000 + n)
    X = np.stack([rng.normal(size=n), rng.integers(0, 5, n), rng.uniform(size=n)],
                 axis=1).astype(np.float32)
    X[rng.random(X.shape) < 0.1] = np.nan
    cuts = orc.sketch_cuts_dense(X, B)
    for j in range(3):
        got = cuts.cut_values[cuts.cut_ptr[j]:cuts.cut_ptr[j + 1]]
        assert np.array_equal(got, numpy_cuts(X[:, j], B)), j


def test_cuts_every_bin_nonempty_and_balanced(orc):
    rng = np.random.default_rng(5)
    X = rng.normal(size=(20000, 2)).astype(np.float32)
    cuts = orc.sketch_cuts_dense(X, 256)
    b = orc.bin_dense(X, cuts)
    for j in range(2):
        counts = np.bincount(b.dense[:, j], minlength=cuts.nbins[j])
        assert len(counts) == cuts.nbins[j] == 256
        assert counts.min() >= 1
        assert counts.max() <= 20000 / 256 + 2


def test_cuts_constant_and_all_missing_features(orc):
    X = np.zeros((50, 2), np.float32)
    X[:, 1] = np.nan
    cuts = orc.sketch_cuts_dense(X, 256)
    assert list(cuts.nbins) == [1, 1]


def test_negative_zero_is_canonical(orc):
    X = np.array([[-0.0], [0.0], [1.0], [2.0]] * 4, np.float32)
    cuts = orc.sketch_cuts_dense(X, 4)
    assert not np.signbit(cuts.cut_values).any()


def test_inf_is_rejected(orc):
    X = np.array([[1.0], [np.inf]], np.float32)
    with pytest.raises(ValueError):
        orc.sketch_cuts_dense(X, 4)


def test_sketch_stride_sample(orc):
    # above sketch_max_rows only rows i with i % ceil(n/max) == 0 are sketched
    rng = np.random.default_rng(8)
    X = rng.normal(size=(1003, 1)).astype(np.float32)
    cuts = orc.sketch_cuts_dense(X, 16, sketch_max_rows=100)
    stride = -(-1003 // 100)
    assert np.array_equal(cuts.cut_values, numpy_cuts(X[::stride, 0], 16))


def test_bins_are_searchsorted(orc):
    rng = np.random.default_rng(9)
    X = rng.normal(size=(3000, 4)).astype(np.float32)
    X[rng.random(X.shape) < 0.05] = np.nan
    cuts = orc.sketch_cuts_dense(X, 32)
    b = orc.bin_dense(X, cuts)
    for j in range(4):
        c = cuts.cut_values[cuts.cut_ptr[j]:cuts.cut_ptr[j + 1]]
        ref = np.searchsorted(c, X[:, j], side="left").astype(np.int64)
        ref[np.isnan(X[:, j])] = orc.MISSING
        assert np.array_equal(b.dense[:, j], ref)
    # x <= t_s  <=>  bin(x) < s  (the raw-value split predicate)
    j, s = 2, 5
    t = cuts.cut_values[cuts.cut_ptr[j] + s - 1]
    ok = ~np.isnan(X[:, j])
    assert np.array_equal(X[ok, j] <= t, b.dense[ok, j] < s)


def test_csr_cuts_equal_dense_cuts_with_absent_as_missing(orc):
    rng = np.random.default_rng(10)
    X = rng.normal(size=(500, 6)).astype(np.float32)
    X[rng.random(X.shape) < 0.6] = np.nan
    rows, cols = np.nonzero(~np.isnan(X))
    indptr = np.concatenate([[0], np.cumsum(np.bincount(rows, minlength=500))])
    vals = X[rows, cols]
    c1 = orc.sketch_cuts_dense(X, 16)
    c2 = orc.sketch_cuts_csr(indptr, cols, vals, 6, 16)
    assert np.array_equal(c1.cut_ptr, c2.cut_ptr)
    assert np.array_equal(c1.cut_values, c2.cut_values)
    b = orc.bin_csr(indptr, cols, vals, 6, c2)
    d = orc.bin_dense(X, c1)
    assert np.array_equal(d.dense[rows, cols], b.bin)


def test_csr_rejects_unsorted_indices(orc):
    cuts = orc.Cuts(np.array([0, 0, 0], np.int32), np.zeros(0, np.float32))
    with pytest.raises(ValueError):
        orc.bin_csr([0, 2], [1, 0], [1.0, 2.0], 2, cuts)


def decode(words, w, stride):
    """Independent decoder: read the LSB-first bit stream symbol by symbol."""
    n = words.shape[0]
    bits = np.unpackbits(words.astype("<u4").view(np.uint8).reshape(n, -1), axis=1,
                         bitorder="little")
    out = np.zeros((n, stride), np.int64)
    for s in range(stride):
        for b in range(w):
            out[:, s] |= bits[:, s * w + b].astype(np.int64) << b
    return out


def test_ellpack_hand_packed_golden(orc):
    g = json.load(open(os.path.join(GOLDEN, "ellpack_hand_packed.json")))
    for case in g["cases"]:
        bins = np.array(case["bins"], np.uint16)
        nb = np.array(case["nbins"], np.int32)
        cuts = orc.Cuts(np.concatenate([[0], np.cumsum(nb - 1)]).astype(np.int32),
                        np.zeros(int((nb - 1).sum()), np.float32))
        b = orc.Binned(bins.shape[0], bins.shape[1], cuts, dense=bins)
        geo = orc.ellpack_geometry(b)
        assert (geo.w, geo.null, geo.row_words) == (case["w"], case["null"], case["row_words"])
        assert orc.ellpack(b, geo).tolist() == case["words"]


def test_ellpack_dense_roundtrip(orc):
    rng = np.random.default_rng(12)
    X = rng.normal(size=(2001, 50)).astype(np.float32)
    X[rng.random(X.shape) < 0.2] = np.nan
    cuts = orc.sketch_cuts_dense(X, 256)
    b = orc.bin_dense(X, cuts)
    geo = orc.ellpack_geometry(b)
    assert geo.w == 9 and geo.null == 511 and geo.row_words == 16  # 450 bits -> 15 -> 16 words
    page = orc.ellpack(b, geo)
    sym = decode(page, geo.w, geo.stride)
    ref = b.dense.astype(np.int64)
    ref[ref == orc.MISSING] = geo.null
    assert np.array_equal(sym, ref)
    # padding words are zero
    assert (page[:, 15] == 0).all()


def test_ellpack_dense_without_missing_uses_8_bits(orc):
    rng = np.random.default_rng(13)
    X = rng.normal(size=(1000, 28)).astype(np.float32)
    b = orc.bin_dense(X, orc.sketch_cuts_dense(X, 256))
    geo = orc.ellpack_geometry(b)
    assert (geo.w, geo.stride, geo.row_words) == (8, 28, 8)


def test_ellpack_sparse_roundtrip(orc):
    rng = np.random.default_rng(14)
    n, m = 300, 40
    X = rng.lognormal(size=(n, m)).astype(np.float32)
    X[rng.random(X.shape) < 0.8] = np.nan
    rows, cols = np.nonzero(~np.isnan(X))
    indptr = np.concatenate([[0], np.cumsum(np.bincount(rows, minlength=n))])
    vals = X[rows, cols]
    cuts = orc.sketch_cuts_csr(indptr, cols, vals, m, 64)
    b = orc.bin_csr(indptr, cols, vals, m, cuts)
    geo = orc.ellpack_geometry(b)
    tb = int(cuts.nbins.sum())
    assert geo.null == tb and geo.stride == int(np.diff(indptr).max())
    assert (1 << geo.w) > tb >= (1 << (geo.w - 1))
    sym = decode(orc.ellpack(b, geo), geo.w, geo.stride)
    off = np.concatenate([[0], np.cumsum(cuts.nbins)])
    for i in range(n):
        e0, e1 = indptr[i], indptr[i + 1]
        want = list(off[b.feat[e0:e1]] + b.bin[e0:e1]) + [tb] * (geo.stride - (e1 - e0))
        assert list(sym[i]) == want
