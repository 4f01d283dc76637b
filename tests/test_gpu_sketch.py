"""Alg. 3's merged quantile sketch on the GPU against the oracle: the cuts
of every feature must equal the oracle's batch-merged cuts bit for bit, for
dense and CSR batches, host and device input, lossless (few distinct
values) and lossy (continuous) features, missing values, constant and
all-missing features, ragged batches and a strided sketch sample; a tree
trained on the pages equals the oracle's tree on the same cuts; and the
device holds one batch's keys, not the whole sample."""
import numpy as np
import pytest

from oracle import oracle as orc
from tests.gpu_helpers import node_diff, same_bits

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def gbt():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2005_09148_amd import gbt as g
    return g


@pytest.fixture(scope="module")
def ctx(gbt):
    c = gbt.Context(0)
    yield c
    c.close()


def make_dense(seed, n, m, kind, missing):
    rng = np.random.default_rng(seed)
    if kind == "normal":
        X = rng.normal(size=(n, m)).astype(np.float32)
    elif kind == "ties":
        X = (rng.integers(-5, 6, size=(n, m)) * 0.25).astype(np.float32)
    else:  # mixed: continuous, ties, heavy tail
        X = np.stack([rng.normal(size=n), rng.integers(0, 3, n), rng.lognormal(0, 3, n)] * ((m + 2) // 3),
                     1)[:, :m].astype(np.float32)
    if missing:
        X[rng.random(X.shape) < missing] = np.nan
    X[:, 0] = 1.5             # constant
    if m > 1:
        X[:, 1] = np.nan      # all missing
    if m > 2:
        X[::7, 2] = -0.0
    return X


def quantize_batches(gbt, ctx, X, max_bin, S, batch_rows, sketch_max_rows=0, device=False, **kw):
    n, m = X.shape
    q = gbt.Quantizer(ctx, m, n, max_bin=max_bin, sketch_max_rows=sketch_max_rows, sketch_summary=S, **kw)
    parts = [X[b:b + batch_rows] for b in range(0, n, batch_rows)]
    for p in parts:
        q.sketch(torch.from_numpy(np.ascontiguousarray(p)).cuda() if device else p)
    q.finalize()
    for p in parts:
        q.encode(p)
    return q.end()


@pytest.mark.parametrize("n,m,kind,missing,max_bin,S,batch_rows,smr", [
    (40_000, 6, "ties", 0.1, 256, 64, 7_000, 0),       # lossless: equals the exact rule
    (40_000, 6, "normal", 0.0, 256, 1024, 7_000, 0),   # lossy, ragged last batch
    (50_003, 9, "mixed", 0.2, 64, 256, 4_096, 0),
    (30_000, 5, "normal", 0.05, 2, 16, 1_000, 0),      # tiny summaries, many batches
    (25_000, 4, "normal", 0.0, 256, 8192, 25_000, 0),  # one batch, pruned once
    (60_001, 7, "mixed", 0.1, 128, 512, 9_999, 20_000),  # strided sample (every 4th row)
    (600_000, 3, "normal", 0.0, 256, 65_536, 150_000, 0),  # large summaries, pruned at every merge
])
def test_dense_merged_cuts_match_oracle(gbt, ctx, n, m, kind, missing, max_bin, S, batch_rows, smr):
    X = make_dense(n + m, n, m, kind, missing)
    mx = quantize_batches(gbt, ctx, X, max_bin, S, batch_rows, smr)
    cuts, _ = orc.sketch_cuts_merge_dense(X, max_bin, S, batch_rows, smr or (1 << 24))
    cp, cv = mx.cuts()
    assert same_bits(cp, cuts.cut_ptr) and same_bits(cv, cuts.cut_values)
    # the pages encode with these cuts
    b = orc.bin_dense(X, cuts)
    assert same_bits(mx.page(0), orc.ellpack(b, orc.ellpack_geometry(b)))
    mx.free()


def test_device_batches_match_host_batches(gbt, ctx):
    X = make_dense(3, 20_000, 5, "normal", 0.1)
    a = quantize_batches(gbt, ctx, X, 256, 300, 6_000)
    b = quantize_batches(gbt, ctx, X, 256, 300, 6_000, device=True)
    assert all(same_bits(u, v) for u, v in zip(a.cuts(), b.cuts()))
    a.free()
    b.free()


def to_csr(X):
    rows, cols = np.nonzero(~np.isnan(X))
    n = X.shape[0]
    indptr = np.concatenate([[0], np.cumsum(np.bincount(rows, minlength=n))]).astype(np.int64)
    return indptr, cols.astype(np.int32), X[rows, cols].astype(np.float32)


@pytest.mark.parametrize("S,batch_rows,max_bin", [(64, 3_000, 32), (1024, 11_000, 64), (8, 500, 16)])
def test_csr_merged_cuts_match_oracle(gbt, ctx, S, batch_rows, max_bin):
    rng = np.random.default_rng(S)
    n, m = 20_000, 120
    X = rng.lognormal(size=(n, m)).astype(np.float32)
    X[:, :10] = np.round(X[:, :10])
    X[rng.random((n, m)) > 0.08] = np.nan
    X[:, 5] = np.nan
    indptr, idx, val = to_csr(X)
    q = gbt.Quantizer(ctx, m, n, max_bin=max_bin, sketch_summary=S, kind=gbt.INPUT_CSR)
    batches = []
    for b0 in range(0, n, batch_rows):
        b1 = min(n, b0 + batch_rows)
        lo, hi = indptr[b0], indptr[b1]
        batches.append({"kind": "csr", "indptr": indptr[b0:b1 + 1] - lo, "indices": idx[lo:hi],
                        "values": val[lo:hi], "m": m})
    for bt in batches:
        q.sketch(bt)
    q.finalize()
    for bt in batches:
        q.encode(bt)
    mx = q.end()
    cuts, _ = orc.sketch_cuts_merge_csr(indptr, idx, val, m, max_bin, S, batch_rows)
    cp, cv = mx.cuts()
    assert same_bits(cp, cuts.cut_ptr) and same_bits(cv, cuts.cut_values)
    mx.free()


def test_trees_on_merged_cuts_match_oracle(gbt, ctx):
    # pinned pages quantized with the merged sketch, MVS sampling, three trees
    from paper_2005_09148_amd import datagen
    d = datagen.config2(n=30_000)
    X, y = d["X"], d["y"]
    mx = quantize_batches(gbt, ctx, X, 256, 512, 7_000, page_rows=7_000, page_home=gbt.HOME_PINNED_HOST)
    kw = dict(loss=orc.LOSS_LOGISTIC, max_depth=6, eta=0.1, f=0.3)
    trees, margin = gbt.train(ctx, mx, torch.from_numpy(y).cuda(), gbt.make_train_params(**kw), 3, 0.0)
    cuts, _ = orc.sketch_cuts_merge_dense(X, 256, 512, 7_000)
    otrees, omargin = orc.train(orc.bin_dense(X, cuts), y, orc.Params(**kw), 3, 0.0)
    for t, (g, o) in enumerate(zip(trees, otrees)):
        dd = node_diff(g.nodes, o.nodes)
        assert dd is None, f"tree {t} node {dd[0]}"
    assert same_bits(margin.cpu().numpy(), omargin)
    mx.free()


def test_merged_sketch_holds_one_batch(gbt):
    # 2^22 rows x 20 features in batches of 2^19: the exact sketch would
    # hold all 2^22 x 20 keys (320 MiB); the merged one a batch's keys
    # twice (for the sort), the staged batch and the summaries
    n, m, br, S = 1 << 22, 20, 1 << 19, 4096
    rng = np.random.default_rng(7)
    X = rng.normal(size=(n, m)).astype(np.float32)
    c = gbt.Context(0)
    try:
        q = gbt.Quantizer(c, m, n, max_bin=256, sketch_max_rows=n, sketch_summary=S,
                          page_rows=1 << 20, page_home=gbt.HOME_PINNED_HOST)
        for b0 in range(0, n, br):
            q.sketch(X[b0:b0 + br])
        q.finalize()
        peak = c.memory()[1]
        batch = br * m * 4
        assert peak < 3 * batch + 5 * m * S * 12 + (32 << 20), peak
        assert peak < (n * m * 4) // 2
        for b0 in range(0, n, br):
            q.encode(X[b0:b0 + br])
        mx = q.end()
        cuts, _ = orc.sketch_cuts_merge_dense(X, 256, S, br, n)
        cp, cv = mx.cuts()
        assert same_bits(cp, cuts.cut_ptr) and same_bits(cv, cuts.cut_values)
        mx.free()
    finally:
        c.close()


def test_rejects_bad_summary_size(gbt, ctx):
    for S in (1, -3, (1 << 20) + 1):
        with pytest.raises(gbt.GbtError):
            gbt.Quantizer(ctx, 3, 100, sketch_summary=S)


@pytest.mark.parametrize("S,batch_rows,n", [(2, 5_000, 30_000), (4, 1, 300), (3, 777, 9_001)])
def test_merged_sketch_small_summaries_and_tiny_batches(gbt, ctx, S, batch_rows, n):
    """The smallest summaries (S = 2: the minimum and the maximum survive each
    prune), one-row batches, and features missing in some batches only."""
    rng = np.random.default_rng(S * 1000 + batch_rows)
    m = 5
    X = rng.normal(size=(n, m)).astype(np.float32)
    X[: n // 2, 1] = np.nan          # missing in the first batches only
    X[n // 3:, 2] = np.nan           # present in the first batches only
    X[:, 3] = np.round(X[:, 3] * 2)  # ties
    X[rng.random((n, m)) < 0.1] = np.nan
    mx = quantize_batches(gbt, ctx, X, 64, S, batch_rows)
    cuts, _ = orc.sketch_cuts_merge_dense(X, 64, S, batch_rows)
    cp, cv = mx.cuts()
    assert same_bits(cp, cuts.cut_ptr) and same_bits(cv, cuts.cut_values)
    mx.free()


def test_empty_batches_change_nothing(gbt, ctx):
    X = make_dense(11, 20_000, 4, "normal", 0.1)
    q = gbt.Quantizer(ctx, 4, len(X), max_bin=128, sketch_summary=200)
    empty = X[:0]
    parts = [X[b:b + 3_000] for b in range(0, len(X), 3_000)]
    for p in parts:
        q.sketch(empty)
        q.sketch(p)
    q.sketch(empty)
    q.finalize()
    for p in parts:
        q.encode(p)
    mx = q.end()
    cuts, _ = orc.sketch_cuts_merge_dense(X, 128, 200, 3_000)
    cp, cv = mx.cuts()
    assert same_bits(cp, cuts.cut_ptr) and same_bits(cv, cuts.cut_values)
    mx.free()


def test_wide_csr_tiny_summaries(gbt, ctx):
    """3000 features, most of them empty in most batches, S = 4."""
    rng = np.random.default_rng(12)
    n, m = 6_000, 3_000
    X = np.full((n, m), np.nan, np.float32)
    nnz = 40_000
    r, cidx = rng.integers(0, n, nnz), (rng.zipf(1.3, nnz) - 1) % m
    X[r, cidx] = rng.lognormal(size=nnz).astype(np.float32)
    indptr, idx, val = to_csr(X)
    q = gbt.Quantizer(ctx, m, n, max_bin=16, sketch_summary=4, kind=gbt.INPUT_CSR)
    bounds = list(range(0, n, 1_000)) + [n]
    for b0, b1 in zip(bounds, bounds[1:]):
        lo, hi = indptr[b0], indptr[b1]
        q.sketch({"kind": "csr", "indptr": indptr[b0:b1 + 1] - lo, "indices": idx[lo:hi], "values": val[lo:hi],
                  "m": m})
    q.finalize()
    for b0, b1 in zip(bounds, bounds[1:]):
        lo, hi = indptr[b0], indptr[b1]
        q.encode({"kind": "csr", "indptr": indptr[b0:b1 + 1] - lo, "indices": idx[lo:hi], "values": val[lo:hi],
                  "m": m})
    mx = q.end()
    cuts, _ = orc.sketch_cuts_merge_csr(indptr, idx, val, m, 16, 4, 1_000)
    cp, cv = mx.cuts()
    assert same_bits(cp, cuts.cut_ptr) and same_bits(cv, cuts.cut_values)
    mx.free()


def test_outofcore_batch_shape(gbt, ctx):
    # the out-of-core workload's sketch at its own per-batch shape: N(0,1)
    # features, batches of 2^21 rows, every 12th row sampled (200M rows
    # under a 2^24-row sample take stride 12; here sketch_max_rows sets it),
    # so each batch adds about 174763 keys per feature to summaries of
    # 65536 entries, and every merge prunes
    n, m, br, S = 8 << 21, 4, 1 << 21, 65_536
    smr = -(-n // 12)
    assert -(-n // smr) == 12 and -(-200_000_000 // (1 << 24)) == 12
    X = np.random.default_rng(2005).standard_normal((n, m), dtype=np.float32)
    q = gbt.Quantizer(ctx, m, n, max_bin=256, sketch_max_rows=smr, sketch_summary=S)
    for b0 in range(0, n, br):
        q.sketch(X[b0:b0 + br])
    q.finalize()
    for b0 in range(0, n, br):
        q.encode(X[b0:b0 + br])
    mx = q.end()
    cuts, ent = orc.sketch_cuts_merge_dense(X, 256, S, br, smr)
    assert (ent <= S).all() and n // 12 > 16 * S  # pruned: the sample is far larger than a summary
    cp, cv = mx.cuts()
    assert same_bits(cp, cuts.cut_ptr) and same_bits(cv, cuts.cut_values)
    mx.free()
