"""Trees of the workloads at their full row counts against the oracle.

Each test trains one workload at full size, with its whole tree count, on
the GPU and with the oracle (its OpenMP build), on the same seeded data, and
requires identical node tables and margins after every tree: margins drift
tree by tree, so late trees are where a difference in the fp32 margins or in
the fixed-point exponents would show.  GBT_FULL_TREES=0 trains only the
first trees (a quick run).  The 200M-row out-of-core workload is checked here at
a reduced row count with the same page shape, feature count, sampling and
device budget; its full size runs in bench.py's out-of-core mode.
"""
import os

import numpy as np
import pytest

from oracle import oracle as orc
from paper_2005_09148_amd import datagen
from tests.gpu_helpers import node_diff, same_bits

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

FULL = os.environ.get("GBT_FULL_TREES", "1") == "1"


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


def oracle_bins(data, max_bin):
    if isinstance(data, dict):
        cuts = orc.sketch_cuts_csr(data["indptr"], data["indices"], data["values"], data["m"], max_bin)
        return orc.bin_csr(data["indptr"], data["indices"], data["values"], data["m"], cuts)
    return orc.bin_dense(data, orc.sketch_cuts_dense(data, max_bin))


def params(gbt, cfg):
    kw = dict(loss=cfg.loss, max_depth=cfg.max_depth, eta=cfg.eta, lambda_=cfg.lambda_, gamma=cfg.gamma,
              min_child_weight=cfg.min_child_weight, f=cfg.f, mvs_lambda=cfg.mvs_lambda, seed=cfg.seed)
    return gbt.make_train_params(**kw), orc.Params(**kw)


def check_trees(trees, margin, otrees, omargin):
    for t, (g, o) in enumerate(zip(trees, otrees)):
        d = node_diff(g.nodes, o.nodes)
        assert d is None, f"tree {t} node {d[0]}: gpu {d[1]} oracle {d[2]}"
    assert same_bits(margin, omargin)


def run_workload(gbt, ctx, cfg_id, n_trees):
    cfg = datagen.CONFIGS[cfg_id]
    d = datagen.make(cfg_id)
    data = d if d["kind"] == "csr" else d["X"]
    y = d["y"]
    mx = gbt.gbt_quantize(ctx, data, max_bin=cfg.max_bin)
    P, OP = params(gbt, cfg)
    trees, margin = gbt.train(ctx, mx, torch.from_numpy(y).cuda(), P, n_trees, cfg.base_margin)
    print(f"[fullsize] workload {cfg_id}: {n_trees} GPU trees done", flush=True)
    b = oracle_bins(data, cfg.max_bin)
    otrees, omargin = orc.train(b, y, OP, n_trees, cfg.base_margin)
    print(f"[fullsize] workload {cfg_id}: {n_trees} oracle trees done", flush=True)
    check_trees(trees, margin.cpu().numpy(), otrees, omargin)
    return trees


def test_full_tiny_dense(gbt, ctx):
    run_workload(gbt, ctx, 1, datagen.CONFIGS[1].n_trees)


def test_full_higgs_shaped(gbt, ctx):
    run_workload(gbt, ctx, 2, datagen.CONFIGS[2].n_trees if FULL else 3)


def test_full_sampled_regression(gbt, ctx):
    trees = run_workload(gbt, ctx, 3, datagen.CONFIGS[3].n_trees if FULL else 2)
    n = datagen.FULL_ROWS[3]
    for t in trees:  # about f n rows per tree
        assert 0.09 * n < t.stats.n_sampled < 0.11 * n


def test_full_wide_sparse(gbt, ctx):
    run_workload(gbt, ctx, 5, datagen.CONFIGS[5].n_trees if FULL else 2)


def test_out_of_core_shape(gbt):
    """Pages in pinned host memory, 100 features, MVS f = 0.1, depth 8, under a
    device budget (the out-of-core workload's shape at 2 pages of 2^17 rows):
    every tree streams the pages and matches the oracle."""
    cfg = datagen.CONFIGS[4]
    page_rows = 1 << 17
    parts = [datagen.config4_page(p, rows=page_rows) for p in range(2)]
    X = np.concatenate([p["X"] for p in parts])
    y = np.concatenate([p["y"] for p in parts])
    budget = 512 << 20
    c = gbt.Context(0, budget_bytes=budget)
    q = gbt.Quantizer(c, X.shape[1], len(y), max_bin=cfg.max_bin, page_rows=page_rows,
                      page_home=gbt.HOME_PINNED_HOST)
    for p in parts:
        q.sketch(p["X"])
    q.finalize()
    for p in parts:
        q.encode(p["X"])
    mx = q.end()
    assert mx.info().n_pages == 2
    P, OP = params(gbt, cfg)
    trees, margin = gbt.train(c, mx, torch.from_numpy(y).cuda(), P, 3, cfg.base_margin)
    used, peak = c.memory()
    assert peak <= budget
    assert all(t.stats.h2d_bytes > 0 for t in trees)
    b = oracle_bins(X, cfg.max_bin)
    otrees, omargin = orc.train(b, y, OP, 3, cfg.base_margin)
    check_trees(trees, margin.cpu().numpy(), otrees, omargin)
    del mx
    c.close()
