"""Seeded synthetic workloads shaped like the paper's (Sec. 4) and the five
benchmark configurations.

This module only draws random data.  It holds none of the boosting method's
arithmetic, and both the HIP path's tests/benchmark and the CPU oracle consume
the same arrays from it.  Every generator is deterministic given
``numpy.random.SeedSequence([0, config_id, part])``; the row count can be
scaled down for tests while keeping the recipe.

Stand-ins:
  * config 2 has the shape of the Higgs data used in Sec. 4.3 (21 low-level and
    7 derived features, binary labels); the Higgs data are not available.
  * config 4 stands in for the 500-column scikit-learn set of Sec. 4.1
    (Table 1), whose generator the paper does not name.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

LOSS_LOGISTIC = 0
LOSS_SQUARED = 1


def _rng(cfg, part=0):
    return np.random.default_rng(np.random.SeedSequence([0, cfg, part]))


def _sigmoid(z):
    return 1.0 / (1.0 + np.exp(-z))


@dataclass
class TrainConfig:
    """Hyperparameters of a workload (unstated values use the defaults the
    paper implies: lambda=1, gamma=0, min_child_weight=1, eta=0.1)."""
    name: str
    loss: int
    max_bin: int
    max_depth: int
    n_trees: int
    eta: float = 0.1
    lambda_: float = 1.0
    gamma: float = 0.0
    min_child_weight: float = 1.0
    f: float = 1.0
    mvs_lambda: float = 1.0
    seed: int = 0

    @property
    def base_margin(self):
        # base_score 0.5: logit(0.5) = 0 for the logistic loss, 0.5 otherwise
        return 0.0 if self.loss == LOSS_LOGISTIC else 0.5


CONFIGS = {
    1: TrainConfig("tiny-dense-10k", LOSS_LOGISTIC, 256, 6, 10, eta=0.3),
    2: TrainConfig("higgs-shaped-1M", LOSS_LOGISTIC, 256, 8, 100, eta=0.1),
    3: TrainConfig("sampled-regression-10M", LOSS_SQUARED, 256, 8, 50, f=0.1),
    4: TrainConfig("out-of-core-200M", LOSS_LOGISTIC, 256, 8, 20, f=0.1),
    5: TrainConfig("wide-sparse-2M", LOSS_LOGISTIC, 64, 10, 20, gamma=0.1),
}

FULL_ROWS = {1: 10_000, 2: 1_000_000, 3: 10_000_000, 4: 200_000_000, 5: 2_000_000}
C4_PAGE_ROWS = 1 << 24


def config1(n=FULL_ROWS[1]):
    """n x 28 N(0,1) features, y ~ Bernoulli(sigmoid(X.w)), w ~ N(0,1)."""
    r = _rng(1)
    X = r.standard_normal((n, 28), dtype=np.float32)
    w = r.standard_normal(28)
    u = r.random(n)
    y = (u < _sigmoid(X.astype(np.float64) @ w)).astype(np.float32)
    return {"kind": "dense", "X": X, "y": y}


def _derived7(b):
    """Seven nonlinear columns built from the 21 base columns."""
    def ratio(a, c):
        return b[:, a] / (np.abs(b[:, c]) + np.float32(0.5))
    cols = [b[:, 0] * b[:, 1], b[:, 2] * b[:, 3], ratio(4, 5), b[:, 6] * b[:, 7],
            ratio(8, 9), b[:, 10] * b[:, 11], ratio(12, 13)]
    return np.stack(cols, axis=1).astype(np.float32)


def _mlp_labels(r, X, hidden, flip):
    m = X.shape[1]
    W1 = r.standard_normal((m, hidden)) / np.sqrt(m)
    w2 = r.standard_normal(hidden) / np.sqrt(hidden)
    z = np.tanh(X.astype(np.float64) @ W1) @ w2
    z = (z - z.mean()) / (z.std() + 1e-12)
    y = r.random(len(X)) < _sigmoid(2.0 * z)
    fl = r.random(len(X)) < flip
    return (y ^ fl).astype(np.float32)


def config2(n=FULL_ROWS[2]):
    """Higgs-shaped: 21 N(0,1) columns + 7 products/ratios; labels from a
    random 28-16-1 tanh network, then 5% label flips."""
    r = _rng(2)
    b = r.standard_normal((n, 21), dtype=np.float32)
    X = np.concatenate([b, _derived7(b)], axis=1)
    y = _mlp_labels(r, X, 16, 0.05)
    return {"kind": "dense", "X": np.ascontiguousarray(X), "y": y}


def config3(n=FULL_ROWS[3], m=50):
    """U(0,1) features; y = sum of 10 random depth-3 step functions +
    N(0, 0.1^2); then 20% of the entries are set missing (NaN)."""
    r = _rng(3)
    X = r.random((n, m), dtype=np.float32)
    y = np.zeros(n, np.float64)
    for _ in range(10):
        feats = r.integers(0, m, size=7)
        thr = r.uniform(0.2, 0.8, size=7).astype(np.float32)
        leaves = r.standard_normal(8)
        node = np.zeros(n, np.int64)
        for _level in range(3):
            go_right = X[np.arange(n), feats[node]] > thr[node]
            node = 2 * node + 1 + go_right
        y += leaves[node - 7]
    y += 0.1 * r.standard_normal(n)
    mask = r.random((n, m), dtype=np.float32) < np.float32(0.2)
    X[mask] = np.nan
    return {"kind": "dense", "X": X, "y": y.astype(np.float32)}


def config4_page(page, rows=C4_PAGE_ROWS, m=100):
    """One page of the out-of-core workload: N(0,1) features and labels of a
    fixed random 100-16-1 tanh network (weights shared by all pages) with 5%
    flips.  Pages are regenerated on demand; the 80 GB of raw floats are never
    held at once."""
    wr = _rng(4, 1_000_000)
    W1 = wr.standard_normal((m, 16)) / np.sqrt(m)
    w2 = wr.standard_normal(16) / np.sqrt(16)
    scale = float(wr.uniform(0.9, 1.1))
    r = _rng(4, page)
    X = r.standard_normal((rows, m), dtype=np.float32)
    z = np.tanh(X.astype(np.float64) @ W1) @ w2
    # the network output of N(0,1) inputs has std ~0.6: fixed scale, no
    # cross-page statistics
    y = r.random(rows) < _sigmoid(2.0 * scale * z / 0.6)
    fl = r.random(rows) < 0.05
    return {"kind": "dense", "X": X, "y": (y ^ fl).astype(np.float32)}


def config4_page_rows(n=FULL_ROWS[4], page_rows=C4_PAGE_ROWS):
    sizes = []
    left = n
    while left > 0:
        sizes.append(min(page_rows, left))
        left -= sizes[-1]
    return sizes


def config5(n=FULL_ROWS[5], m=2000, n_informative=50):
    """Wide sparse CSR: feature j (1-based) is present in each row with
    probability d_j = min(1, c * j^-1.1), c = 4.103 (Zipf popularity s=1.1,
    about 20 entries per row); values ~ LogNormal(0,1); labels from 50
    random informative features."""
    r = _rng(5)
    j = np.arange(1, m + 1, dtype=np.float64)
    dens = np.minimum(1.0, 4.103 * j ** -1.1)
    rows_l, feats_l = [], []
    for f in range(m):
        k = int(r.binomial(n, dens[f]))
        if k == 0:
            continue
        rows_l.append(r.choice(n, size=k, replace=False).astype(np.int64))
        feats_l.append(np.full(k, f, np.int64))
    rows_a = np.concatenate(rows_l)
    feats_a = np.concatenate(feats_l)
    order = np.argsort(rows_a * m + feats_a, kind="stable")
    rows_a, feats_a = rows_a[order], feats_a[order]
    vals = r.lognormal(0.0, 1.0, size=len(rows_a)).astype(np.float32)
    indptr = np.zeros(n + 1, np.int64)
    np.cumsum(np.bincount(rows_a, minlength=n), out=indptr[1:])
    info = r.choice(m, size=n_informative, replace=False)
    wts = r.standard_normal(n_informative)
    wfull = np.zeros(m)
    wfull[info] = wts
    z = np.bincount(rows_a, weights=vals.astype(np.float64) * wfull[feats_a], minlength=n)
    z = (z - z.mean()) / (z.std() + 1e-12)
    y = (r.random(n) < _sigmoid(2.0 * z)).astype(np.float32)
    return {"kind": "csr", "indptr": indptr, "indices": feats_a.astype(np.int32),
            "values": vals, "m": m, "y": y}


def make(cfg, n=None):
    """Data of config ``cfg`` (1, 2, 3 or 5) at n rows (default: full size)."""
    n = FULL_ROWS[cfg] if n is None else n
    return {1: config1, 2: config2, 3: config3, 5: config5}[cfg](n)
