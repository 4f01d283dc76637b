"""CPU oracle for out-of-core GPU gradient boosting (Ou, KDD 2020).

TEST INFRASTRUCTURE ONLY: the tests, the smoke check and the benchmark's
CPU-baseline leg are the only callers.  The product library never imports
this module and this module never imports the product library.

A thin ctypes layer over ``gbt_oracle.c`` (plain C, double precision, built
with -O2 -ffp-contract=off).  Every function cites the passage of the paper
it follows; the readings of passages the paper leaves open are written out
in ``gbt_oracle.c``.  Two builds of the same source: ``plain`` (single
threaded) and ``omp`` (-fopenmp: loops over independent rows or features,
and integer or maximum reductions, spread over threads; the same bits, which
a CPU test checks).  ``select()`` chooses the build the functions below call;
the default is ``omp`` unless GBT_ORACLE=plain is set.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess
from dataclasses import dataclass, field

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "gbt_oracle.c")
_LIBS = {"plain": os.path.join(_HERE, "liboracle.so"), "omp": os.path.join(_HERE, "liboracle_omp.so")}

LOSS_LOGISTIC = 0
LOSS_SQUARED = 1
NODE_PRESENT = 1
NODE_LEAF = 2
NODE_DEFAULT_LEFT = 4
MISSING = 0xFFFF


def build(force: bool = True) -> str:
    """Compile gbt_oracle.c into liboracle.so (plain gcc, no fast-math) and
    liboracle_omp.so (the same with -fopenmp)."""
    for kind, path in _LIBS.items():
        if force or not os.path.exists(path) or os.path.getmtime(path) < os.path.getmtime(_SRC):
            tmp = path + ".tmp"
            extra = ["-fopenmp"] if kind == "omp" else []
            subprocess.check_call(
                ["gcc", "-O2", "-ffp-contract=off", "-fno-fast-math", "-std=gnu11", "-fPIC",
                 "-shared", *extra, "-o", tmp, _SRC, "-lm"])
            os.replace(tmp, path)
    return _LIBS["plain"]


class OrcData(C.Structure):
    _fields_ = [("n", C.c_int64), ("m", C.c_int32), ("pad0", C.c_int32),
                ("dense", C.c_void_p), ("indptr", C.c_void_p), ("feat", C.c_void_p),
                ("bin", C.c_void_p), ("nbins", C.c_void_p), ("cut_ptr", C.c_void_p),
                ("cut_values", C.c_void_p)]


class OrcParams(C.Structure):
    _fields_ = [("loss", C.c_int32), ("max_depth", C.c_int32), ("eta", C.c_double),
                ("lambda_", C.c_double), ("gamma", C.c_double),
                ("min_child_weight", C.c_double), ("f", C.c_double),
                ("mvs_lambda", C.c_double), ("seed", C.c_uint64), ("iteration", C.c_uint64),
                ("sampler", C.c_int32), ("pad0", C.c_int32), ("goss_a", C.c_double)]


class OrcInfo(C.Structure):
    _fields_ = [("n_sampled", C.c_int64), ("K", C.c_int64), ("T", C.c_int64),
                ("e_key", C.c_int32), ("e_g", C.c_int32), ("e_h", C.c_int32),
                ("n_nodes", C.c_int32)]


class OrcSplit(C.Structure):
    _fields_ = [("gain", C.c_double), ("left_g", C.c_int64), ("left_h", C.c_int64),
                ("right_g", C.c_int64), ("right_h", C.c_int64), ("feature", C.c_int32),
                ("split_bin", C.c_int32), ("default_left", C.c_int32), ("valid", C.c_int32)]


NODE_DTYPE = np.dtype([("feature", "<i4"), ("split_bin", "<i4"), ("threshold", "<f4"),
                       ("leaf_value", "<f4"), ("gain", "<f8"), ("sum_g", "<i8"),
                       ("sum_h", "<i8"), ("n_rows", "<i4"), ("flags", "u1"),
                       ("pad", "u1", (3,))])
assert NODE_DTYPE.itemsize == 48

_loaded = {}
_kind = os.environ.get("GBT_ORACLE", "omp")
if _kind not in _LIBS:
    raise ValueError(f"GBT_ORACLE={_kind!r}: expected 'plain' or 'omp'")


def select(kind: str) -> str:
    """Make the functions of this module call build `kind` ('plain' or
    'omp'); returns the previous choice."""
    global _kind
    if kind not in _LIBS:
        raise ValueError(kind)
    prev, _kind = _kind, kind
    return prev


def threads(n: int = 0) -> int:
    """Threads of the omp build (n > 0 sets them); 1 for the plain build."""
    L = lib()
    return int(L.orc_threads(int(n)))


def lib():
    if _kind not in _loaded:
        path = _LIBS[_kind]
        if not os.path.exists(path) or os.path.getmtime(path) < os.path.getmtime(_SRC):
            build(force=False)
        L = C.CDLL(path)
        vp, i64, i32, f64, u64 = C.c_void_p, C.c_int64, C.c_int32, C.c_double, C.c_uint64
        sig = {
            "orc_exp": (f64, [f64]),
            "orc_philox4x64_10": (None, [vp, vp, vp]),
            "orc_sketch_cuts_dense": (C.c_int, [vp, i64, i32, i64, i32, i64, vp, vp]),
            "orc_sketch_cuts_csr": (C.c_int, [vp, vp, vp, i64, i32, i32, i64, vp, vp]),
            "orc_sketch_cuts_merge_dense": (C.c_int, [vp, i64, i32, i64, i32, i64, i32, i64, vp, vp, vp]),
            "orc_sketch_cuts_merge_csr": (C.c_int, [vp, vp, vp, i64, i32, i32, i64, i32, i64, vp, vp, vp]),
            "orc_sketch_summary_dense": (i64, [vp, i64, i32, i64, i64, i32, i64, i32, vp, vp]),
            "orc_bin_dense": (C.c_int, [vp, i64, i32, i64, vp, vp, vp]),
            "orc_bin_csr": (C.c_int, [vp, vp, vp, i64, i32, vp, vp, vp, vp, vp]),
            "orc_ellpack_geometry": (None, [i32, i32, vp, i32, i32, vp]),
            "orc_ellpack_dense": (None, [vp, i64, i32, i32, i32, C.c_uint32, vp]),
            "orc_ellpack_csr": (None, [vp, vp, vp, i64, i32, vp, i32, i32, i32, C.c_uint32, vp]),
            "orc_gradients": (C.c_int, [i32, vp, vp, vp, i64, vp]),
            "orc_mvs_keys": (C.c_int, [vp, i64, f64, vp, vp]),
            "orc_mvs_target": (i64, [f64, i64]),
            "orc_mvs_threshold": (i64, [vp, i64, i64]),
            "orc_mvs_uniform": (u64, [u64, u64, u64]),
            "orc_mvs_select": (None, [vp, i64, i64, u64, u64, i64, vp]),
            "orc_mvs_weight": (f64, [i64, i64]),
            "orc_sgb_select": (None, [i64, f64, u64, u64, i64, vp]),
            "orc_goss_top_threshold": (i64, [vp, i64, i64]),
            "orc_goss_top_count": (i64, [f64, i64]),
            "orc_goss_select": (None, [vp, i64, i64, f64, f64, u64, u64, i64, vp]),
            "orc_goss_weight": (f64, [i64, i64, f64, f64]),
            "orc_fixed_point": (None, [vp, i64, vp, vp, vp]),
            "orc_build_hist": (None, [vp, vp, i64, vp, vp]),
            "orc_eval_node": (None, [vp, vp, vp, i32, vp, i32, i32, vp]),
            "orc_partition": (i64, [vp, vp, i64, i32, i32, i32, vp]),
            "orc_leaf_value": (C.c_float, [i64, i64, i32, i32, f64, f64]),
            "orc_mvs_lambda_estimate": (f64, [i32, vp, vp, i64]),
            "orc_train_tree": (C.c_int, [vp, vp, vp, vp, vp, vp, vp, vp, vp]),
            "orc_predict_binned": (None, [vp, vp, vp, i32, C.c_float, vp]),
            "orc_predict_raw_dense": (None, [vp, i64, i64, vp, vp, i32, C.c_float, vp]),
            "orc_predict_raw_csr": (None, [vp, vp, vp, i64, vp, vp, i32, C.c_float, vp]),
            "orc_threads": (i32, [i32]),
        }
        for name, (res, args) in sig.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _loaded[_kind] = L
    return _loaded[_kind]


def _p(a):
    return None if a is None else a.ctypes.data_as(C.c_void_p)


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


# --------------------------------------------------------------------------
# helpers
# --------------------------------------------------------------------------
def exp(x: float) -> float:
    """Cody-Waite / Taylor exp used by the logistic loss (Eq. 4-5 helper)."""
    return lib().orc_exp(float(x))


def philox4x64_10(ctr, key):
    """Philox4x64-10 block (Salmon et al., SC'11) of a 256-bit counter."""
    c = np.asarray(ctr, dtype=np.uint64)
    k = np.asarray(key, dtype=np.uint64)
    out = np.zeros(4, dtype=np.uint64)
    lib().orc_philox4x64_10(_p(c), _p(k), _p(out))
    return out


# --------------------------------------------------------------------------
# Sec. 3.1 (Alg. 2/3) cuts and Sec. 3.2 (Alg. 4/5) ELLPACK rows
# --------------------------------------------------------------------------
@dataclass
class Cuts:
    cut_ptr: np.ndarray      # int32 [m+1]
    cut_values: np.ndarray   # float32 [cut_ptr[m]]

    @property
    def m(self):
        return len(self.cut_ptr) - 1

    @property
    def nbins(self):
        return (np.diff(self.cut_ptr) + 1).astype(np.int32)


def sketch_cuts_dense(X, max_bin, sketch_max_rows=1 << 24) -> Cuts:
    X = _c(X, np.float32)
    n, m = X.shape
    cp = np.zeros(m + 1, np.int32)
    cv = np.zeros(m * (max_bin - 1) + 1, np.float32)
    rc = lib().orc_sketch_cuts_dense(_p(X), n, m, m, max_bin, sketch_max_rows, _p(cp), _p(cv))
    if rc:
        raise ValueError(f"orc_sketch_cuts_dense failed ({rc})")
    return Cuts(cp, cv[:cp[m]].copy())


def sketch_cuts_csr(indptr, indices, values, m, max_bin, sketch_max_rows=1 << 24) -> Cuts:
    indptr, indices, values = _c(indptr, np.int64), _c(indices, np.int32), _c(values, np.float32)
    n = len(indptr) - 1
    cp = np.zeros(m + 1, np.int32)
    cv = np.zeros(m * (max_bin - 1) + 1, np.float32)
    rc = lib().orc_sketch_cuts_csr(_p(indptr), _p(indices), _p(values), n, m, max_bin,
                                   sketch_max_rows, _p(cp), _p(cv))
    if rc:
        raise ValueError(f"orc_sketch_cuts_csr failed ({rc})")
    return Cuts(cp, cv[:cp[m]].copy())


def sketch_cuts_merge_dense(X, max_bin, summary_size, batch_rows, sketch_max_rows=1 << 24):
    """Sec. 3.1 Alg. 3: cuts from per-batch summaries (batches of batch_rows
    rows) merged into one running summary of at most summary_size entries
    per feature; returns (Cuts, entries per feature)."""
    X = _c(X, np.float32)
    n, m = X.shape
    cp = np.zeros(m + 1, np.int32)
    cv = np.zeros(m * (max_bin - 1) + 1, np.float32)
    ent = np.zeros(m, np.int64)
    rc = lib().orc_sketch_cuts_merge_dense(_p(X), n, m, m, max_bin, sketch_max_rows, summary_size, batch_rows,
                                           _p(cp), _p(cv), _p(ent))
    if rc:
        raise ValueError(f"orc_sketch_cuts_merge_dense failed ({rc})")
    return Cuts(cp, cv[:cp[m]].copy()), ent


def sketch_cuts_merge_csr(indptr, indices, values, m, max_bin, summary_size, batch_rows,
                          sketch_max_rows=1 << 24):
    indptr, indices, values = _c(indptr, np.int64), _c(indices, np.int32), _c(values, np.float32)
    n = len(indptr) - 1
    cp = np.zeros(m + 1, np.int32)
    cv = np.zeros(m * (max_bin - 1) + 1, np.float32)
    ent = np.zeros(m, np.int64)
    rc = lib().orc_sketch_cuts_merge_csr(_p(indptr), _p(indices), _p(values), n, m, max_bin, sketch_max_rows,
                                         summary_size, batch_rows, _p(cp), _p(cv), _p(ent))
    if rc:
        raise ValueError(f"orc_sketch_cuts_merge_csr failed ({rc})")
    return Cuts(cp, cv[:cp[m]].copy()), ent


def sketch_summary_dense(X, j, summary_size, batch_rows, sketch_max_rows=1 << 24):
    """The final running summary of feature j: (values, counts)."""
    X = _c(X, np.float32)
    n, m = X.shape
    v = np.zeros(summary_size + 1, np.float32)
    c = np.zeros(summary_size + 1, np.int64)
    k = lib().orc_sketch_summary_dense(_p(X), n, m, m, sketch_max_rows, summary_size, batch_rows, j, _p(v), _p(c))
    if k < 0:
        raise ValueError("orc_sketch_summary_dense failed")
    return v[:k].copy(), c[:k].copy()


@dataclass
class Binned:
    """A binned matrix: dense uint16 bins (MISSING = 0xFFFF) or CSR bins."""
    n: int
    m: int
    cuts: Cuts
    dense: np.ndarray | None = None
    indptr: np.ndarray | None = None
    feat: np.ndarray | None = None
    bin: np.ndarray | None = None
    _keep: list = field(default_factory=list)

    @property
    def sparse(self):
        return self.dense is None

    def struct(self) -> OrcData:
        nb = self.cuts.nbins
        cp = self.cuts.cut_ptr
        cv = self.cuts.cut_values if len(self.cuts.cut_values) else np.zeros(1, np.float32)
        self._keep = [nb, cp, cv]
        s = OrcData()
        s.n, s.m = self.n, self.m
        s.dense = _p(self.dense) if self.dense is not None else None
        s.indptr = _p(self.indptr)
        s.feat = _p(self.feat)
        s.bin = _p(self.bin)
        s.nbins, s.cut_ptr, s.cut_values = _p(nb), _p(cp), _p(cv)
        return s

    def has_missing(self) -> bool:
        return bool(self.dense is not None and (self.dense == MISSING).any())

    def max_row_nnz(self) -> int:
        if self.dense is not None:
            return self.m
        return int(np.diff(self.indptr).max()) if self.n else 0


def bin_dense(X, cuts: Cuts) -> Binned:
    X = _c(X, np.float32)
    n, m = X.shape
    out = np.empty((n, m), np.uint16)
    cv = cuts.cut_values if len(cuts.cut_values) else np.zeros(1, np.float32)
    rc = lib().orc_bin_dense(_p(X), n, m, m, _p(cuts.cut_ptr), _p(cv), _p(out))
    if rc:
        raise ValueError("orc_bin_dense failed")
    return Binned(n, m, cuts, dense=out)


def bin_csr(indptr, indices, values, m, cuts: Cuts) -> Binned:
    indptr, indices, values = _c(indptr, np.int64), _c(indices, np.int32), _c(values, np.float32)
    n = len(indptr) - 1
    nnz = len(values)
    oi = np.zeros(n + 1, np.int64)
    of = np.zeros(max(nnz, 1), np.int32)
    ob = np.zeros(max(nnz, 1), np.uint16)
    cv = cuts.cut_values if len(cuts.cut_values) else np.zeros(1, np.float32)
    rc = lib().orc_bin_csr(_p(indptr), _p(indices), _p(values), n, m, _p(cuts.cut_ptr), _p(cv),
                           _p(oi), _p(of), _p(ob))
    if rc:
        raise ValueError("orc_bin_csr failed (unsorted/duplicate indices or inf)")
    k = int(oi[-1])
    return Binned(n, m, cuts, indptr=oi, feat=of[:k].copy(), bin=ob[:k].copy())


@dataclass
class Geometry:
    w: int
    stride: int
    row_words: int
    null: int


def ellpack_geometry(b: Binned, has_missing=None, max_row_nnz=None) -> Geometry:
    out = np.zeros(4, np.int32)
    hm = b.has_missing() if has_missing is None else has_missing
    mr = b.max_row_nnz() if max_row_nnz is None else max_row_nnz
    lib().orc_ellpack_geometry(int(b.sparse), b.m, _p(b.cuts.nbins), int(hm), int(mr), _p(out))
    return Geometry(*[int(v) for v in out])


def ellpack(b: Binned, geo: Geometry | None = None) -> np.ndarray:
    """ELLPACK rows (uint32 [n, row_words]) of a binned matrix."""
    geo = geo or ellpack_geometry(b)
    out = np.zeros((b.n, geo.row_words), np.uint32)
    if b.sparse:
        lib().orc_ellpack_csr(_p(b.indptr), _p(b.feat), _p(b.bin), b.n, b.m, _p(b.cuts.nbins),
                              geo.w, geo.stride, geo.row_words, geo.null, _p(out))
    else:
        lib().orc_ellpack_dense(_p(b.dense), b.n, b.m, geo.w, geo.row_words, geo.null, _p(out))
    return out


# --------------------------------------------------------------------------
# Eq. 4-5 gradients, Eq. 9 / Alg. 7 sampling, fixed point
# --------------------------------------------------------------------------
def gradients(loss, margin, label, weight=None):
    margin, label = _c(margin, np.float32), _c(label, np.float32)
    w = None if weight is None else _c(weight, np.float32)
    out = np.empty((len(margin), 2), np.float32)
    rc = lib().orc_gradients(loss, _p(margin), _p(label), _p(w), len(margin), _p(out))
    if rc:
        raise ValueError("orc_gradients failed")
    return out


def mvs_keys(gpair, mvs_lambda):
    gpair = _c(gpair, np.float32)
    n = len(gpair)
    keys = np.empty(n, np.int64)
    e = np.zeros(1, np.int32)
    rc = lib().orc_mvs_keys(_p(gpair), n, float(mvs_lambda), _p(keys), _p(e))
    if rc:
        raise ValueError("orc_mvs_keys failed")
    return keys, int(e[0])


def mvs_target(f, n):
    return int(lib().orc_mvs_target(float(f), int(n)))


def mvs_threshold(keys, K):
    keys = _c(keys, np.int64)
    return int(lib().orc_mvs_threshold(_p(keys), len(keys), int(K)))


def mvs_uniform(seed, iteration, row):
    return int(lib().orc_mvs_uniform(seed, iteration, row))


def mvs_select(keys, T, seed, iteration, row_offset=0):
    keys = _c(keys, np.int64)
    keep = np.zeros(len(keys), np.uint8)
    lib().orc_mvs_select(_p(keys), len(keys), int(T), seed, iteration, row_offset, _p(keep))
    return keep.astype(bool)


def mvs_weight(a, T):
    return lib().orc_mvs_weight(int(a), int(T))


SAMPLE_MVS, SAMPLE_SGB, SAMPLE_GOSS = 0, 1, 2


def sgb_select(n, f, seed, iteration, row_offset=0):
    keep = np.zeros(max(n, 1), np.uint8)
    lib().orc_sgb_select(int(n), float(f), seed, iteration, row_offset, _p(keep))
    return keep[:n].astype(bool)


def goss_top_count(a, n):
    return int(lib().orc_goss_top_count(float(a), int(n)))


def goss_top_threshold(keys, A):
    keys = _c(keys, np.int64)
    if keys.size == 0:
        keys = np.zeros(1, np.int64)
        return int(lib().orc_goss_top_threshold(_p(keys), 0, int(A)))
    return int(lib().orc_goss_top_threshold(_p(keys), len(keys), int(A)))


def goss_select(keys, T_top, a, b, seed, iteration, row_offset=0):
    keys = _c(keys, np.int64)
    keep = np.zeros(len(keys), np.uint8)
    lib().orc_goss_select(_p(keys), len(keys), int(T_top), float(a), float(b), seed, iteration, row_offset,
                          _p(keep))
    return keep.astype(bool)


def goss_weight(key, T_top, a, b):
    return lib().orc_goss_weight(int(key), int(T_top), float(a), float(b))


def fixed_point(gw):
    gw = _c(gw, np.float64).reshape(-1, 2)
    q = np.empty_like(gw, dtype=np.int64)
    eg, eh = np.zeros(1, np.int32), np.zeros(1, np.int32)
    lib().orc_fixed_point(_p(gw), len(gw), _p(q), _p(eg), _p(eh))
    return q, int(eg[0]), int(eh[0])


# --------------------------------------------------------------------------
# Alg. 1 steps
# --------------------------------------------------------------------------
def build_hist(b: Binned, rows, q):
    rows = _c(rows, np.int64)
    q = _c(q, np.int64)
    tb = int(b.cuts.nbins.sum())
    hist = np.zeros((max(tb, 1), 2), np.int64)
    s = b.struct()
    lib().orc_build_hist(C.byref(s), _p(rows), len(rows), _p(q), _p(hist))
    return hist[:tb]


@dataclass
class Params:
    loss: int = LOSS_LOGISTIC
    max_depth: int = 6
    eta: float = 0.3
    lambda_: float = 1.0
    gamma: float = 0.0
    min_child_weight: float = 1.0
    f: float = 1.0
    mvs_lambda: float = 1.0
    seed: int = 0
    sampler: int = 0      # SAMPLE_MVS, SAMPLE_SGB or SAMPLE_GOSS (when f < 1)
    goss_a: float = 0.0   # GOSS top fraction a (the rest fraction is f - a)

    def struct(self, iteration=0) -> OrcParams:
        return OrcParams(self.loss, self.max_depth, self.eta, self.lambda_, self.gamma,
                         self.min_child_weight, self.f, self.mvs_lambda, self.seed, iteration,
                         self.sampler, 0, self.goss_a)


def eval_node(hist, node_sum, nbins, params: Params, e_g, e_h):
    hist = _c(hist, np.int64)
    ns = _c(node_sum, np.int64)
    nb = _c(nbins, np.int32)
    ps = params.struct()
    out = OrcSplit()
    if hist.size == 0:
        hist = np.zeros((1, 2), np.int64)
    lib().orc_eval_node(_p(hist), _p(ns), _p(nb), len(nb), C.byref(ps), e_g, e_h, C.byref(out))
    return out


def partition(b: Binned, rows, feature, split_bin, default_left):
    rows = _c(rows, np.int64)
    out = np.empty_like(rows)
    s = b.struct()
    nl = lib().orc_partition(C.byref(s), _p(rows), len(rows), feature, split_bin,
                             int(default_left), _p(out))
    return out[:nl], out[nl:]


def mvs_lambda_estimate(loss, margin, label):
    """Sec. 2.4: MVS lambda as the squared initial leaf value (-G/H of every
    row at the given margins, from the exact fixed-point sums)."""
    margin, label = _c(margin, np.float32), _c(label, np.float32)
    v = lib().orc_mvs_lambda_estimate(int(loss), _p(margin), _p(label), len(margin))
    if v < 0:
        raise ValueError("orc_mvs_lambda_estimate failed")
    return float(v)


def leaf_value(Qg, Qh, e_g, e_h, lambda_, eta):
    return float(lib().orc_leaf_value(int(Qg), int(Qh), e_g, e_h, lambda_, eta))


@dataclass
class TreeResult:
    nodes: np.ndarray
    info: OrcInfo
    sel: np.ndarray | None
    q: np.ndarray | None
    gpair: np.ndarray | None


def train_tree(b: Binned, label, margin, params: Params, iteration=0, want_detail=False):
    """One boosting iteration (Alg. 7 then Alg. 1); margin is updated in place."""
    label = _c(label, np.float32)
    assert margin.dtype == np.float32 and margin.flags.c_contiguous
    nn = (1 << (params.max_depth + 1)) - 1
    nodes = np.zeros(nn, NODE_DTYPE)
    info = OrcInfo()
    sel = np.empty(max(b.n, 1), np.int64) if want_detail else None
    q = np.empty((max(b.n, 1), 2), np.int64) if want_detail else None
    gp = np.empty((max(b.n, 1), 2), np.float32) if want_detail else None
    s = b.struct()
    ps = params.struct(iteration)
    rc = lib().orc_train_tree(C.byref(s), _p(label), _p(margin), C.byref(ps), _p(nodes),
                              C.byref(info), _p(sel), _p(q), _p(gp))
    if rc:
        raise ValueError(f"orc_train_tree failed ({rc})")
    R = info.n_sampled
    return TreeResult(nodes, info, sel[:R] if want_detail else None,
                      q[:R] if want_detail else None, gp[:b.n] if want_detail else None)


def train(b: Binned, label, params: Params, n_trees, base_margin, want_detail=False):
    """n_trees iterations from a constant base margin; returns (trees, margin)."""
    margin = np.full(b.n, base_margin, np.float32)
    trees = []
    for t in range(n_trees):
        trees.append(train_tree(b, label, margin, params, iteration=t, want_detail=want_detail))
    return trees, margin


def _concat(trees):
    nodes = np.concatenate([t.nodes if hasattr(t, "nodes") else t for t in trees])
    offs = np.zeros(len(trees) + 1, np.int64)
    for i, t in enumerate(trees):
        offs[i + 1] = offs[i] + len(t.nodes if hasattr(t, "nodes") else t)
    return nodes, offs


def predict_binned(b: Binned, trees, base):
    nodes, offs = _concat(trees)
    out = np.empty(b.n, np.float32)
    s = b.struct()
    lib().orc_predict_binned(C.byref(s), _p(nodes), _p(offs), len(trees), float(base), _p(out))
    return out


def predict_raw_dense(X, trees, base):
    X = _c(X, np.float32)
    nodes, offs = _concat(trees)
    out = np.empty(len(X), np.float32)
    lib().orc_predict_raw_dense(_p(X), len(X), X.shape[1], _p(nodes), _p(offs), len(trees),
                                float(base), _p(out))
    return out


def predict_raw_csr(indptr, indices, values, trees, base):
    indptr, indices, values = _c(indptr, np.int64), _c(indices, np.int32), _c(values, np.float32)
    nodes, offs = _concat(trees)
    n = len(indptr) - 1
    out = np.empty(n, np.float32)
    lib().orc_predict_raw_csr(_p(indptr), _p(indices), _p(values), n, _p(nodes), _p(offs),
                              len(trees), float(base), _p(out))
    return out
