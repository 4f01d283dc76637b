"""ctypes binding of libgbt.so (the C-ABI in include/gbt.h).

Argument marshalling only: every step of the boosting iteration runs in the
library's HIP kernels.  torch supplies device memory and the stream.  There
is no fallback: importing this module fails when libgbt.so is missing or does
not load.
"""
from __future__ import annotations

import ctypes as C
import os
import weakref
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libgbt.so")

GBT_OK = 0
GBT_E_INVALID = -1
GBT_E_OOM = -2
GBT_E_BUDGET = -3
GBT_E_DEVICE = -4
GBT_E_UNSUPPORTED = -5
GBT_E_IO = -6

INPUT_DENSE = 0
INPUT_CSR = 1
LOC_HOST = 0
LOC_DEVICE = 1
HOME_DEVICE = 0
HOME_PINNED_HOST = 1
HOME_DISK = 2
LOSS_LOGISTIC = 0
LOSS_SQUARED = 1
SAMPLE_MVS = 0
SAMPLE_SGB = 1
SAMPLE_GOSS = 2
NODE_PRESENT = 1
NODE_LEAF = 2
NODE_DEFAULT_LEFT = 4


class GbtError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"libgbt error {code}: {msg}")
        self.code = code


class Input(C.Structure):
    _fields_ = [("kind", C.c_int32), ("location", C.c_int32), ("n_rows", C.c_int64),
                ("n_cols", C.c_int32), ("pad0", C.c_int32), ("values", C.c_void_p),
                ("ld", C.c_int64), ("indptr", C.c_void_p), ("indices", C.c_void_p),
                ("nnz", C.c_int64)]


class QuantParams(C.Structure):
    _fields_ = [("max_bin", C.c_int32), ("page_home", C.c_int32),
                ("sketch_max_rows", C.c_int64), ("page_rows", C.c_int64), ("page_dir", C.c_char_p),
                ("sketch_summary", C.c_int32), ("pad0", C.c_int32)]


def _quant_params(max_bin, page_home, sketch_max_rows, page_rows, page_dir, sketch_summary=0):
    return QuantParams(max_bin, page_home, sketch_max_rows, page_rows,
                       None if page_dir is None else os.fsencode(page_dir), int(sketch_summary), 0)


class MatrixInfo(C.Structure):
    _fields_ = [("n_rows", C.c_int64), ("n_cols", C.c_int32), ("sparse", C.c_int32),
                ("has_missing", C.c_int32), ("symbol_bits", C.c_int32), ("stride", C.c_int32),
                ("row_words", C.c_int32), ("null_symbol", C.c_uint32), ("n_pages", C.c_int32),
                ("total_bins", C.c_int64), ("page_rows", C.c_int64), ("page_home", C.c_int32),
                ("pad0", C.c_int32)]


class TrainParams(C.Structure):
    _fields_ = [("loss", C.c_int32), ("max_depth", C.c_int32), ("eta", C.c_double),
                ("lambda_", C.c_double), ("gamma", C.c_double), ("min_child_weight", C.c_double),
                ("f", C.c_double), ("mvs_lambda", C.c_double), ("seed", C.c_uint64),
                ("iteration", C.c_uint64), ("sampler", C.c_int32), ("pad0", C.c_int32),
                ("goss_a", C.c_double)]


class Seg(C.Structure):
    _fields_ = [("node_slot", C.c_int32), ("pad0", C.c_int32), ("begin", C.c_int64),
                ("end", C.c_int64)]


class Sub(C.Structure):
    _fields_ = [("parent_slot", C.c_int32), ("built_slot", C.c_int32),
                ("target_slot", C.c_int32), ("pad0", C.c_int32)]


SPLIT_DTYPE = np.dtype([("gain", "<f8"), ("left_g", "<i8"), ("left_h", "<i8"),
                        ("right_g", "<i8"), ("right_h", "<i8"), ("feature", "<i4"),
                        ("split_bin", "<i4"), ("default_left", "<i4"), ("valid", "<i4"),
                        ("threshold", "<f4"), ("pad0", "<i4")])
SEG_DTYPE = np.dtype([("node_slot", "<i4"), ("pad0", "<i4"), ("begin", "<i8"), ("end", "<i8")])
NODE_DTYPE = np.dtype([("feature", "<i4"), ("split_bin", "<i4"), ("threshold", "<f4"),
                       ("leaf_value", "<f4"), ("gain", "<f8"), ("sum_g", "<i8"),
                       ("sum_h", "<i8"), ("n_rows", "<i4"), ("flags", "u1"),
                       ("pad", "u1", (3,))])
assert SPLIT_DTYPE.itemsize == 64 and NODE_DTYPE.itemsize == 48 and SEG_DTYPE.itemsize == 24


class Split(C.Structure):
    _fields_ = [("gain", C.c_double), ("left_g", C.c_int64), ("left_h", C.c_int64),
                ("right_g", C.c_int64), ("right_h", C.c_int64), ("feature", C.c_int32),
                ("split_bin", C.c_int32), ("default_left", C.c_int32), ("valid", C.c_int32),
                ("threshold", C.c_float), ("pad0", C.c_int32)]


class Tree(C.Structure):
    _fields_ = [("max_depth", C.c_int32), ("n_nodes", C.c_int32), ("exp_g", C.c_int32),
                ("exp_h", C.c_int32), ("nodes", C.c_void_p)]


# gbt_tree's layout, for arrays of trees built with numpy
_TREE_DTYPE = np.dtype([("max_depth", "<i4"), ("n_nodes", "<i4"), ("exp_g", "<i4"), ("exp_h", "<i4"),
                        ("nodes", "<u8")], align=True)
assert _TREE_DTYPE.itemsize == C.sizeof(Tree)


class TreeStats(C.Structure):
    _fields_ = [("n_sampled", C.c_int64), ("threshold", C.c_int64), ("exp_key", C.c_int32),
                ("hist_launches", C.c_int32), ("hist_rows", C.c_int64),
                ("hist_updates", C.c_int64), ("hist_bytes", C.c_int64), ("ms_hist", C.c_double),
                ("ms_hist_aux", C.c_double), ("ms_sample", C.c_double), ("ms_split", C.c_double),
                ("ms_margin", C.c_double), ("ms_total", C.c_double), ("h2d_bytes", C.c_double),
                ("hist_kernel", C.c_int32), ("hist_cols", C.c_int32)]


class SampleParams(C.Structure):
    _fields_ = [("f", C.c_double), ("mvs_lambda", C.c_double), ("seed", C.c_uint64),
                ("iteration", C.c_uint64), ("loss", C.c_int32), ("sampler", C.c_int32),
                ("goss_a", C.c_double)]


class SampledInfo(C.Structure):
    _fields_ = [("n_sampled", C.c_int64), ("threshold", C.c_int64), ("target", C.c_int64),
                ("exp_key", C.c_int32), ("exp_g", C.c_int32), ("exp_h", C.c_int32),
                ("is_alias", C.c_int32), ("page_d", C.c_void_p), ("rows_d", C.c_void_p),
                ("gpair_d", C.c_void_p), ("gpair_fx_d", C.c_void_p)]


# every symbol the header declares, with its signature
_vp, _i32, _i64, _u64, _f32, _f64 = (C.c_void_p, C.c_int32, C.c_int64, C.c_uint64, C.c_float,
                                     C.c_double)
SIGNATURES = {
    "gbt_abi_version": (_i32, []),
    "gbt_last_error": (C.c_char_p, []),
    "gbt_ctx_create": (_i32, [_i32, _u64, _vp, _vp]),
    "gbt_ctx_destroy": (_i32, [_vp]),
    "gbt_ctx_memory": (_i32, [_vp, _vp, _vp]),
    "gbt_ctx_set_timing": (_i32, [_vp, _i32]),
    "gbt_ctx_set_hist_kernel": (_i32, [_vp, _i32]),
    "gbt_ctx_set_compaction": (_i32, [_vp, _i32]),
    "gbt_ctx_set_stream_chunk_rows": (_i32, [_vp, _i64]),
    "gbt_mvs_lambda_estimate": (_i32, [_vp, _i32, _vp, _vp, _i64, _vp]),
    "gbt_quantize": (_i32, [_vp, _vp, _vp, _vp]),
    "gbt_quantize_begin": (_i32, [_vp, _vp, _i32, _i64, _i32, _vp]),
    "gbt_quantize_sketch_batch": (_i32, [_vp, _vp]),
    "gbt_quantize_finalize_cuts": (_i32, [_vp]),
    "gbt_quantize_encode_batch": (_i32, [_vp, _vp]),
    "gbt_quantize_end": (_i32, [_vp, _vp]),
    "gbt_quantizer_free": (_i32, [_vp]),
    "gbt_matrix_info_get": (_i32, [_vp, _vp]),
    "gbt_matrix_get_cuts": (_i32, [_vp, _vp, _vp]),
    "gbt_matrix_copy_page": (_i32, [_vp, _i32, _vp, _i64]),
    "gbt_matrix_page_rows": (_i32, [_vp, _i32, _vp, _vp]),
    "gbt_matrix_free": (_i32, [_vp]),
    "gbt_gradients": (_i32, [_vp, _i32, _vp, _vp, _vp, _i64, _vp]),
    "gbt_sample": (_i32, [_vp, _vp, _vp, _vp, _vp, _vp, _vp]),
    "gbt_sampled_info_get": (_i32, [_vp, _vp]),
    "gbt_sampled_free": (_i32, [_vp]),
    "gbt_build_hist": (_i32, [_vp, _vp, _vp, _vp, _vp, _vp, _i32, _vp, _i32, _vp, _vp]),
    "gbt_build_hist_noalloc": (_i32, [_vp, _vp, _vp, _vp, _vp, _vp, _i32, _vp, _i32, _vp, _vp]),
    "gbt_eval_splits": (_i32, [_vp, _vp, _vp, _vp, _vp, _i32, _vp, _i32, _i32, _vp]),
    "gbt_partition": (_i32, [_vp, _vp, _vp, _vp, _vp, _vp, _i32, _vp, _vp, _i64, _vp, _vp, _vp]),
    "gbt_update_leaves": (_i32, [_vp, _vp, _vp, _vp, _vp, _vp, _i64, _vp]),
    "gbt_train_tree": (_i32, [_vp, _vp, _vp, _vp, _vp, _vp, _vp]),
    "gbt_train_trees": (_i32, [_vp, _vp, _vp, _vp, _vp, _i32, _vp, _vp]),
    "gbt_train_tree_naive": (_i32, [_vp, _vp, _vp, _vp, _vp, _vp, _vp]),
    "gbt_predict": (_i32, [_vp, _vp, _i32, _vp, _vp, _f32, _vp]),
}


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run `python -m paper_2005_09148_amd.build`")
    lib = C.CDLL(LIB_PATH)
    for name, (res, args) in SIGNATURES.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    return lib


_lib = _load()


def lib():
    return _lib


def last_error() -> str:
    return _lib.gbt_last_error().decode()


def _check(code):
    if code != GBT_OK:
        raise GbtError(code, last_error())


def abi_version() -> int:
    return _lib.gbt_abi_version()


# ---------------------------------------------------------------- torch glue
def _torch():
    import torch
    return torch


def _ptr(t):
    if t is None:
        return None
    if isinstance(t, int):
        return t
    if isinstance(t, np.ndarray):
        return t.ctypes.data
    return t.data_ptr()


def _dev_args(ctx, *specs):
    """Device pointers of the tensors in specs, each (tensor, name, dtype,
    numel or None, optional), after checking that every one is a contiguous
    torch tensor of its dtype and size on the context's device: a host or
    short buffer handed to a kernel would be an out-of-bounds device access.
    The layout of every argument is checked before any device placement."""
    torch = _torch()
    for t, name, dtype, numel, optional in specs:
        if t is None:
            if optional:
                continue
            raise ValueError(f"{name}: a device tensor is required")
        if not isinstance(t, torch.Tensor):
            raise ValueError(f"{name}: expected a torch tensor, got {type(t).__name__}")
        if t.dtype != dtype:
            raise ValueError(f"{name}: dtype {t.dtype}, expected {dtype}")
        if not t.is_contiguous():
            raise ValueError(f"{name}: must be contiguous")
        if numel is not None and t.numel() != numel:
            raise ValueError(f"{name}: {t.numel()} elements, expected {numel}")
    for t, name, _, _, _ in specs:
        if t is not None and (not t.is_cuda or t.device.index != ctx.device):
            raise ValueError(f"{name}: must be on cuda:{ctx.device}, is on {t.device}")
    return [None if t is None else t.data_ptr() for t, *_ in specs]


def _dev_tensor(a, dtype, device):
    """A contiguous device tensor of `a` (numpy array or tensor)."""
    torch = _torch()
    if isinstance(a, np.ndarray):
        a = torch.from_numpy(np.ascontiguousarray(a))
    return a.to(device=device, dtype=dtype).contiguous()


class Context:
    """A libgbt context bound to one device and torch's current stream."""

    def __init__(self, device: int = 0, budget_bytes: int = 0, stream=None):
        torch = _torch()
        self.device = device
        torch.cuda.set_device(device)
        s = stream if stream is not None else torch.cuda.current_stream(device)
        self.stream = s
        h = C.c_void_p()
        _check(_lib.gbt_ctx_create(device, budget_bytes, s.cuda_stream, C.byref(h)))
        self.h = h
        # library objects made on this context, released before it
        self._owned = weakref.WeakSet()

    def _own(self, obj):
        self._owned.add(obj)

    def close(self):
        if self.h:
            for obj in list(self._owned):
                obj.free()
            _lib.gbt_ctx_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def memory(self):
        used, peak = C.c_uint64(), C.c_uint64()
        _check(_lib.gbt_ctx_memory(self.h, C.byref(used), C.byref(peak)))
        return used.value, peak.value

    def set_timing(self, level: int):
        """0 off, 1 events around the histogram kernel only, 2 every phase."""
        _check(_lib.gbt_ctx_set_timing(self.h, int(level)))

    HIST_AUTO, HIST_PLAIN, HIST_ROTATED = 0, 1, 2

    def set_hist_kernel(self, choice: int):
        """Dense histogram kernel: HIST_AUTO (by pass size), HIST_PLAIN or
        HIST_ROTATED; results are identical."""
        _check(_lib.gbt_ctx_set_hist_kernel(self.h, int(choice)))

    COMPACT_AUTO, COMPACT_STREAM, COMPACT_GATHER = 0, 1, 2

    def set_compaction(self, mode: int):
        """How the compaction reads pinned-host pages: COMPACT_STREAM (copy
        every page over the link), COMPACT_GATHER (read only the kept rows
        through the pages' device mapping) or COMPACT_AUTO; results are
        identical."""
        _check(_lib.gbt_ctx_set_compaction(self.h, int(mode)))

    def set_stream_chunk_rows(self, rows: int):
        """Rows per chunk when host or disk pages stream through the device
        (0 = the default 2^22); results are identical."""
        _check(_lib.gbt_ctx_set_stream_chunk_rows(self.h, int(rows)))

    @property
    def torch_device(self):
        return _torch().device("cuda", self.device)


# ---------------------------------------------------------------- quantization
def _make_input(data, location):
    """gbt_input for dense X (2-D float32) or CSR (indptr, indices, values, m)."""
    inp = Input()
    keep = []
    if isinstance(data, dict) and data.get("kind") == "csr":
        ip, ix, v = data["indptr"], data["indices"], data["values"]
        inp.kind = INPUT_CSR
        inp.n_rows = len(ip) - 1
        inp.n_cols = int(data["m"])
        inp.nnz = int(ip[-1] - ip[0])
        arrs = [ip, ix, v]
    else:
        X = data
        inp.kind = INPUT_DENSE
        inp.n_rows, inp.n_cols = int(X.shape[0]), int(X.shape[1])
        inp.ld = int(X.shape[1])
        arrs = [X]
    if location == LOC_HOST:
        arrs = [np.ascontiguousarray(a) for a in arrs]
    keep.extend(arrs)
    inp.location = location
    if inp.kind == INPUT_CSR:
        inp.indptr, inp.indices, inp.values = (_ptr(a) for a in arrs)
    else:
        inp.values = _ptr(arrs[0])
    return inp, keep


def dense_input(X, location=None):
    if location is None:
        location = LOC_HOST if isinstance(X, np.ndarray) else LOC_DEVICE
    if isinstance(X, np.ndarray):
        X = np.ascontiguousarray(X, dtype=np.float32)
    return _make_input(X, location)


def csr_input(indptr, indices, values, m, location=LOC_HOST):
    if location == LOC_HOST:
        d = {"kind": "csr", "indptr": np.ascontiguousarray(indptr, np.int64),
             "indices": np.ascontiguousarray(indices, np.int32),
             "values": np.ascontiguousarray(values, np.float32), "m": m}
    else:
        d = {"kind": "csr", "indptr": indptr, "indices": indices, "values": values, "m": m}
    return _make_input(d, location)


class Matrix:
    """A quantized ELLPACK matrix owned by the library."""

    def __init__(self, ctx: Context, handle):
        self.ctx = ctx
        self.h = handle
        self._info = None
        ctx._own(self)

    def free(self):
        if self.h:
            _lib.gbt_matrix_free(self.h)
            self.h = None

    def __del__(self):
        try:
            self.free()
        except Exception:
            pass

    def info(self) -> MatrixInfo:
        if self._info is None:
            inf = MatrixInfo()
            _check(_lib.gbt_matrix_info_get(self.h, C.byref(inf)))
            self._info = inf
        return self._info

    def cuts(self):
        inf = self.info()
        cp = np.zeros(inf.n_cols + 1, np.int32)
        _check(_lib.gbt_matrix_get_cuts(self.h, _ptr(cp), None))
        cv = np.zeros(max(int(cp[-1]), 1), np.float32)
        _check(_lib.gbt_matrix_get_cuts(self.h, None, _ptr(cv)))
        return cp, cv[: int(cp[-1])]

    def page_rows(self, i):
        r0, r = C.c_int64(), C.c_int64()
        _check(_lib.gbt_matrix_page_rows(self.h, i, C.byref(r0), C.byref(r)))
        return r0.value, r.value

    def page(self, i=0) -> np.ndarray:
        inf = self.info()
        _, rows = self.page_rows(i)
        out = np.zeros((rows, inf.row_words), np.uint32)
        _check(_lib.gbt_matrix_copy_page(self.h, i, _ptr(out), out.size))
        return out

    def pages(self) -> np.ndarray:
        return np.concatenate([self.page(i) for i in range(self.info().n_pages)])


def gbt_quantize(ctx: Context, data, max_bin=256, page_rows=0, page_home=HOME_DEVICE,
                 sketch_max_rows=0, page_dir=None, sketch_summary=0) -> Matrix:
    """Sec. 3.1-3.2: quantile cuts and ELLPACK pages of dense X (numpy host
    array or device tensor) or CSR (a dict kind='csr'); HOME_DISK pages live
    in files under page_dir; sketch_summary > 0: Alg. 3's merged sketch
    with summaries of at most that many entries (one batch)."""
    if isinstance(data, dict):
        loc = LOC_HOST if isinstance(data["indptr"], np.ndarray) else LOC_DEVICE
        inp, keep = csr_input(data["indptr"], data["indices"], data["values"], data["m"], loc)
    else:
        inp, keep = dense_input(data)
    qp = _quant_params(max_bin, page_home, sketch_max_rows, page_rows, page_dir, sketch_summary)
    h = C.c_void_p()
    _check(_lib.gbt_quantize(ctx.h, C.byref(inp), C.byref(qp), C.byref(h)))
    del keep
    return Matrix(ctx, h)


class Quantizer:
    """Incremental quantization (Alg. 3 sketch batches, then Alg. 5 pages)."""

    def __init__(self, ctx, n_cols, n_rows_total, max_bin=256, page_rows=0,
                 page_home=HOME_DEVICE, sketch_max_rows=0, kind=INPUT_DENSE, page_dir=None, sketch_summary=0):
        self.ctx = ctx
        qp = _quant_params(max_bin, page_home, sketch_max_rows, page_rows, page_dir, sketch_summary)
        h = C.c_void_p()
        _check(_lib.gbt_quantize_begin(ctx.h, C.byref(qp), n_cols, n_rows_total, kind,
                                       C.byref(h)))
        self.h = h
        ctx._own(self)

    def sketch(self, X):
        """One batch (Alg. 3): dense X, or CSR as a dict kind='csr'."""
        if isinstance(X, dict):
            loc = LOC_HOST if isinstance(X["indptr"], np.ndarray) else LOC_DEVICE
            inp, keep = csr_input(X["indptr"], X["indices"], X["values"], X["m"], loc)
        else:
            inp, keep = dense_input(X)
        _check(_lib.gbt_quantize_sketch_batch(self.h, C.byref(inp)))

    def finalize(self):
        _check(_lib.gbt_quantize_finalize_cuts(self.h))

    def encode(self, X):
        if isinstance(X, dict):
            loc = LOC_HOST if isinstance(X["indptr"], np.ndarray) else LOC_DEVICE
            inp, keep = csr_input(X["indptr"], X["indices"], X["values"], X["m"], loc)
        else:
            inp, keep = dense_input(X)
        _check(_lib.gbt_quantize_encode_batch(self.h, C.byref(inp)))

    def end(self) -> Matrix:
        m = C.c_void_p()
        _check(_lib.gbt_quantize_end(self.h, C.byref(m)))
        self.h = None
        return Matrix(self.ctx, m)

    def free(self):
        if getattr(self, "h", None):
            _lib.gbt_quantizer_free(self.h)
            self.h = None

    def __del__(self):
        try:
            self.free()
        except Exception:
            pass


# ---------------------------------------------------------------- iteration steps
def gbt_gradients(ctx, loss, margin, label, weight=None, out=None):
    torch = _torch()
    f32 = torch.float32
    n = margin.numel() if isinstance(margin, torch.Tensor) else 0
    if out is None and isinstance(margin, torch.Tensor):
        out = torch.empty((n, 2), dtype=f32, device=margin.device)
    m_p, y_p, w_p, o_p = _dev_args(ctx, (margin, "margin", f32, None, False), (label, "label", f32, n, False),
                                   (weight, "weight", f32, n, True), (out, "out", f32, 2 * n, False))
    _check(_lib.gbt_gradients(ctx.h, loss, m_p, y_p, w_p, n, o_p))
    return out


def gbt_mvs_lambda_estimate(ctx, loss, margin, label):
    """MVS lambda as the squared initial leaf value -G/H of every row at
    `margin` (device tensors of equal length)."""
    torch = _torch()
    n = margin.numel() if isinstance(margin, torch.Tensor) else 0
    m_p, y_p = _dev_args(ctx, (margin, "margin", torch.float32, None, False),
                         (label, "label", torch.float32, n, False))
    out = C.c_double()
    _check(_lib.gbt_mvs_lambda_estimate(ctx.h, int(loss), m_p, y_p, margin.numel(), C.byref(out)))
    return out.value


def _hip():
    hip = getattr(_hip, "lib", None)
    if hip is None:
        hip = C.CDLL("libamdhip64.so")
        hip.hipMemcpy.argtypes = [C.c_void_p, C.c_void_p, C.c_size_t, C.c_int]
        hip.hipMemcpy.restype = C.c_int
        _hip.lib = hip
    return hip


def _copy_out(dev_ptr, nbytes, dtype, shape, device):
    """A new torch tensor holding a copy of library-owned device memory."""
    torch = _torch()
    t = torch.empty(shape, dtype=dtype, device=device)
    if nbytes:
        torch.cuda.synchronize(device)
        rc = _hip().hipMemcpy(t.data_ptr(), dev_ptr, nbytes, 3)  # device to device
        if rc != 0:
            raise RuntimeError(f"hipMemcpy failed ({rc})")
    return t


@dataclass
class SampleResult:
    info: SampledInfo
    page: object      # uint32 [R, row_words] (torch, int32 view)
    rows: object      # int32 [R] global row ids (None when aliased)
    gw: object        # float64 [R, 2]
    q: object         # int64 [R, 2]


def gbt_sample(ctx, matrix: Matrix, gpair=None, margin=None, label=None, f=1.0, mvs_lambda=1.0,
               seed=0, iteration=0, loss=LOSS_LOGISTIC, keep_handle=False, sampler=SAMPLE_MVS, goss_a=0.0):
    """Alg. 7 sampling + compaction; returns copies of the sampled arrays."""
    torch = _torch()
    n = matrix.info().n_rows
    f32 = torch.float32
    g_p, m_p, y_p = _dev_args(ctx, (gpair, "gpair", f32, 2 * n, True), (margin, "margin", f32, n, True),
                              (label, "label", f32, n, True))
    sp = SampleParams(f, mvs_lambda, seed, iteration, loss, sampler, goss_a)
    h = C.c_void_p()
    _check(_lib.gbt_sample(ctx.h, matrix.h, g_p, m_p, y_p, C.byref(sp), C.byref(h)))
    try:
        inf = SampledInfo()
        _check(_lib.gbt_sampled_info_get(h, C.byref(inf)))
        R = inf.n_sampled
        rw = matrix.info().row_words
        dev = ctx.torch_device
        page = _copy_out(inf.page_d, R * rw * 4, torch.int32, (R, rw), dev)
        rows = None if inf.is_alias else _copy_out(inf.rows_d, R * 4, torch.int32, (R,), dev)
        gw = _copy_out(inf.gpair_d, R * 16, torch.float64, (R, 2), dev)
        q = _copy_out(inf.gpair_fx_d, R * 16, torch.int64, (R, 2), dev)
        info = SampledInfo.from_buffer_copy(inf)
    finally:
        _lib.gbt_sampled_free(h)
    return SampleResult(info, page, rows, gw, q)


def gbt_build_hist(ctx, matrix: Matrix, page, q, rows, build, sub=(), parent_hist=None, hist=None,
                   noalloc=False):
    """build: [(slot, begin, end)], sub: [(parent_slot, built_slot, target_slot)].
    noalloc: call gbt_build_hist_noalloc (no device allocation; the
    library's static scratch) instead of gbt_build_hist."""
    torch = _torch()
    inf = matrix.info()
    if page is None or page.dim() != 2 or page.shape[1] != inf.row_words:
        raise ValueError(f"page: expected [rows, {inf.row_words}] words")
    n_page = page.shape[0]
    if q is not None and q.numel() < 2 * n_page:
        raise ValueError(f"q: {q.numel()} elements for {n_page} page rows")
    n_idx = rows.numel() if rows is not None else n_page
    slots = [s for s, _, _ in build] + [t for _, _, t in sub]
    for s, b, e in build:
        if not (0 <= b <= e <= n_idx):
            raise ValueError(f"build segment ({s}, {b}, {e}) outside the {n_idx} rows")
    tb = inf.total_bins
    if hist is not None and slots and hist.numel() < (max(slots) + 1) * tb * 2:
        raise ValueError(f"hist: {hist.numel()} elements, slot {max(slots)} needs {(max(slots) + 1) * tb * 2}")
    if sub and parent_hist is not None and parent_hist.numel() < (max(p for p, _, _ in sub) + 1) * tb * 2:
        raise ValueError("parent_hist: too short for the parent slots")
    i32, i64 = torch.int32, torch.int64
    pg_p, q_p, r_p, h_p, ph_p = _dev_args(ctx, (page, "page", i32, None, False), (q, "q", i64, None, False),
                                          (rows, "rows", i32, None, True), (hist, "hist", i64, None, False),
                                          (parent_hist, "parent_hist", i64, None, not sub))
    bl = (Seg * max(len(build), 1))(*[Seg(s, 0, b, e) for s, b, e in build])
    sl = (Sub * max(len(sub), 1))(*[Sub(p, b, t, 0) for p, b, t in sub])
    fn = _lib.gbt_build_hist_noalloc if noalloc else _lib.gbt_build_hist
    _check(fn(ctx.h, matrix.h, pg_p, q_p, r_p, bl, len(build), sl, len(sub), ph_p, h_p))
    return hist


def make_train_params(loss=LOSS_LOGISTIC, max_depth=6, eta=0.3, lambda_=1.0, gamma=0.0,
                      min_child_weight=1.0, f=1.0, mvs_lambda=1.0, seed=0, iteration=0,
                      sampler=SAMPLE_MVS, goss_a=0.0):
    return TrainParams(loss, max_depth, eta, lambda_, gamma, min_child_weight, f, mvs_lambda,
                       seed, iteration, sampler, 0, goss_a)


def _int_range(t, name, lo, hi):
    """Checks lo <= every value < hi of an int tensor or sequence (a device
    tensor is read back: its values index device memory)."""
    torch = _torch()
    if isinstance(t, torch.Tensor):
        if t.numel() == 0:
            return
        a, b = int(t.min()), int(t.max())
    else:
        v = np.asarray(t)
        if v.size == 0:
            return
        a, b = int(v.min()), int(v.max())
    if a < lo or b >= hi:
        raise ValueError(f"{name}: values in [{a}, {b}], expected [{lo}, {hi})")


def gbt_eval_splits(ctx, matrix: Matrix, hist, node_sums, slots, params: TrainParams, e_g, e_h,
                    out=None):
    """hist: int64 device [slots, total_bins, 2]; node_sums: int64 device
    [n, 2]; slots: n histogram slots (sequence or int32 device tensor).
    Returns the n splits (SPLIT_DTYPE) on the host, or, when out (an int64
    device tensor of n * 8 words) is given, fills it and returns it."""
    torch = _torch()
    dev = ctx.torch_device
    sl = slots if isinstance(slots, torch.Tensor) else _dev_tensor(np.asarray(slots, np.int32), torch.int32, dev)
    n = sl.numel()
    tb = matrix.info().total_bins
    if hist is None or hist.numel() % (2 * tb):
        raise ValueError(f"hist: expected [slots, {tb}, 2]")
    _int_range(sl, "slots", 0, hist.numel() // (2 * tb))
    res = out if out is not None else torch.zeros((max(n, 1), SPLIT_DTYPE.itemsize // 8), dtype=torch.int64,
                                                  device=dev)
    if res.numel() < n * SPLIT_DTYPE.itemsize // 8:
        raise ValueError(f"out: {res.numel()} words for {n} splits")
    h_p, s_p, sl_p, o_p = _dev_args(ctx, (hist, "hist", torch.int64, None, False),
                                    (node_sums, "node_sums", torch.int64, 2 * n, False),
                                    (sl, "slots", torch.int32, n, False), (res, "out", torch.int64, None, False))
    _check(_lib.gbt_eval_splits(ctx.h, matrix.h, h_p, s_p, sl_p, n, C.byref(params), e_g, e_h, o_p))
    if out is not None:
        return out
    return res.cpu().numpy().view(SPLIT_DTYPE).reshape(-1)[:n]


def gbt_partition(ctx, matrix: Matrix, page, splits, segs, children, rows, position):
    """splits: n splits (SPLIT_DTYPE array, or an int64 device tensor of
    n * 8 words as gbt_eval_splits fills); segs: [(slot, begin, end)];
    children: [l0, r0, l1, r1, ...].  rows/position are int32 device tensors
    (partitioned/updated in place).  Every node array goes to the device and
    the library works from there.  Returns the child segments as a list of
    (child, begin, end); raises GbtError when the library counted malformed
    entries."""
    torch = _torch()
    dev = ctx.torch_device
    n = len(segs)
    inf = matrix.info()
    if page is None or page.dim() != 2 or page.shape[1] != inf.row_words:
        raise ValueError(f"page: expected [rows, {inf.row_words}] words")
    if isinstance(splits, torch.Tensor):
        sp = splits
    else:
        sp = _dev_tensor(np.ascontiguousarray(splits, SPLIT_DTYPE).view(np.int64), torch.int64, dev)
    sg = np.zeros(max(n, 1), SEG_DTYPE)
    for k, (slot, b, e) in enumerate(segs):
        sg[k] = (slot, 0, b, e)
    sg_d = _dev_tensor(sg.view(np.int64), torch.int64, dev)
    ch = _dev_tensor(np.ascontiguousarray(children, np.int32).reshape(-1), torch.int32, dev)
    if ch.numel() != 2 * n:
        raise ValueError(f"children: {ch.numel()} ids for {n} nodes")
    seg_out = torch.zeros(max(2 * n, 1) * SEG_DTYPE.itemsize // 8, dtype=torch.int64, device=dev)
    status = torch.zeros(1, dtype=torch.int32, device=dev)
    tmp = torch.empty_like(rows)
    _int_range(rows, "rows", 0, page.shape[0])
    pg_p, sp_p, r_p, t_p, ps_p = _dev_args(ctx, (page, "page", torch.int32, None, False),
                                           (sp, "splits", torch.int64, None, False),
                                           (rows, "rows", torch.int32, None, False),
                                           (tmp, "rows_tmp", torch.int32, rows.numel(), False),
                                           (position, "position", torch.int32, None, False))
    if sp.numel() < n * SPLIT_DTYPE.itemsize // 8:
        raise ValueError(f"splits: {sp.numel()} words for {n} splits")
    if position.numel() < page.shape[0]:
        raise ValueError(f"position: {position.numel()} entries for {page.shape[0]} page rows")
    _check(_lib.gbt_partition(ctx.h, matrix.h, pg_p, sp_p, _ptr(sg_d), _ptr(ch), n, r_p, t_p, rows.numel(),
                              ps_p, _ptr(seg_out), _ptr(status)))
    bad = int(status.item())
    if bad:
        raise GbtError(GBT_E_INVALID, f"gbt_partition: {bad} malformed segment/split entries")
    so = seg_out.cpu().numpy().view(SEG_DTYPE)[:2 * n]
    return [(int(x["node_slot"]), int(x["begin"]), int(x["end"])) for x in so]


@dataclass
class TreeOut:
    nodes: np.ndarray
    exp_g: int
    exp_h: int
    max_depth: int
    stats: TreeStats | None = None

    def as_struct(self):
        t = Tree(self.max_depth, len(self.nodes), self.exp_g, self.exp_h, self.nodes.ctypes.data)
        return t


def _label_margin(ctx, matrix, label, margin):
    torch = _torch()
    n = matrix.info().n_rows
    return _dev_args(ctx, (label, "label", torch.float32, n, False), (margin, "margin", torch.float32, n, False))


def gbt_train_tree(ctx, matrix: Matrix, label, margin, params: TrainParams, stats=True) -> TreeOut:
    y_p, m_p = _label_margin(ctx, matrix, label, margin)
    nn = (1 << (params.max_depth + 1)) - 1
    nodes = np.zeros(nn, NODE_DTYPE)
    t = Tree(params.max_depth, nn, 0, 0, nodes.ctypes.data)
    st = TreeStats() if stats else None
    _check(_lib.gbt_train_tree(ctx.h, matrix.h, y_p, m_p, C.byref(params),
                               C.byref(t), C.byref(st) if st is not None else None))
    return TreeOut(nodes, t.exp_g, t.exp_h, params.max_depth, st)


def gbt_train_trees(ctx, matrix: Matrix, label, margin, params: TrainParams, n_trees: int,
                    stats=True) -> list[TreeOut]:
    """n_trees boosting iterations from params.iteration on, in one call."""
    y_p, m_p = _label_margin(ctx, matrix, label, margin)
    if n_trees < 0:
        raise ValueError(f"n_trees {n_trees} < 0")
    nn = (1 << (params.max_depth + 1)) - 1
    # the gbt_tree array as a structured array (one numpy call per field, not
    # one ctypes object per tree); tree t's nodes are row t of one array
    nodes = np.zeros((max(n_trees, 1), nn), NODE_DTYPE)
    ts = np.zeros(max(n_trees, 1), _TREE_DTYPE)
    ts["max_depth"] = params.max_depth
    ts["n_nodes"] = nn
    ts["nodes"] = nodes.ctypes.data + np.arange(len(ts), dtype=np.uint64) * np.uint64(nn * NODE_DTYPE.itemsize)
    st = (TreeStats * max(n_trees, 1))() if stats else None
    _check(_lib.gbt_train_trees(ctx.h, matrix.h, y_p, m_p, C.byref(params), n_trees, ts.ctypes.data, st))
    eg, eh = ts["exp_g"].tolist(), ts["exp_h"].tolist()
    return [TreeOut(nodes[t], eg[t], eh[t], params.max_depth, st[t] if st is not None else None)
            for t in range(n_trees)]


def gbt_train_tree_naive(ctx, matrix: Matrix, label, margin, params: TrainParams, stats=True) -> TreeOut:
    """Alg. 6, the naive out-of-core construction (a negative baseline)."""
    y_p, m_p = _label_margin(ctx, matrix, label, margin)
    nn = (1 << (params.max_depth + 1)) - 1
    nodes = np.zeros(nn, NODE_DTYPE)
    t = Tree(params.max_depth, nn, 0, 0, nodes.ctypes.data)
    st = TreeStats() if stats else None
    _check(_lib.gbt_train_tree_naive(ctx.h, matrix.h, y_p, m_p, C.byref(params),
                                     C.byref(t), C.byref(st) if st is not None else None))
    return TreeOut(nodes, t.exp_g, t.exp_h, params.max_depth, st)


def gbt_update_leaves(ctx, tree: TreeOut, params: TrainParams, matrix: Matrix, margin, rows=None,
                      position=None):
    """Leaf values of `tree` and the margin update of every row of `matrix`.
    position (int32 device, optional): the leaf of each training row
    (entry i: row rows[i], or row i without rows), as gbt_partition leaves
    it; those rows take their leaf without traversal."""
    torch = _torch()
    n_pos = position.numel() if position is not None else 0
    if rows is not None and position is None:
        raise ValueError("rows without position")
    m_p, r_p, p_p = _dev_args(ctx, (margin, "margin", torch.float32, matrix.info().n_rows, False),
                              (rows, "rows", torch.int32, n_pos, True),
                              (position, "position", torch.int32, None, True))
    t = tree.as_struct()
    _check(_lib.gbt_update_leaves(ctx.h, C.byref(t), C.byref(params), matrix.h, r_p, p_p, n_pos, m_p))
    return tree


def gbt_predict(ctx, trees, base_margin, binned: Matrix | None = None, raw=None, out=None):
    """raw: dense device tensor or dict(kind='csr') of device tensors."""
    torch = _torch()
    arr = (Tree * max(len(trees), 1))(*[t.as_struct() for t in trees])
    if binned is not None:
        n = binned.info().n_rows
        if out is None:
            out = torch.empty(n, dtype=torch.float32, device=ctx.torch_device)
        o_p, = _dev_args(ctx, (out, "out", torch.float32, n, False))
        _check(_lib.gbt_predict(ctx.h, arr, len(trees), None, binned.h, base_margin, o_p))
        return out
    if isinstance(raw, dict):
        inp, keep = csr_input(raw["indptr"], raw["indices"], raw["values"], raw["m"], LOC_DEVICE)
    else:
        inp, keep = dense_input(raw, LOC_DEVICE)
    if out is None:
        out = torch.empty(inp.n_rows, dtype=torch.float32, device=ctx.torch_device)
    o_p, = _dev_args(ctx, (out, "out", torch.float32, inp.n_rows, False))
    _check(_lib.gbt_predict(ctx.h, arr, len(trees), C.byref(inp), None, base_margin, o_p))
    return out


def train(ctx, matrix: Matrix, label, params: TrainParams, n_trees, base_margin, margin=None):
    """n_trees boosting iterations; returns (trees, margin)."""
    torch = _torch()
    n = matrix.info().n_rows
    if margin is None:
        margin = torch.full((n,), base_margin, dtype=torch.float32, device=ctx.torch_device)
    p = TrainParams.from_buffer_copy(params)
    p.iteration = 0
    return gbt_train_trees(ctx, matrix, label, margin, p, n_trees), margin
