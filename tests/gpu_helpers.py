"""Shared helpers of the GPU parity tests: oracle-side equivalents of a
quantized matrix and comparison utilities."""
import numpy as np

from oracle import oracle as orc


def oracle_quantize(data, max_bin, sketch_max_rows=1 << 24):
    """(cuts, binned, geometry, page words) of the oracle for dense X or a CSR dict."""
    if isinstance(data, dict):
        cuts = orc.sketch_cuts_csr(data["indptr"], data["indices"], data["values"], data["m"],
                                   max_bin, sketch_max_rows)
        b = orc.bin_csr(data["indptr"], data["indices"], data["values"], data["m"], cuts)
    else:
        cuts = orc.sketch_cuts_dense(data, max_bin, sketch_max_rows)
        b = orc.bin_dense(data, cuts)
    geo = orc.ellpack_geometry(b)
    return cuts, b, geo, orc.ellpack(b, geo)


def same_bits(a, b):
    a = np.ascontiguousarray(a)
    b = np.ascontiguousarray(b)
    return a.shape == b.shape and a.dtype == b.dtype and a.tobytes() == b.tobytes()


def node_diff(gpu_nodes, orc_nodes):
    """First differing node (index, gpu, oracle) or None."""
    for i, (g, o) in enumerate(zip(gpu_nodes, orc_nodes)):
        if g.tobytes() != o.tobytes():
            return i, g, o
    return None


def small_csr(n, m, density, seed):
    rng = np.random.default_rng(seed)
    X = rng.lognormal(size=(n, m)).astype(np.float32)
    X[rng.random(X.shape) >= density] = np.nan
    rows, cols = np.nonzero(~np.isnan(X))
    indptr = np.concatenate([[0], np.cumsum(np.bincount(rows, minlength=n))]).astype(np.int64)
    return {"kind": "csr", "indptr": indptr, "indices": cols.astype(np.int32),
            "values": X[rows, cols].astype(np.float32), "m": m}, X
