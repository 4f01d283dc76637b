"""gbt_build_hist_noalloc (the histogram call for callers that cannot
allocate device memory) against gbt_build_hist on the same inputs, bit for
bit, over calls in a row that share the static scratch: a large call, then
smaller ones, then one whose plan must be cut into fewer chunks to fit, and
one too large for the scratch, which must be refused."""
import numpy as np
import pytest

from oracle import oracle as orc
from tests.gpu_helpers import oracle_quantize, same_bits, small_csr

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


def dense(seed, n, m, missing):
    rng = np.random.default_rng(seed)
    X = rng.random((n, m), dtype=np.float32)
    X[rng.random(X.shape) < missing] = np.nan
    return X


def both(gbt, ctx, mx, page, q, rows, build, sub=(), parent=None, slots=None):
    """Histograms of `build` (+ `sub`) from both entry points."""
    tb = mx.info().total_bins
    out = []
    for noalloc in (False, True):
        h = torch.full((slots, tb, 2), 77, dtype=torch.int64, device="cuda")
        gbt.gbt_build_hist(ctx, mx, page, q, rows, build, sub=sub, parent_hist=parent, hist=h, noalloc=noalloc)
        out.append(h.cpu().numpy())
    return out


def test_noalloc_matches_build_hist_on_calls_in_a_row(gbt, ctx):
    rng = np.random.default_rng(90)
    # call 1: 400,000 rows x 50 features (one root of 400,000 rows, then a
    # parent / child / sibling triple)
    n, m = 400_000, 50
    X = dense(91, n, m, 0.2)
    mx = gbt.gbt_quantize(ctx, X, max_bin=256)
    page = torch.from_numpy(mx.page(0).view(np.int32)).cuda()
    q = torch.from_numpy(rng.integers(-2**40, 2**40, size=(n, 2)).astype(np.int64)).cuda()
    a, b = both(gbt, ctx, mx, page, q, None, [(0, 0, n)], slots=1)
    assert same_bits(a, b)
    parent = torch.from_numpy(a).cuda()
    perm = torch.from_numpy(np.sort(rng.permutation(n)[: n // 3]).astype(np.int32)).cuda()
    a, b = both(gbt, ctx, mx, page, q, perm, [(1, 0, n // 3)], sub=[(0, 1, 2)], parent=parent, slots=3)
    assert same_bits(a, b)
    # call 2, right after: a smaller matrix and input (stale scratch from
    # call 1 must not leak into it)
    n2, m2 = 5003, 13
    X2 = dense(92, n2, m2, 0.1)
    mx2 = gbt.gbt_quantize(ctx, X2, max_bin=64)
    page2 = torch.from_numpy(mx2.page(0).view(np.int32)).cuda()
    q2np = rng.integers(-2**40, 2**40, size=(n2, 2)).astype(np.int64)
    q2 = torch.from_numpy(q2np).cuda()
    rows2 = rng.permutation(n2).astype(np.int32)
    segs = [(0, 0, 1000), (1, 1000, 1001), (2, 1001, 1001), (3, 1001, n2)]
    a, b = both(gbt, ctx, mx2, page2, q2, torch.from_numpy(rows2).cuda(), segs, slots=4)
    assert same_bits(a, b)
    _, b2, _, _ = oracle_quantize(X2, 64)
    for slot, lo, hi in segs:
        assert same_bits(b[slot], orc.build_hist(b2, rows2[lo:hi], q2np))
    mx.free()
    mx2.free()


def test_noalloc_cuts_chunks_to_fit_and_refuses_what_cannot(gbt, ctx):
    # wide sparse rows with up to 128 bins per feature: about 4 MiB of
    # histogram per node, so only about 16 chunk partials fit the 64 MiB
    # scratch, fewer than gbt_build_hist's usual chunking makes
    rng = np.random.default_rng(93)
    data, _ = small_csr(60_000, 2000, 0.01, 94)
    mx = gbt.gbt_quantize(ctx, data, max_bin=128)
    tb = mx.info().total_bins
    assert tb * 16 > (3 << 20)
    n = mx.info().n_rows
    page = torch.from_numpy(mx.page(0).view(np.int32)).cuda()
    qnp = rng.integers(-2**40, 2**40, size=(n, 2)).astype(np.int64)
    q = torch.from_numpy(qnp).cuda()
    # one node of every row, in fewer chunks than gbt_build_hist takes
    a, b = both(gbt, ctx, mx, page, q, None, [(0, 0, n)], slots=1)
    assert same_bits(a, b)
    # 12 nodes of 5000 rows: one chunk each
    perm = rng.permutation(n).astype(np.int32)
    rows = torch.from_numpy(perm).cuda()
    segs = [(k, 5000 * k, 5000 * (k + 1)) for k in range(12)]
    a, b = both(gbt, ctx, mx, page, q, rows, segs, slots=12)
    assert same_bits(a, b)
    _, binned, _, _ = oracle_quantize(data, 128)
    assert same_bits(b[5], orc.build_hist(binned, perm[25_000:30_000], qnp))
    # 40 non-empty nodes cannot fit: a clear error, nothing written
    segs = [(k, 1500 * k, 1500 * (k + 1)) for k in range(40)]
    h = torch.zeros((40, tb, 2), dtype=torch.int64, device="cuda")
    with pytest.raises(gbt.GbtError, match="static scratch"):
        gbt.gbt_build_hist(ctx, mx, page, q, rows, segs, hist=h, noalloc=True)
    assert not h.any().item()
    # and the scratch still serves a smaller call afterwards
    a, b = both(gbt, ctx, mx, page, q, rows, segs[:3], slots=3)
    assert same_bits(a, b)
    mx.free()
