"""The binding refuses device arguments that a kernel would read out of
bounds (host memory, another dtype, a strided view, a short buffer) before
anything reaches the library: host logic, checked on the CPU with stand-in
context and matrix objects that the library never sees."""
import os
from types import SimpleNamespace

import pytest

torch = pytest.importorskip("torch")

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIB = os.path.join(ROOT, "paper_2005_09148_amd", "libgbt.so")
pytestmark = pytest.mark.skipif(not os.path.exists(LIB), reason="libgbt.so not built")


@pytest.fixture(scope="module")
def gbt():
    from paper_2005_09148_amd import gbt as g
    return g


N = 100


class FakeMatrix:
    h = None

    def info(self):
        return SimpleNamespace(n_rows=N, row_words=4, total_bins=10)


CTX = SimpleNamespace(h=None, device=0)


def good(n=N, dtype=torch.float32):
    return torch.zeros(n, dtype=dtype)


@pytest.mark.parametrize("label,margin,msg", [
    (good(), good(), "must be on cuda:0"),                 # host tensors
    (good(dtype=torch.float64), good(), "dtype"),          # float64 labels
    (good(N - 1), good(), "elements"),                     # short label
    (good(), good(2 * N)[::2], "contiguous"),              # strided margin
    (None, good(), "required"),
    ([0.0] * N, good(), "torch tensor"),
])
def test_train_tree_refuses_bad_device_arguments(gbt, label, margin, msg):
    P = gbt.make_train_params()
    for fn in (gbt.gbt_train_tree, gbt.gbt_train_tree_naive):
        with pytest.raises(ValueError, match=msg):
            fn(CTX, FakeMatrix(), label, margin, P)


def test_gradients_and_lambda_estimate_checks(gbt):
    with pytest.raises(ValueError, match="elements"):
        gbt.gbt_gradients(CTX, 0, good(), good(N + 1))
    with pytest.raises(ValueError, match="dtype"):
        gbt.gbt_gradients(CTX, 0, good(dtype=torch.float16), good())
    with pytest.raises(ValueError, match="elements"):
        gbt.gbt_gradients(CTX, 0, good(), good(), weight=good(3))
    with pytest.raises(ValueError, match="must be on cuda"):
        gbt.gbt_mvs_lambda_estimate(CTX, 0, good(), good())
    with pytest.raises(ValueError, match="elements"):
        gbt.gbt_mvs_lambda_estimate(CTX, 0, good(), good(N - 1))


def test_sample_update_predict_checks(gbt):
    with pytest.raises(ValueError, match="elements"):
        gbt.gbt_sample(CTX, FakeMatrix(), gpair=good(N))  # n pairs are 2n floats
    with pytest.raises(ValueError, match="elements"):
        gbt.gbt_sample(CTX, FakeMatrix(), margin=good(N), label=good(7))
    with pytest.raises(ValueError, match="dtype"):
        gbt.gbt_update_leaves(CTX, None, None, FakeMatrix(), good(dtype=torch.float64))


def test_build_hist_checks(gbt):
    page = torch.zeros((N, 4), dtype=torch.int32)
    q = torch.zeros((N, 2), dtype=torch.int64)
    hist = torch.zeros((2, 10, 2), dtype=torch.int64)
    with pytest.raises(ValueError, match="words"):
        gbt.gbt_build_hist(CTX, FakeMatrix(), torch.zeros((N, 3), dtype=torch.int32), q, None, [(0, 0, N)], hist=hist)
    with pytest.raises(ValueError, match="outside"):
        gbt.gbt_build_hist(CTX, FakeMatrix(), page, q, None, [(0, 0, N + 1)], hist=hist)
    with pytest.raises(ValueError, match="slot"):
        gbt.gbt_build_hist(CTX, FakeMatrix(), page, q, None, [(2, 0, N)], hist=hist)
    with pytest.raises(ValueError, match="q:"):
        gbt.gbt_build_hist(CTX, FakeMatrix(), page, q[: N // 2], None, [(0, 0, N)], hist=hist)
    with pytest.raises(ValueError, match="must be on cuda"):
        gbt.gbt_build_hist(CTX, FakeMatrix(), page, q, None, [(0, 0, N)], hist=hist)
