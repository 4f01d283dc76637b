"""Oracle pins: the exp used by the logistic loss, Philox, and the gradients
of Eq. 4-5.  CPU only."""
import math

import numpy as np
import pytest


def ulp_diff(a, b):
    ia = np.frombuffer(np.float64(a).tobytes(), np.int64)[0]
    ib = np.frombuffer(np.float64(b).tobytes(), np.int64)[0]
    return abs(int(ia) - int(ib))


def test_exp_close_to_libm(orc):
    rng = np.random.default_rng(11)
    xs = np.concatenate([rng.uniform(-708, 708, 20000), rng.uniform(-40, 40, 20000),
                         rng.uniform(-1e-3, 1e-3, 2000), [0.0, -0.0, 1.0, -1.0, 708.0, -708.0,
                                                           0.5 * math.log(2), -0.5 * math.log(2)]])
    worst = max(ulp_diff(orc.exp(float(x)), math.exp(float(x))) for x in xs)
    assert worst <= 2, worst


def test_exp_special_values(orc):
    assert orc.exp(0.0) == 1.0
    assert orc.exp(800.0) == math.inf
    assert orc.exp(-800.0) == 0.0
    assert math.isnan(orc.exp(math.nan))


@pytest.mark.parametrize("row,it,seed", [(1, 0, 0), (5, 0, 0), (123456789, 7, 42),
                                         (2**40 + 3, 99, 2**63 + 5)])
def test_philox_matches_numpy(orc, row, it, seed):
    # numpy's Philox bit generator is Philox4x64-10; it increments the
    # counter before producing its first block
    bg = np.random.Philox(counter=np.array([row - 1, it, 0, 0], np.uint64),
                          key=np.array([seed, 0], np.uint64))
    ref = bg.random_raw(4)
    out = orc.philox4x64_10([row, it, 0, 0], [seed, 0])
    assert (ref == out).all()


def test_philox_counter_zero_matches_numpy(orc):
    # counter (0, it) = numpy counter (2^64-1, it-1) incremented with carry
    bg = np.random.Philox(counter=np.array([2**64 - 1, 2, 0, 0], np.uint64),
                          key=np.array([9, 0], np.uint64))
    assert (bg.random_raw(4) == orc.philox4x64_10([0, 3, 0, 0], [9, 0])).all()


def test_logistic_gradient_closed_form_at_zero(orc):
    # sigmoid(0) = 1/2, so g = 1/2 - y and h = 1/4 exactly
    gp = orc.gradients(orc.LOSS_LOGISTIC, np.zeros(3, np.float32),
                       np.array([0, 1, 0.25], np.float32))
    assert gp.tolist() == [[0.5, 0.25], [-0.5, 0.25], [0.25, 0.25]]


def test_logistic_gradient_against_libm(orc):
    rng = np.random.default_rng(3)
    z = rng.normal(0, 6, 5000).astype(np.float32)
    y = (rng.random(5000) < 0.5).astype(np.float32)
    gp = orc.gradients(orc.LOSS_LOGISTIC, z, y)
    s = 1.0 / (1.0 + np.exp(-z.astype(np.float64)))
    g_ref = (s - y).astype(np.float32)
    h_ref = np.maximum(s * (1 - s), 1e-16).astype(np.float32)
    # float32 outputs of a double computation: at most 1 ulp apart
    assert np.all(np.abs(gp[:, 0].view(np.int32) - g_ref.view(np.int32)) <= 1)
    assert np.all(np.abs(gp[:, 1].view(np.int32) - h_ref.view(np.int32)) <= 1)


def test_logistic_hessian_floor(orc):
    gp = orc.gradients(orc.LOSS_LOGISTIC, np.array([60.0, -60.0], np.float32),
                       np.array([1, 0], np.float32))
    assert gp[0, 1] == np.float32(1e-16) and gp[1, 1] == np.float32(1e-16)


def test_squared_gradient_exact(orc):
    rng = np.random.default_rng(4)
    z = rng.normal(size=1000).astype(np.float32)
    y = rng.normal(size=1000).astype(np.float32)
    gp = orc.gradients(orc.LOSS_SQUARED, z, y)
    assert (gp[:, 0] == (z.astype(np.float64) - y).astype(np.float32)).all()
    assert (gp[:, 1] == 1.0).all()


def test_weighted_gradients(orc):
    z = np.array([0.0, 0.0], np.float32)
    y = np.array([1.0, 0.0], np.float32)
    gp = orc.gradients(orc.LOSS_LOGISTIC, z, y, np.array([2.0, 0.5], np.float32))
    assert gp.tolist() == [[-1.0, 0.5], [0.25, 0.125]]
