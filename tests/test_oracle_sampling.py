"""Oracle pins for minimal variance sampling (Sec. 2.4, Eq. 9; Sec. 3.4,
Alg. 7) and for the exact integer gradient sums.  CPU only."""
from fractions import Fraction
import math

import numpy as np
import pytest


def phi(keys, T):
    """sum_i min(1, a_i / T), exactly."""
    return sum(Fraction(1) if a >= T else Fraction(int(a), T) for a in keys)


@pytest.mark.parametrize("seed", range(12))
def test_threshold_is_least_T_with_expected_count_at_most_K(orc, seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(1, 9))
    keys = rng.integers(0, 40, n).astype(np.int64)
    if seed % 3 == 0:
        keys[: n // 2] = 0
    K = int(rng.integers(1, n + 1))
    T = orc.mvs_threshold(keys, K)
    # brute force over every candidate T with exact rationals
    brute = next(t for t in range(1, 10**6) if phi(keys, t) <= K)
    assert T == brute


def test_threshold_minimality_at_scale(orc):
    rng = np.random.default_rng(1)
    keys = (rng.exponential(size=2000) * 2**30).astype(np.int64)
    K = 200
    T = orc.mvs_threshold(keys, K)
    assert phi(keys, T) <= K < phi(keys, T - 1)


def test_all_zero_keys_give_empty_sample(orc):
    keys = np.zeros(10, np.int64)
    T = orc.mvs_threshold(keys, 3)
    assert T == 1
    assert not orc.mvs_select(keys, T, 0, 0).any()


def test_equal_keys_reduce_to_uniform_sampling(orc):
    # with every a_i equal, p_i = a/T* = K/n: plain uniform subsampling (SGB)
    n, K = 1000, 100
    keys = np.full(n, 12345, np.int64)
    T = orc.mvs_threshold(keys, K)
    assert phi(keys, T) == K
    assert Fraction(12345, T) == Fraction(K, n)


def numpy_philox_block(block, it, seed):
    # numpy's Philox increments its 256-bit counter (little-endian words)
    # before producing a block: start from (block, it, 0, 0) - 1
    c = (block + (it << 64)) - 1
    ctr = np.array([c & (2**64 - 1), c >> 64, 0, 0], np.uint64)
    return np.random.Philox(counter=ctr, key=np.array([seed, 0], np.uint64)).random_raw(4)


@pytest.mark.parametrize("off", [1000, 1001, 2])
def test_selection_uses_philox_words(orc, off):
    # row r draws word r mod 4 of the Philox block r div 4
    rng = np.random.default_rng(2)
    keys = rng.integers(0, 1000, 500).astype(np.int64)
    T, seed, it = 700, 17, 3
    keep = orc.mvs_select(keys, T, seed, it, off)
    for i in range(500):
        row = off + i
        U = int(numpy_philox_block(row // 4, it, seed)[row % 4])
        assert orc.mvs_uniform(seed, it, row) == U
        want = keys[i] >= T or U * T < int(keys[i]) * 2**64
        assert keep[i] == want


def test_inverse_probability_weights_are_unbiased(orc):
    # E[keep_i * w_i] = P(U*T < a*2^64) * T/a = ceil(a*2^64/T)/2^64 * T/a ~ 1
    rng = np.random.default_rng(3)
    gp = np.stack([rng.normal(size=3000), rng.uniform(0.05, 0.25, 3000)], 1).astype(np.float32)
    keys, _ = orc.mvs_keys(gp, 1.0)
    K = orc.mvs_target(0.1, len(keys))
    T = orc.mvs_threshold(keys, K)
    exp_g = exp_h = Fraction(0)
    for a, (g, h) in zip(keys.tolist(), gp.tolist()):
        if a == 0:
            continue
        p = Fraction(1) if a >= T else Fraction(-(-a * 2**64 // T), 2**64)
        w = orc.mvs_weight(a, T)
        exp_g += p * Fraction(w) * Fraction(g)
        exp_h += p * Fraction(w) * Fraction(h)
    tot_g = sum(Fraction(g) for g in gp[:, 0].tolist() if True)
    tot_h = sum(Fraction(h) for h in gp[:, 1].tolist())
    assert abs(float(exp_g - tot_g)) <= 1e-12 * float(np.abs(gp[:, 0]).sum())
    assert abs(float(exp_h - tot_h)) <= 1e-12 * float(gp[:, 1].sum())
    # the expected sample size is K
    assert abs(float(sum(Fraction(1) if a >= T else Fraction(-(-a * 2**64 // T), 2**64)
                         for a in keys.tolist())) - K) < 1.0


def test_monte_carlo_over_seeds(orc):
    rng = np.random.default_rng(4)
    n = 400
    gp = np.stack([rng.normal(size=n), np.full(n, 0.25)], 1).astype(np.float32)
    keys, _ = orc.mvs_keys(gp, 1.0)
    K = orc.mvs_target(0.2, n)
    T = orc.mvs_threshold(keys, K)
    w = np.array([orc.mvs_weight(a, T) if a else 0.0 for a in keys])
    totals, counts = [], []
    for s in range(2000):
        keep = orc.mvs_select(keys, T, s, 0)
        totals.append(float((gp[keep, 0].astype(np.float64) * w[keep]).sum()))
        counts.append(int(keep.sum()))
    totals = np.array(totals)
    true = float(gp[:, 0].astype(np.float64).sum())
    se = totals.std() / math.sqrt(len(totals))
    assert abs(totals.mean() - true) < 4 * se + 1e-9
    assert abs(np.mean(counts) - K) < 4 * np.std(counts) / math.sqrt(len(counts)) + 1e-9


def test_keys_scale_and_zero_gradient_rows(orc):
    gp = np.array([[0.0, 0.0], [3.0, 4.0], [-1.5, 2.0]], np.float32)
    keys, e = orc.mvs_keys(gp, 1.0)
    # r = (0, 5, 2.5); max 5 < 2^3, L = ceil(log2 3) = 2, e = 62 - 3 - 2
    assert e == 57
    assert keys.tolist() == [0, 5 * 2**57, int(2.5 * 2**57)]


def test_mvs_lambda_enters_keys(orc):
    gp = np.array([[3.0, 2.0], [0.0, 1.0]], np.float32)
    k1, e1 = orc.mvs_keys(gp, 0.0)
    k4, e4 = orc.mvs_keys(gp, 4.0)
    # lambda=0: r=(3,0); lambda=4: r=(5,2)
    assert k1[1] == 0 and k1[0] == 3 * 2**e1
    assert k4.tolist() == [5 * 2**e4, 2 * 2**e4]


def test_fixed_point_bounds_and_error(orc):
    rng = np.random.default_rng(6)
    for R in [1, 2, 3, 1000, 4097]:
        gw = np.stack([rng.normal(size=R) * 1e3, rng.uniform(0, 1, R)], 1)
        q, eg, eh = orc.fixed_point(gw)
        L = math.ceil(math.log2(R)) if R > 1 else 0
        assert np.abs(q[:, 0]).max() <= 2 ** (62 - L)
        assert np.abs(q[:, 1]).max() <= 2 ** (62 - L)
        # any subset sum stays below 2^62
        assert abs(int(q[:, 0].astype(object).sum())) < 2**62
        assert int(q[:, 1].astype(object).sum()) < 2**62
        # |G_fx - G_exact| <= R * 2^-(e+1)
        G_fx = Fraction(int(q[:, 0].astype(object).sum()), 2**eg) if eg >= 0 else None
        G_ex = sum(Fraction(x) for x in gw[:, 0].tolist())
        assert abs(G_fx - G_ex) <= Fraction(R, 2 ** (eg + 1))
        # the exponent is maximal: doubling it would overflow the bound
        M = np.abs(gw[:, 0]).max()
        assert M * 2.0 ** (eg + 1) >= 2 ** (62 - L)


def test_fixed_point_zero_input(orc):
    q, eg, eh = orc.fixed_point(np.zeros((4, 2)))
    assert (q == 0).all() and eg == 60 and eh == 60


# ---------------------------------------------------------------- SGB and GOSS
# Sec. 2.3.  Each random draw is the row's Philox word (the MVS stream),
# compared with floor(p 2^64) for p < 1; the thresholds below are computed
# with exact rationals, independently of the oracle's floating-point ldexp.
def draw_limit(p):
    return math.floor(Fraction(p) * 2**64)


@pytest.mark.parametrize("f,off", [(0.5, 0), (0.3, 1001), (0.07, 6)])
def test_sgb_keeps_rows_whose_word_is_below_f(orc, f, off):
    seed, it = 21, 4
    keep = orc.sgb_select(400, f, seed, it, off)
    lim = draw_limit(f)
    for i in range(400):
        row = off + i
        U = int(numpy_philox_block(row // 4, it, seed)[row % 4])
        assert keep[i] == (U < lim)


def test_sgb_fraction_is_close_to_f(orc):
    keep = orc.sgb_select(200_000, 0.3, 5, 0)
    # Binomial(n, 0.3): 6 standard deviations
    assert abs(keep.mean() - 0.3) < 6 * math.sqrt(0.3 * 0.7 / 200_000)


@pytest.mark.parametrize("seed", range(6))
def test_goss_top_threshold_is_the_a_th_largest_key(orc, seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(1, 60))
    keys = rng.integers(0, 12, n).astype(np.int64)  # many ties
    for A in range(0, n + 1):
        t = orc.goss_top_threshold(keys, A)
        if A == 0:
            assert t == 2**63 - 1
            continue
        assert t == np.sort(keys)[::-1][A - 1]
        # at least A rows at or above it, fewer than A strictly above it
        assert (keys >= t).sum() >= A > (keys > t).sum()


@pytest.mark.parametrize("f,n,K", [
    (0.25, 10, 2),    # 2.5 rounds to even (half-up would give 3)
    (0.75, 10, 8),    # 7.5 rounds to even (floor would give 7)
    (0.1, 35, 4),     # f n is 3.5 in double: to even, up
    (0.1, 25, 2),     # 2.5: to even, down
    (0.29, 10, 3),    # 2.9 to nearest (floor would give 2)
    (0.5, 3, 2),      # 1.5 to even, up
    (0.05, 10, 1),    # 0.5 rounds to 0, clamped to one row
    (1e-9, 10, 1),    # far below one row: clamped
    (1.0, 7, 7),      # every row
    (0.1, 200_000_000, 20_000_000),  # the out-of-core workload's target
])
def test_mvs_target_is_clamped_round_half_even(orc, f, n, K):
    """K = max(1, rint(f n)) with IEEE round-half-to-even (the sample-size
    reading of Eq. 9); hand-computed values that a floor, a round-half-up or
    an unclamped rule would each get wrong."""
    assert orc.mvs_target(f, n) == K


def test_goss_top_count_rounds(orc):
    assert orc.goss_top_count(0.1, 1000) == 100
    assert orc.goss_top_count(0.0, 1000) == 0
    assert orc.goss_top_count(0.25, 10) == 2  # rint(2.5) to even
    assert orc.goss_top_count(1.0, 7) == 7


@pytest.mark.parametrize("off", [0, 3])
def test_goss_selection_and_weights(orc, off):
    rng = np.random.default_rng(7)
    keys = rng.integers(0, 1000, 500).astype(np.int64)
    a, b, seed, it = 0.1, 0.2, 9, 2
    A = orc.goss_top_count(a, len(keys))
    t = orc.goss_top_threshold(keys, A)
    keep = orc.goss_select(keys, t, a, b, seed, it, off)
    lim = draw_limit(b / (1.0 - a))
    for i in range(len(keys)):
        row = off + i
        U = int(numpy_philox_block(row // 4, it, seed)[row % 4])
        assert keep[i] == (keys[i] >= t or U < lim)
        w = orc.goss_weight(keys[i], t, a, b)
        assert w == (1.0 if keys[i] >= t else (1.0 - a) / b)


def test_goss_rest_weights_are_unbiased(orc):
    # E[keep_i * w_i] over the draw, for a row outside the top set:
    # floor(p 2^64) / 2^64 * (1 - a) / b, with p = b / (1 - a)
    for a, b in [(0.1, 0.2), (0.05, 0.05), (0.2, 0.8)]:
        p = b / (1.0 - a)
        e = Fraction(draw_limit(p), 2**64) * Fraction((1.0 - a) / b) if p < 1 else Fraction((1.0 - a) / b)
        assert abs(e - 1) < Fraction(1, 2**50)


def test_goss_keys_are_gradient_magnitudes(orc):
    # the top set ranks rows by |g| alone (the MVS lambda does not enter):
    # rows with large hessians but small gradients stay out of it
    n = 64
    g = np.linspace(-1.0, 1.0, n).astype(np.float32)
    h = np.where(np.arange(n) % 2 == 0, 50.0, 0.01).astype(np.float32)
    gp = np.stack([g, h], 1).astype(np.float32)
    keys, _ = orc.mvs_keys(gp, 0.0)
    A = 10
    t = orc.goss_top_threshold(keys, A)
    top = set(np.nonzero(keys >= t)[0].tolist())
    assert top == set(np.argsort(-np.abs(g.astype(np.float64)), kind="stable")[:A].tolist())


@pytest.mark.parametrize("sampler", [1, 2])
def test_training_with_sgb_and_goss(orc, sampler):
    # a whole iteration samples as the selection functions say, and the
    # training rows are the kept rows in ascending order
    rng = np.random.default_rng(11)
    X = rng.normal(size=(3000, 5)).astype(np.float32)
    y = (X[:, 0] + 0.3 * rng.normal(size=3000) > 0).astype(np.float32)
    b = orc.bin_dense(X, orc.sketch_cuts_dense(X, 32))
    P = orc.Params(loss=orc.LOSS_LOGISTIC, max_depth=4, eta=0.3, f=0.3, seed=3, sampler=sampler, goss_a=0.1)
    margin = np.zeros(3000, np.float32)
    r = orc.train_tree(b, y, margin, P, iteration=1, want_detail=True)
    gp = r.gpair
    if sampler == 1:
        want = orc.sgb_select(3000, 0.3, 3, 1)
    else:
        keys, _ = orc.mvs_keys(gp, 0.0)
        t = orc.goss_top_threshold(keys, orc.goss_top_count(0.1, 3000))
        want = orc.goss_select(keys, t, 0.1, 0.3 - 0.1, 3, 1)
        assert r.info.T == t
    assert np.array_equal(r.sel, np.nonzero(want)[0])
    assert (margin != 0).any()


# ------------------------------------------------- MVS lambda estimated from data
@pytest.mark.parametrize("n", [1, 7, 1000])
def test_lambda_estimate_squared_loss_is_squared_mean_label(orc, n):
    # squared error at margin 0: g = -y, h = 1, so the initial Newton leaf is
    # mean(y) and lambda = mean(y)^2; labels are multiples of 1/8, so the
    # fixed-point sums are exact and the result is the correctly rounded
    # (sum y / n)^2
    rng = np.random.default_rng(n)
    y = (rng.integers(-16, 40, n) / 8.0).astype(np.float32)
    lam = orc.mvs_lambda_estimate(orc.LOSS_SQUARED, np.zeros(n, np.float32), y)
    w0 = float(np.sum(y.astype(np.float64))) / n
    assert lam == w0 * w0


def test_lambda_estimate_logistic_at_zero_margin(orc):
    # logistic at margin 0: p = 1/2, g = 1/2 - y, h = 1/4, so the leaf is
    # -4 * sum(1/2 - y) / n
    rng = np.random.default_rng(5)
    y = (rng.random(777) < 0.3).astype(np.float32)
    lam = orc.mvs_lambda_estimate(orc.LOSS_LOGISTIC, np.zeros(777, np.float32), y)
    w0 = -float(np.sum(0.5 - y.astype(np.float64))) / (0.25 * 777)
    assert lam == w0 * w0
    assert lam > 0


def test_lambda_estimate_general_margins_and_degenerate_cases(orc):
    # at arbitrary margins the estimate is (sum g / sum h)^2 of the float32
    # gradients up to the fixed-point rounding (relative 2^-40 here)
    rng = np.random.default_rng(9)
    n = 5000
    m = rng.normal(0.0, 1.5, n).astype(np.float32)
    y = (rng.random(n) < 0.8).astype(np.float32)
    gp = orc.gradients(orc.LOSS_LOGISTIC, m, y).astype(np.float64)
    want = (gp[:, 0].sum() / gp[:, 1].sum()) ** 2
    assert orc.mvs_lambda_estimate(orc.LOSS_LOGISTIC, m, y) == pytest.approx(want, rel=2.0**-40)
    # a label equal to every margin gives a zero leaf; no rows give 0
    assert orc.mvs_lambda_estimate(orc.LOSS_SQUARED, y, y) == 0.0
    assert orc.mvs_lambda_estimate(orc.LOSS_SQUARED, np.zeros(0, np.float32), np.zeros(0, np.float32)) == 0.0
