"""Pins for the oracle's per-image budget (Sec. 3.3.3 ratio rule, appendix clamp).

Independent checks: hand-derived examples, a float bisection and a generic QP
solver for the real quotas, an exhaustive integer search for the rounding, and
invariants (sum, bounds, monotonicity).
"""
import itertools
import math
from fractions import Fraction

import numpy as np
import pytest
from scipy.optimize import minimize

from oracle import avtp_oracle as O
from oracle import brute
from paper_2608_26806_amd.workloads import build_layout


def _one_seq(n, keep_total):
    lay = build_layout([n], 0, 1, 0)
    lay.keep_total[:] = keep_total
    return lay


def test_hand_examples():
    # n = (64, 64), K = 64, alpha = 1: quotas proportional to the image sums.
    lay = _one_seq([64, 64], 64)
    assert list(O.budget(lay, [3.0, 1.0], 1.0)) == [48, 16]
    # S = (99, 1): quota (63.36, 0.64) -> image 1 lifted to ceil(5 % of 64) = 4,
    # image 0 then takes the remaining 60 = floor(95 % of 64).
    assert list(O.budget(lay, [99.0, 1.0], 1.0)) == [60, 4]
    # alpha = 0: uniform ratio; equal images split evenly, odd unit to index 0.
    lay = _one_seq([10, 10, 10], 5)
    assert list(O.budget(lay, [5.0, 1.0, 2.0], 0.0)) == [2, 2, 1]
    # absolute floor dominates the 5 % floor for small images
    lay = _one_seq([20, 20, 200], 60)
    k = O.budget(lay, [0.0, 0.0, 10.0], 1.0, floor_abs=16)
    assert list(k) == [16, 16, 28]


def test_proportional_closed_form_when_unclamped():
    lay = _one_seq([100, 200, 300], 150)
    S = [30.0, 20.0, 50.0]
    k, q = O.budget(lay, S, 1.0, return_quota=True)
    for qi, s in zip(q, S):
        assert float(qi) == pytest.approx(150 * s / 100.0, rel=1e-7)
    assert list(k) == [45, 30, 75]


def test_raw_mode_is_literal_ratio_rule():
    """r_i = r_base + alpha (Ibar_i - Ibar_avg) with r_base = K / M."""
    n = [100, 300]
    S = [50.0, 30.0]                  # Ibar = 0.5, 0.1 ; Ibar_avg = 80 / 400 = 0.2
    lay = _one_seq(n, 100)            # r_base = 0.25
    k, q = O.budget(lay, S, 0.5, mode=O.BUDGET_RAW, return_quota=True)
    r = [0.25 + 0.5 * (0.5 - 0.2), 0.25 + 0.5 * (0.1 - 0.2)]
    for qi, ri, ni in zip(q, r, n):
        assert float(qi) == pytest.approx(ri * ni, rel=1e-7)
    assert sum(k) == 100


def _bisect_quota(W, lo, hi, K):
    """Float bisection on f(lam) = sum clamp(lam W, lo, hi) = K (independent of the walk)."""
    a, b = 0.0, 1.0
    f = lambda lam: sum(min(max(lam * w, l), h) for w, l, h in zip(W, lo, hi))
    while f(b) < K:
        b *= 2.0
    for _ in range(200):
        m = 0.5 * (a + b)
        if f(m) < K:
            a = m
        else:
            b = m
    lam = 0.5 * (a + b)
    return [min(max(lam * w, l), h) for w, l, h in zip(W, lo, hi)]


def _qp_quota(W, lo, hi, K):
    """argmin sum q^2 / W  s.t.  sum q = K, lo <= q <= hi  (generic solver)."""
    from scipy.optimize import Bounds, LinearConstraint
    w = np.asarray(W, dtype=np.float64) / max(W)
    lo_, hi_ = np.asarray(lo, float) / K, np.asarray(hi, float) / K
    x0 = np.clip(w / w.sum(), lo_, hi_)
    res = minimize(lambda x: float(np.sum(x * x / w)), x0, method="trust-constr",
                   jac=lambda x: 2 * x / w, hess=lambda x: np.diag(2 / w),
                   bounds=Bounds(lo_, hi_), constraints=[LinearConstraint(np.ones((1, len(w))), 1.0, 1.0)],
                   options={"gtol": 1e-12, "xtol": 1e-14, "maxiter": 5000})
    return res.x * K


@pytest.mark.parametrize("seed", range(12))
def test_water_level_against_bisection_and_qp(seed):
    rng = np.random.default_rng(seed)
    m = int(rng.integers(2, 7))
    n = [int(x) for x in rng.integers(20, 400, size=m)]
    S = list(rng.lognormal(0.0, 1.5, size=m))
    bounds = [O.budget_bounds(x, 50, 950, 0) for x in n]
    lo, hi = [b[0] for b in bounds], [b[1] for b in bounds]
    K = int(rng.integers(sum(lo), sum(hi) + 1))
    alpha = 2.0 if seed % 2 else 1.0
    W = O.budget_weights(n, S, K, alpha)
    q = [float(x) for x in O.water_level(W, lo, hi, K)]
    assert sum(O.water_level(W, lo, hi, K)) == K
    np.testing.assert_allclose(q, _bisect_quota(W, lo, hi, K), rtol=1e-9, atol=1e-9)
    if min(W) > 1e-3 * max(W):    # the generic solver needs a well-conditioned objective
        np.testing.assert_allclose(q, _qp_quota(W, lo, hi, K), rtol=1e-4, atol=1e-4)


def _cases():
    rng = np.random.default_rng(123)
    out = []
    for m in (1, 2, 3):
        for n in itertools.product(range(1, 9), repeat=m):
            for pattern in range(2):
                S = [1.0 + ((i * 7 + pattern * 3) % 5) for i in range(m)]
                out.append((list(n), S))
    rng.shuffle(out)
    return out[:260]


def test_rounding_is_the_integer_minimiser():
    """Largest remainder with the lowest-index tie rule equals the exhaustive
    minimiser of sum (k - q*)^2 over every feasible integer vector."""
    checked = 0
    for n, S in _cases():
        bounds = [O.budget_bounds(x, 50, 950, 1) for x in n]
        lo, hi = [b[0] for b in bounds], [b[1] for b in bounds]
        for K in range(sum(lo), sum(hi) + 1):
            lay = _one_seq(n, K)
            k, q = O.budget(lay, S, 1.0, floor_abs=1, return_quota=True)
            assert sum(k) == K
            assert all(a <= x <= b for a, x, b in zip(lo, k, hi))
            assert list(k) == brute.min_dev_integer_budget(q, lo, hi, K)
            checked += 1
    assert checked > 500


def test_ties_in_remainder_go_to_lowest_index():
    lay = _one_seq([10, 10, 10, 10], 6)
    assert list(O.budget(lay, [1.0, 1.0, 1.0, 1.0], 1.0)) == [2, 2, 1, 1]


def test_monotone_in_image_sum():
    n = [64, 64, 64]
    lay = _one_seq(n, 60)
    prev = -1
    for s0 in [0.1, 0.5, 1.0, 2.0, 4.0, 8.0, 100.0]:
        k = O.budget(lay, [s0, 1.0, 1.0], 1.0)
        assert k[0] >= prev
        prev = k[0]


@pytest.mark.parametrize("alpha", [0.0, 1.0, 2.0, 5.0])
def test_invariants_random(alpha):
    rng = np.random.default_rng(int(alpha * 10) + 1)
    for _ in range(30):
        m = int(rng.integers(1, 9))
        n = [int(x) for x in rng.integers(1, 300, size=m)]
        lay = _one_seq(n, 0)
        bounds = [O.budget_bounds(x, 50, 950, 4) for x in n]
        lo, hi = [b[0] for b in bounds], [b[1] for b in bounds]
        K = int(rng.integers(sum(lo), sum(hi) + 1))
        lay.keep_total[:] = K
        S = list(rng.exponential(1.0, size=m) * np.array(n))
        k = O.budget(lay, S, alpha, floor_abs=4)
        assert int(np.sum(k)) == K
        assert all(a <= x <= b <= nn for a, x, b, nn in zip(lo, k, hi, n))


def test_infeasible_and_degenerate():
    lay = _one_seq([10, 10], 0)
    with pytest.raises(ValueError):
        O.budget(lay, [1.0, 1.0], 1.0)            # sum lo = 2 > 0
    lay = _one_seq([10, 10], 20)
    with pytest.raises(ValueError):
        O.budget(lay, [1.0, 1.0], 1.0)            # sum hi = 18 < 20
    # all-zero importance: every image gets its token share
    lay = _one_seq([30, 10], 20)
    assert list(O.budget(lay, [0.0, 0.0], 1.0)) == [15, 5]
    # exactly at the lower / upper bound
    lay = _one_seq([40, 40], 4)
    assert list(O.budget(lay, [5.0, 1.0], 1.0)) == [2, 2]
    lay = _one_seq([40, 40], 76)
    assert list(O.budget(lay, [5.0, 1.0], 1.0)) == [38, 38]


def test_weights_quantisation_is_round_half_even_relative_to_the_largest():
    # w = (0.25, 0.75): the largest becomes 2^28, the other 2^28 / 3 = 89478485.33 -> 89478485
    W = O.budget_weights([1, 1], [1.0, 3.0], 1, 1.0)
    assert W == [89478485, 1 << 28]
    # w = (0.375, 0.625) = (3/8, 5/8): 3/5 * 2^28 = 161061273.6 -> 161061274
    W = O.budget_weights([1, 1], [3.0, 5.0], 1, 1.0)
    assert W == [161061274, 1 << 28]
    # a tiny share keeps its ratio: S = (1, 2^24) -> 2^28 / 2^24 = 16
    W = O.budget_weights([1, 1], [1.0, float(2 ** 24)], 1, 1.0)
    assert W == [16, 1 << 28]
    # zero-importance images keep weight 1 (they only fill what the others cannot)
    W = O.budget_weights([5, 5], [0.0, 2.0], 1, 1.0)
    assert W == [1, 1 << 28]


def test_raw_rule_keeps_ratios_of_large_weights():
    """A hand-derived BUDGET_RAW case with shares far above 1, where only the
    ratio of the weights decides the split (Sec. 3.3.3 ratio rule with
    r_base = K / M, clamp of the appendix).

    Four images of 64 tokens, M = 256, K = 98, alpha = 1, S = (24451, 34251, 0, 0)
    (S = 58702, Ibar_avg = S / M = 229.3046875).  The literal rule gives
        r_1 = 98/256 + (24451/64 - 229.3046875) = 153.125,  q_1 = 64 r_1 = 9800
        r_2 = 98/256 + (34251/64 - 229.3046875) = 306.25,   q_2 = 19600
        r_3 = r_4 = 98/256 - 229.3046875 = -228.921875,     q_3 = q_4 = -14651
    (shares w = q / K = 100, 200, -149.5, -149.5; sum q = K).  Images 3 and 4
    fall to their floor ceil(5 % of 64) = 4; the other 90 units are split in
    the ratio 100 : 200 of the first two, i.e. (30, 60), with 60 = floor(95 %
    of 64) just reached.  A cap on the shares (e.g. at 64) would make the two
    equal and give (45, 45)."""
    lay = _one_seq([64, 64, 64, 64], 98)
    S = [24451.0, 34251.0, 0.0, 0.0]
    W = O.budget_weights([64] * 4, S, 98, 1.0, mode=O.BUDGET_RAW)
    assert W == [1 << 27, 1 << 28, 1, 1]
    k, q = O.budget(lay, S, 1.0, mode=O.BUDGET_RAW, return_quota=True)
    assert list(k) == [30, 60, 4, 4]
    assert [float(x) for x in q] == [30.0, 60.0, 4.0, 4.0]
