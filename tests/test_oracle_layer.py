"""Pins of the oracle's pruning-layer selection (Sec. 3.3.2): the per-sample
attention mass A_l^(i) and the average rank R_l, checked against closed forms,
a hand-worked example, a library ranking routine and invariants."""
import math

import numpy as np
import pytest
from scipy.stats import rankdata

from oracle import avtp_oracle as O
from paper_2608_26806_amd.workloads import build_layout, make_workload


def test_layer_attention_is_the_sum_of_image_sums():
    lay = build_layout([[6, 4, 9], [], [5]], 2, 3, 50)
    img_sum = np.array([3.0, 1.0, 2.0, 7.0], dtype=np.float32)   # integers: exact sums
    A = O.layer_attention(lay, img_sum)
    assert A.tolist() == [6.0, 0.0, 7.0]                            # a sample without images: 0


def test_layer_attention_equals_sum_of_token_scores():
    # A_l^(i) = sum over the sample's visual tokens of Attention(l, v_j): with the
    # per-token score s_j, the sum of the image sums is the sum of the s_j
    wl = make_workload(1, payload=False)
    lay = wl.layout
    s, isum, _, _ = O.attn_scores(lay, wl.q_text, wl.k, wl.Hq, wl.Hkv, wl.softmax_scale, "fp32",
                                  exact_dot=True)
    vis = lay.visual_mask()
    A = O.layer_attention(lay, isum)
    direct = math.fsum(float(x) for x in s[vis])
    assert A.shape == (1,)
    assert A[0] == pytest.approx(direct, rel=1e-12)


def test_hand_worked_example():
    # L = 4 layers, N = 3 samples, worked by hand:
    #   sample 0: 3, 3, 0, -1   -> layers 0 and 1 tie; the lower index ranks first
    #   sample 1: 1, 5, 5, -0.0 -> 5 = 5 again; -0.0 is the smallest here
    #   sample 2: 2, NaN, 2, 0  -> NaN ranks last
    A = np.array([[3.0, 1.0, 2.0],
                  [3.0, 5.0, np.nan],
                  [0.0, 5.0, 2.0],
                  [-1.0, -0.0, 0.0]])
    want = np.array([[1, 3, 1],
                     [2, 1, 4],
                     [3, 2, 2],
                     [4, 4, 3]])
    assert np.array_equal(O.layer_ranks(A), want)
    rank_sum, R, sel = O.layer_select(A, 2)
    assert rank_sum.tolist() == [5, 7, 7, 11]
    assert R.tolist() == pytest.approx([5 / 3, 7 / 3, 7 / 3, 11 / 3])
    assert sel == [0, 1]                 # layers 1 and 2 tie at 7: the lower index is chosen
    assert O.layer_select(A, 3)[2] == [0, 1, 2]


def test_ranks_match_ordinal_rankdata():
    rng = np.random.default_rng(7)
    A = rng.integers(0, 5, size=(9, 40)).astype(np.float64)      # many ties
    A[rng.random(A.shape) < 0.05] = np.nan
    ranks = O.layer_ranks(A)
    for i in range(A.shape[1]):
        col = np.where(np.isnan(A[:, i]), -np.inf, A[:, i])
        # ordinal: equal values ranked in order of appearance (lower layer first)
        assert np.array_equal(ranks[:, i], rankdata(-col, method="ordinal").astype(np.int64))


def test_rank_invariants():
    rng = np.random.default_rng(11)
    L, N = 12, 25
    A = rng.standard_normal((L, N))
    ranks = O.layer_ranks(A)
    for i in range(N):
        assert sorted(ranks[:, i].tolist()) == list(range(1, L + 1))
    rank_sum, _, _ = O.layer_select(A, 3)
    assert rank_sum.sum() == N * L * (L + 1) // 2
    perm = rng.permutation(N)                                    # sample order is irrelevant
    assert np.array_equal(O.layer_select(A[:, perm], 3)[0], rank_sum)
    dec = np.tile(-np.arange(L, dtype=np.float64)[:, None], (1, N))   # A falls with the layer
    assert np.array_equal(O.layer_ranks(dec), np.tile(np.arange(1, L + 1)[:, None], (1, N)))
    eq = np.ones((L, N))                                         # all equal: layer order
    rs, _, sel = O.layer_select(eq, 4)
    assert rs.tolist() == [N * (l + 1) for l in range(L)]
    assert sel == [0, 1, 2, 3]


def test_selection_prefers_highest_attention():
    # one layer dominates every sample, one is always last
    rng = np.random.default_rng(3)
    A = rng.random((6, 10))
    A[4] += 10.0
    A[2] -= 10.0
    rank_sum, _, sel = O.layer_select(A, 1)
    assert sel == [4] and rank_sum[4] == 10 and rank_sum[2] == 60
    assert 2 not in O.layer_select(A, 5)[2]
