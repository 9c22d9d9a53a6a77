"""GPU parity of the pruning-layer selection calls (Sec. 3.3.2) against the
oracle.

avtp_layer_attention: the float64 sum in image order, rounded once, against
the exactly rounded sum (math.fsum) of the same float32 image sums: within
2 ulp, and bit-exact where the sums are exact (integer-valued inputs).
avtp_layer_select: rank sums and the selected layers are integers decided on
the same float32 table on both sides, so they must match bit for bit.
"""
import numpy as np
import pytest
import torch

from gpu_util import TOL, need_gpu, say, to_dev
from oracle import avtp_oracle as O
from paper_2608_26806_amd import avtp as A
from paper_2608_26806_amd.workloads import build_layout, make_workload

pytestmark = pytest.mark.gpu

ULP2 = 2.0 ** -22        # 2 ulp of float32, relative


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    need_gpu()
    A.lib()


LAYOUTS = {
    "mixed": ([[6, 4, 9], [], [5], [3] * 40], 2, 3),
    "one_seq_many_images": ([[2] * 256], 1, 4),
    "no_images": ([[], []], 0, 5),
}


@pytest.mark.parametrize("name", sorted(LAYOUTS))
def test_layer_attention_matches_oracle(name):
    imgs, pre, tail = LAYOUTS[name]
    lay = build_layout(imgs, pre, tail, 50)
    say(f"layer_attention layout={name} B={lay.B} n_img={lay.n_img}")
    dl = A.DeviceLayout(lay)
    rng = np.random.default_rng(5)
    n = max(1, lay.n_img)
    for kind in ("integer", "lognormal"):
        if kind == "integer":
            s = rng.integers(0, 1000, size=n).astype(np.float32)
        else:
            s = np.exp(rng.normal(0.0, 3.0, size=n)).astype(np.float32)
        got = A.layer_attention(dl, torch.from_numpy(s).cuda()).cpu().numpy()
        ref = O.layer_attention(lay, s[: lay.n_img])
        assert got.shape == ref.shape
        if kind == "integer":
            assert np.array_equal(got.astype(np.float64), ref), (got, ref)
        else:
            np.testing.assert_allclose(got.astype(np.float64), ref, rtol=ULP2, atol=0.0)


def test_layer_attention_from_attention_scores():
    # the per-sample attention of one layer, from that layer's own image sums
    wl = make_workload(1, payload=False)
    lay = wl.layout
    dl = A.DeviceLayout(lay)
    say("layer_attention from avtp_score, config 1")
    _, isum_g = A.score_attn(dl, to_dev(wl.q_text, "fp32"), to_dev(wl.k, "fp32"), wl.softmax_scale)
    got = A.layer_attention(dl, isum_g).cpu().numpy().astype(np.float64)
    # same input on both sides: within 2 ulp
    np.testing.assert_allclose(got, O.layer_attention(lay, isum_g.cpu().numpy()), rtol=ULP2)
    # the whole chain against the oracle's scores
    _, isum_o, _, _ = O.attn_scores(lay, wl.q_text, wl.k, wl.Hq, wl.Hkv, wl.softmax_scale, "fp32",
                                    exact_dot=True)
    np.testing.assert_allclose(got, O.layer_attention(lay, isum_o), rtol=TOL["fp32"])


def _table(L, N, seed):
    rng = np.random.default_rng(seed)
    A_ = rng.standard_normal((L, N)).astype(np.float32)
    ties = rng.random((L, N)) < 0.3
    A_[ties] = rng.integers(-2, 3, size=int(ties.sum())).astype(np.float32)   # exact ties
    A_[rng.random((L, N)) < 0.02] = np.nan
    zs = rng.random((L, N)) < 0.02
    A_[zs] = np.where(rng.random(int(zs.sum())) < 0.5, -0.0, 0.0).astype(np.float32)
    return A_


@pytest.mark.parametrize("L,N,k", [(1, 1, 1), (4, 3, 2), (36, 400, 4), (7, 1000, 7), (13, 257, 5),
                                   (1024, 5, 3), (28, 1, 28)])
def test_layer_select_matches_oracle(L, N, k):
    say(f"layer_select L={L} N={N} k={k}")
    A_ = _table(L, N, seed=L * 1000 + N)
    dA = torch.from_numpy(A_).cuda()
    rs_g, sel_g = A.layer_select(dA, k)
    rs_o, _, sel_o = O.layer_select(A_.astype(np.float64), k)
    assert np.array_equal(rs_g.cpu().numpy().astype(np.int64), rs_o)
    assert sel_g.cpu().numpy().tolist() == sel_o
    # a second call with a smaller table reuses the outputs and is exact again
    rs2, sel2 = A.layer_select(dA[: max(1, L // 2)].contiguous(), min(k, max(1, L // 2)),
                               rank_sum=rs_g.clone(), selected=sel_g.clone())
    rs2_o, _, sel2_o = O.layer_select(A_[: max(1, L // 2)].astype(np.float64), min(k, max(1, L // 2)))
    assert np.array_equal(rs2.cpu().numpy().astype(np.int64), rs2_o)
    assert sel2.cpu().numpy().tolist() == sel2_o


def test_layer_select_hand_example():
    A_ = np.array([[3.0, 1.0, 2.0],
                   [3.0, 5.0, np.nan],
                   [0.0, 5.0, 2.0],
                   [-1.0, -0.0, 0.0]], dtype=np.float32)
    rs, sel = A.layer_select(torch.from_numpy(A_).cuda(), 2)
    assert rs.cpu().numpy().tolist() == [5, 7, 7, 11]
    assert sel.cpu().numpy().tolist() == [0, 1]


def test_layer_select_max_layers_single_sample():
    L, N = 1024, 1
    A_ = _table(L, N, seed=99)
    rs, sel = A.layer_select(torch.from_numpy(A_).cuda(), 10)
    rs_o, _, sel_o = O.layer_select(A_.astype(np.float64), 10)
    assert np.array_equal(rs.cpu().numpy().astype(np.int64), rs_o)
    assert sel.cpu().numpy().tolist() == sel_o
    assert sorted(rs.cpu().numpy().tolist()) == list(range(1, L + 1))   # one sample: a permutation
