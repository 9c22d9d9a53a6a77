"""Pins for the oracle's attention-to-visual-token score (CPU only).

The score follows the attention statistic of Sec. 3.3.2 (attention a layer
pays to each visual token), evaluated per token.  The paper prints no worked
example, so the oracle is pinned against: a loops-only brute force, the
textbook softmax (single text row, one head), closed forms and invariants.
"""
import math

import numpy as np
import pytest
import torch
from scipy.special import logsumexp

from oracle import avtp_oracle as O
from oracle import brute
from paper_2608_26806_amd.workloads import build_layout, make_workload, duplicate_key_rows


def _random_case(rng, images, pre, tail, Hq, Hkv, d):
    lay = build_layout([images], pre, tail, 50)
    q = rng.standard_normal((lay.T_tot, Hq, d)).astype(np.float32)
    k = rng.standard_normal((lay.N_tok, Hkv, d)).astype(np.float32)
    return lay, q, k


def _tokens(lay):
    kinds = {}
    for i, (s, n) in enumerate(zip(lay.img_start, lay.img_len)):
        for j in range(s, s + n):
            kinds[j] = ("img", i)
    for t, p in enumerate(lay.text_pos):
        kinds[int(p)] = ("text", t)
    return [kinds[j] for j in range(lay.N_tok)]


@pytest.mark.parametrize("images,pre,tail,Hq,Hkv", [
    ([3, 2], 0, 2, 1, 1),
    ([2, 3], 1, 2, 2, 1),
    ([4], 2, 1, 4, 2),
    ([1, 2, 2], 1, 1, 2, 2),
])
def test_vectorised_matches_loops(images, pre, tail, Hq, Hkv):
    rng = np.random.default_rng(7)
    lay, q, k = _random_case(rng, images, pre, tail, Hq, Hkv, 4)
    scale = 0.5
    s, isum, _, empty = O.attn_scores(lay, q, k, Hq, Hkv, scale, "fp32", exact_dot=True)
    qs = [[list(map(float, q[t, h])) for h in range(Hq)] for t in range(lay.T_tot)]
    ks = [[list(map(float, k[j, g])) for g in range(Hkv)] for j in range(lay.N_tok)]
    bs, bsum = brute.attn_scores_loops(_tokens(lay), qs, ks, Hq, Hkv, scale)
    for j in range(lay.N_tok):
        if bs[j] is None:
            assert s[j] == np.inf
        else:
            assert s[j] == pytest.approx(bs[j], rel=1e-12, abs=1e-15)
    for i in range(lay.n_img):
        assert isum[i] == pytest.approx(bsum[i], rel=1e-12)
    assert not empty


def test_single_row_single_head_is_softmax():
    """T = 1, Hq = Hkv = 1, text after the images: s_j is one softmax entry."""
    rng = np.random.default_rng(3)
    lay, q, k = _random_case(rng, [5, 7], 0, 1, 1, 1, 8)
    scale = 1.0 / math.sqrt(8)
    s, _, _, _ = O.attn_scores(lay, q, k, 1, 1, scale, "fp32")
    ref = torch.softmax(torch.from_numpy(k[:, 0, :]).double() @ torch.from_numpy(q[0, 0]).double() * scale, 0)
    vis = lay.visual_mask()
    np.testing.assert_allclose(s[vis], ref.numpy()[vis], rtol=1e-12)


def test_visual_mass_plus_text_mass_is_one():
    """With every text row after every image, |T_j| = T and the head/row mean of
    the visual attention plus that of the text attention is exactly 1."""
    rng = np.random.default_rng(11)
    lay, q, k = _random_case(rng, [6, 4, 5], 0, 4, 4, 2, 8)
    scale = 0.35
    s, _, _, _ = O.attn_scores(lay, q, k, 4, 2, scale, "fp32")
    vis = lay.visual_mask()
    # text mass from torch's causal softmax, computed independently
    text_mass = 0.0
    for h in range(4):
        kk = torch.from_numpy(k[:, h // 2, :]).double()
        for t, p in enumerate(lay.text_pos):
            row = torch.softmax(kk[: p + 1] @ torch.from_numpy(q[t, h]).double() * scale, 0)
            text_mass += float(row[torch.from_numpy(~vis[: p + 1])].sum())
    text_mass /= 4 * lay.T_tot
    assert s[vis].sum() + text_mass == pytest.approx(1.0, abs=1e-12)


def test_equal_keys_closed_form():
    """All keys equal -> each row spreads 1/(visible keys) evenly."""
    lay = build_layout([[3, 4], [2]], 2, 3, 50)
    Hq, Hkv, d = 2, 1, 4
    rng = np.random.default_rng(5)
    q = rng.standard_normal((lay.T_tot, Hq, d)).astype(np.float32)
    k = np.tile(rng.standard_normal((1, Hkv, d)).astype(np.float32), (lay.N_tok, 1, 1))
    s, isum, _, _ = O.attn_scores(lay, q, k, Hq, Hkv, 0.7, "fp32")
    for b in range(lay.B):
        s0 = int(lay.cu_seqlens[b])
        tp = lay.text_pos[lay.cu_text[b]:lay.cu_text[b + 1]]
        for i in range(lay.cu_img[b], lay.cu_img[b + 1]):
            for j in range(lay.img_start[i], lay.img_start[i] + lay.img_len[i]):
                rows = [p for p in tp if p > j]
                expect = sum(1.0 / (p - s0 + 1) for p in rows) / len(rows)
                assert s[j] == pytest.approx(expect, rel=1e-12)


def test_row_lse_matches_logsumexp():
    rng = np.random.default_rng(9)
    lay, q, k = _random_case(rng, [5, 3], 2, 3, 4, 2, 8)
    lse = O.attn_row_lse(lay, q, k, 4, 2, 0.4, "fp32")
    for h in range(4):
        for t, p in enumerate(lay.text_pos):
            z = 0.4 * (k[: p + 1, h // 2, :].astype(np.float64) @ q[t, h].astype(np.float64))
            assert lse[h, t] == pytest.approx(logsumexp(z), rel=1e-13)


def test_duplicate_keys_bit_identical_and_aligned_key_ranks_first():
    wl = make_workload(1, payload=False)
    lay = wl.layout
    s1 = int(lay.img_start[1])
    duplicate_key_rows(wl, s1 + 10, [s1 + 20, s1 + 30, s1 + 40])
    # a key aligned with every query of its group dominates the image
    qm = wl.q_text[:, :2, :].astype(np.float64).mean(axis=(0, 1))
    wl.k[s1 + 5, 0, :] = (qm / np.linalg.norm(qm) * 40.0).astype(np.float32)
    s, _, _, _ = O.attn_scores(lay, wl.q_text, wl.k, wl.Hq, wl.Hkv, wl.softmax_scale, "fp32",
                               exact_dot=True)
    assert s[s1 + 10] == s[s1 + 20] == s[s1 + 30] == s[s1 + 40]
    img = s[s1:s1 + int(lay.img_len[1])]
    assert int(np.argmax(img)) == 5


def test_interleaved_text_rows_counted():
    """A pre-image text row does not see the image that follows it."""
    lay = build_layout([[2, 2]], 1, 1, 50)   # text, img0, text, img1, text
    assert list(lay.text_pos) == [0, 3, 6]
    assert O.text_rows_after(lay, 1) == 2
    assert O.text_rows_after(lay, 4) == 1


def test_empty_text_after_image_flagged():
    lay = build_layout([[2, 2]], 1, 0, 50)   # text, img0, text, img1  (no tail)
    rng = np.random.default_rng(2)
    q = rng.standard_normal((lay.T_tot, 1, 4)).astype(np.float32)
    k = rng.standard_normal((lay.N_tok, 1, 4)).astype(np.float32)
    s, isum, _, empty = O.attn_scores(lay, q, k, 1, 1, 1.0, "fp32")
    assert empty == {1}
    assert isum[1] == 0.0 and s[4] == 0.0 and s[5] == 0.0


def test_bf16_inputs_widen_exactly():
    x = np.array([0x3F80, 0xC000, 0x0001, 0x7F7F], dtype=np.uint16)
    w = O.widen(x, "bf16")
    ref = torch.from_numpy(x.view(np.int16)).view(torch.bfloat16).double().numpy()
    np.testing.assert_array_equal(w, ref)


@pytest.mark.parametrize("case", ["config1", "interleaved_bf16_gqa"])
def test_score_one_matches_full_scores(case):
    """``attn_score_one`` (the per-token form that checks sampled tokens at full
    size) against ``attn_scores`` for every visual token, rel 1e-12.

    The interleaved case has text before every image, so the row set of a token
    (the text rows after it) differs from image to image, and 8 query heads on
    2 key heads, so a wrong head-to-group map (h % Hkv for h // G) changes every
    score.  Text and visual positions never coincide, so "after" needs no
    tie rule."""
    if case == "config1":
        wl = make_workload(1, payload=False)
        lay, q, k, Hq, Hkv, scale, dt = (wl.layout, wl.q_text, wl.k, wl.Hq, wl.Hkv,
                                         wl.softmax_scale, "fp32")
    else:
        rng = np.random.default_rng(21)
        lay = build_layout([[9, 1, 14], [5, 7]], 3, 4, 50)
        Hq, Hkv, d = 8, 2, 64
        from paper_2608_26806_amd.workloads import f32_to_bf16_bits
        q = f32_to_bf16_bits(rng.standard_normal((lay.T_tot, Hq, d)).astype(np.float32))
        k = f32_to_bf16_bits(rng.standard_normal((lay.N_tok, Hkv, d)).astype(np.float32))
        scale, dt = d ** -0.5, "bf16"
    s, _, lse, _ = O.attn_scores(lay, q, k, Hq, Hkv, scale, dt)
    vis = np.flatnonzero(lay.visual_mask())
    one = np.array([O.attn_score_one(lay, q, k, Hq, Hkv, scale, dt, lse, int(j)) for j in vis])
    np.testing.assert_allclose(one, s[vis], rtol=1e-12, atol=0.0)
    # the per-token form agrees with the loops-only brute force too (one
    # sequence at a time: the brute force takes a single sequence)
    if case == "interleaved_bf16_gqa":
        qf, kf = O.widen(q, dt), O.widen(k, dt)
        toks = _tokens(lay)
        ref = {}
        for b in range(lay.B):
            s0, s1 = int(lay.cu_seqlens[b]), int(lay.cu_seqlens[b + 1])
            t0 = int(lay.cu_text[b])
            seq = [(kind, x - t0 if kind == "text" else x) for kind, x in toks[s0:s1]]
            qs = [[list(map(float, qf[t, h])) for h in range(Hq)]
                  for t in range(t0, int(lay.cu_text[b + 1]))]
            ks = [[list(map(float, kf[j, g])) for g in range(Hkv)] for j in range(s0, s1)]
            bs, _ = brute.attn_scores_loops(seq, qs, ks, Hq, Hkv, scale)
            ref.update({s0 + p: v for p, v in enumerate(bs) if v is not None})
        np.testing.assert_allclose(one, [ref[int(j)] for j in vis], rtol=1e-12, atol=0.0)
