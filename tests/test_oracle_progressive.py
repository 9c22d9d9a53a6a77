"""Pins of the oracle's progressive pruning across layers (Sec. 3.3.1 h^prior
bookkeeping; the Method's subsequence view of pruning): a hand-worked layout
update, invariants of the kept subsequence, and a chained two-layer run."""
import numpy as np

from oracle import avtp_oracle as O
from paper_2608_26806_amd.workloads import build_layout


def test_pruned_layout_hand_example():
    # one sequence: t0 | image 0 = tokens 1..4 | t5 | image 1 = tokens 6..8 | t9 t10
    lay = build_layout([[4, 3]], 1, 2, 50)
    assert lay.img_start.tolist() == [1, 6] and lay.text_pos.tolist() == [0, 5, 9, 10]
    keep = [0, 2, 4, 5, 6, 9, 10]          # image 0 keeps 2 and 4, image 1 keeps 6
    nxt = O.pruned_layout(lay, keep, [0, 7], [1])
    assert nxt.cu_seqlens.tolist() == [0, 7]
    assert nxt.img_start.tolist() == [1, 4]  # after t0; after t0, the 2 kept, t5
    assert nxt.img_len.tolist() == [2, 1]
    assert nxt.text_pos.tolist() == [0, 3, 5, 6]
    assert nxt.cu_img.tolist() == [0, 2] and nxt.cu_text.tolist() == [0, 4]
    assert nxt.keep_total.tolist() == [1] and nxt.N_tok == 7 and nxt.n_img == 2


def test_pruned_layout_empty_image_and_two_sequences():
    lay = build_layout([[3, 2], [2]], 1, 1, 50)
    # seq 0: t0 [1,2,3] t4 [5,6] t7 ; seq 1: t8 [9,10] t11
    keep = [0, 4, 5, 7, 8, 10, 11]        # image 0 keeps none, image 1 keeps 5, image 2 keeps 10
    nxt = O.pruned_layout(lay, keep, [0, 4, 7], [0, 0])
    assert nxt.img_len.tolist() == [0, 1, 1]
    assert nxt.img_start.tolist() == [1, 2, 5]  # the empty image sits where its tokens were
    assert nxt.text_pos.tolist() == [0, 1, 3, 4, 6]


def test_two_layer_chain_invariants():
    rng = np.random.default_rng(4)
    lay = build_layout([[40, 25, 31], [18, 50]], 3, 5, 60)
    N, hid = int(lay.cu_seqlens[-1]), 24
    h_prior = rng.standard_normal((N, hid)).astype(np.float32)
    h_cur = h_prior + 0.3 * rng.standard_normal((N, hid)).astype(np.float32)
    nxt, h_next, keep, bud, s = O.progressive_step(lay, h_cur, h_prior, "fp32", 50)
    # the next layer's layout describes exactly the kept tokens
    assert nxt.N_tok == len(keep) == h_next.shape[0]
    assert nxt.img_len.tolist() == bud.tolist()
    assert int(np.sum(bud)) == int(np.sum(lay.keep_total))
    assert np.array_equal(h_next, h_cur[keep])                 # kept rows, original order
    assert np.array_equal(h_next[nxt.text_pos], h_cur[lay.text_pos])   # text tokens all kept
    for i in range(nxt.n_img):                                  # image i's rows are its kept rows
        s0, n = int(nxt.img_start[i]), int(nxt.img_len[i])
        src = keep[s0:s0 + n]
        assert all(lay.img_start[i] <= j < lay.img_start[i] + lay.img_len[i] for j in src)
    assert nxt.keep_total.tolist() == O.keep_totals(nxt, 50).tolist()
    # second pruning layer: h_prior is the first layer's kept output
    h2 = h_next + 0.3 * rng.standard_normal(h_next.shape).astype(np.float32)
    nxt2, h_next2, keep2, bud2, _ = O.progressive_step(nxt, h2, h_next, "fp32", 50)
    assert nxt2.N_tok == len(keep2) and int(np.sum(bud2)) == int(np.sum(nxt.keep_total))
    assert np.array_equal(h_next2[nxt2.text_pos], h2[nxt.text_pos])
    # the composed map sends every surviving token back to its original position in order
    orig = np.asarray(keep)[np.asarray(keep2)]
    assert np.all(np.diff(orig[0:int(nxt2.cu_seqlens[1])]) > 0)


def test_keep_totals_hand_values():
    """Keep totals of the next layer: keep_pct % of each sequence's remaining
    visual tokens, halves rounded up (hand-computed)."""
    lay = build_layout([[45], [7], [2, 3], []], 1, 1, 0)
    # 22.5 -> 23, 3.5 -> 4, 2.5 -> 3, no visual tokens -> 0
    assert O.keep_totals(lay, 50).tolist() == [23, 4, 3, 0]
    lay = build_layout([[3], [1], [100]], 0, 1, 0)
    # 0.99 -> 1, 0.33 -> 0, 33
    assert O.keep_totals(lay, 33).tolist() == [1, 0, 33]
    assert O.keep_totals(lay, 100).tolist() == [3, 1, 100]
    assert O.keep_totals(lay, 0).tolist() == [0, 0, 0]
