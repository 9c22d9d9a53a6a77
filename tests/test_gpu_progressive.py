"""GPU parity of progressive pruning across layers (avtp_pruned_layout and the
ProgressivePruner driver) against the oracle.

The layout update is integer work and must match bit for bit.  A chained run
checks every stage of every pruning layer against the oracle given the GPU's
own inputs to that stage (scores within the variation tolerance; budgets,
kept indices, compacted rows and the next layout bit-exact), then continues
the chain with the GPU's outputs.
"""
import numpy as np
import pytest
import torch

from gpu_util import TOL, assert_rel, need_gpu, say, to_dev
from oracle import avtp_oracle as O
from paper_2608_26806_amd import avtp as A
from paper_2608_26806_amd.progressive import ProgressivePruner
from paper_2608_26806_amd.workloads import bf16_bits_to_f32, build_layout, f32_to_bf16_bits

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    need_gpu()
    A.lib()


LAYOUTS = {
    "mixed": ([[300, 1, 57], [], [129, 64, 2]], 4, 9),
    "gaps": ([[0, 5], [9000, 3], [], [50, 0, 7]], 0, 6),
    "one": ([[33]], 1, 1),
    # a sequence keeping more than the 16,384 entries the kernel searches in
    # LDS (searched in place) beside one that fits
    "long": ([[60000, 7], [500]], 2, 3),
}


def _random_keep(lay, rng):
    """Kept indices: every text token and a random subset of every image."""
    keep, cu = [], [0]
    for b in range(lay.B):
        s0, s1 = int(lay.cu_seqlens[b]), int(lay.cu_seqlens[b + 1])
        vis = np.zeros(s1 - s0, dtype=bool)
        for i in range(int(lay.cu_img[b]), int(lay.cu_img[b + 1])):
            st, n = int(lay.img_start[i]) - s0, int(lay.img_len[i])
            vis[st:st + n] = True
        take = ~vis | (rng.random(s1 - s0) < 0.3)
        keep.extend((s0 + np.flatnonzero(take)).tolist())
        cu.append(len(keep))
    return np.array(keep, np.int32), np.array(cu, np.int32)


@pytest.mark.parametrize("name", sorted(LAYOUTS))
def test_pruned_layout_matches_oracle(name):
    imgs, pre, tail = LAYOUTS[name]
    lay = build_layout(imgs, pre, tail, 50)
    say(f"pruned_layout layout={name}")
    rng = np.random.default_rng(8)
    keep, cu = _random_keep(lay, rng)
    dl = A.DeviceLayout(lay)
    got = A.pruned_layout(dl, torch.from_numpy(keep).cuda(), torch.from_numpy(cu).cuda())
    ref = O.pruned_layout(lay, keep, cu, np.zeros(lay.B, np.int32))
    for n in ("cu_seqlens", "img_start", "img_len", "cu_img", "text_pos", "cu_text"):
        assert got[n].cpu().numpy().tolist() == getattr(ref, n).tolist(), n


def _to_host(t, dtype):
    x = t.detach().cpu()
    if dtype == "bf16":
        return x.view(torch.int16).numpy().view(np.uint16)
    return x.numpy()


def _noisy(h_host, dtype, rng, sigma):
    """h + sigma N(0,1), in the storage type (bf16 bits or float32)."""
    base = bf16_bits_to_f32(h_host) if dtype == "bf16" else h_host
    x = (base + sigma * rng.standard_normal(base.shape)).astype(np.float32)
    return f32_to_bf16_bits(x) if dtype == "bf16" else x


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_three_pruning_layers_match_oracle_stage_by_stage(dtype):
    lay = build_layout([[600, 200, 401], [300, 64], [1000]], 4, 16, 60)
    hid = 256
    rng = np.random.default_rng(21)
    N = int(lay.cu_seqlens[-1])
    h0 = rng.standard_normal((N, hid)).astype(np.float32)
    h_prior_host = f32_to_bf16_bits(h0) if dtype == "bf16" else h0
    pos = torch.arange(N, dtype=torch.int64, device="cuda")[None, :].repeat(2, 1).contiguous()
    pruner = ProgressivePruner(A.DeviceLayout(lay), to_dev(h_prior_host, dtype))
    cur_lay = lay
    for layer, pct in enumerate([50, 40, 30]):
        say(f"progressive dtype={dtype} layer={layer} N_tok={cur_lay.cu_seqlens[-1]}")
        h_prior_host = _to_host(pruner.h_prior, dtype)
        h_cur_host = _noisy(h_prior_host, dtype, rng, 0.2 + 0.1 * layer)
        h_cur = to_dev(h_cur_host, dtype)
        h_out, (pos_out,), keep, bud, scores, isum = pruner.step(h_cur, [(pos, 1)],
                                                                keep_pct_next=pct)
        keep_h, bud_h = keep.cpu().numpy(), bud.cpu().numpy()
        # scores of this layer on the same inputs
        s_o, isum_o = O.variation_scores(cur_lay, h_cur_host, h_prior_host, dtype)
        vis = np.isfinite(s_o)
        assert_rel(scores.cpu().numpy()[vis], s_o[vis], TOL[dtype], "variation scores", abs_floor=1e-6)
        assert_rel(isum.cpu().numpy(), isum_o, TOL[dtype], "variation sums", abs_floor=1e-5)
        # budgets from the GPU's image sums, selection from its scores and budgets
        bud_o = O.budget(cur_lay, isum.cpu().numpy().astype(np.float32), 1.0, 50, 950, 0)
        assert bud_h.tolist() == bud_o.tolist()
        keep_o, cu_o = O.select(cur_lay, scores.cpu().numpy().astype(np.float32), bud_h)
        assert keep_h.tolist() == keep_o.tolist()
        assert int(bud_h.sum()) == int(np.sum(cur_lay.keep_total))
        # compacted rows are bit copies, position ids keep their original values
        assert np.array_equal(_to_host(h_out, dtype), h_cur_host[keep_h])
        assert np.array_equal(pos_out.cpu().numpy(), pos.cpu().numpy()[:, keep_h])
        # the next layout
        nxt = O.pruned_layout(cur_lay, keep_h, cu_o, O.keep_totals(
            O.pruned_layout(cur_lay, keep_h, cu_o, np.zeros(cur_lay.B, np.int32)), pct))
        for n in ("cu_seqlens", "img_start", "img_len", "cu_img", "text_pos", "cu_text", "keep_total"):
            assert pruner.dl.host[n].tolist() == getattr(nxt, n).tolist(), n
        assert pruner.dl.host["img_len"].tolist() == bud_h.tolist()
        pos = pos_out
        cur_lay = nxt
