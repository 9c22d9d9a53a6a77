"""Seeded random layouts through the variation score and the next layer's
layout update, against the oracle.

Variation: every visual score and image sum within the dtype's tolerance
(plus an absolute floor for the cancellation of near-identical rows), over
random hidden sizes and both dtypes, with visual tokens whose two states are
identical (score 0), opposite (2), zero (1, the norm guard) or scaled copies.
Layout update: the next layer's arrays bit-exact for random kept subsets of
the same random layouts (every text token kept)."""
import numpy as np
import pytest
import torch

from gpu_util import TOL, assert_rel, need_gpu, say, to_dev
from oracle import avtp_oracle as O
from paper_2608_26806_amd import avtp as A
from paper_2608_26806_amd.workloads import f32_to_bf16_bits
from test_gpu_random_scores import _random_layout

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    need_gpu()
    A.lib()


@pytest.mark.parametrize("seed", range(12))
def test_random_layout_variation(seed):
    rng = np.random.default_rng(3000 + seed)
    lay = _random_layout(rng)
    dt = "fp32" if rng.random() < 0.3 else "bf16"
    hidden = int(rng.choice([8, 64, 256, 1000, 4096]))
    h = rng.standard_normal((lay.N_tok, hidden)).astype(np.float32)
    h *= rng.lognormal(0.0, 1.0, size=(lay.N_tok, 1)).astype(np.float32)
    hp = h + 0.5 * rng.standard_normal(h.shape).astype(np.float32)
    vis = np.flatnonzero(lay.visual_mask())
    if len(vis):
        pick = rng.choice(vis, size=min(len(vis), 40), replace=False)
        for j, kind in zip(pick, rng.integers(0, 5, size=len(pick))):
            if kind == 0:
                hp[j] = h[j]                        # identical: 0
            elif kind == 1:
                hp[j] = -h[j]                       # opposite: 2
            elif kind == 2:
                h[j] = 0.0
                hp[j] = 0.0                         # both zero: the guard gives 1
            elif kind == 3:
                hp[j] = 0.0                         # one zero: 1
            else:
                hp[j] = 3.0 * h[j]                  # scaled copy: 0
    hc_h, hp_h = (f32_to_bf16_bits(h), f32_to_bf16_bits(hp)) if dt == "bf16" else (h, hp)
    say(f"[random variation] seed {seed}: B={lay.B} images={lay.n_img} N_tok={lay.N_tok} "
        f"hidden={hidden} {dt}")
    dl = A.DeviceLayout(lay)
    status = torch.zeros(lay.B, dtype=torch.int32, device="cuda")
    s_g, isum_g = A.score_variation(dl, to_dev(hc_h, dt), to_dev(hp_h, dt), status=status)
    s_o, isum_o = O.variation_scores(lay, hc_h, hp_h, dt)
    m = lay.visual_mask()
    s_g = s_g.cpu().numpy()
    assert_rel(s_g[m], s_o[m], TOL[dt], "variation scores", abs_floor=1e-6)
    assert np.all(np.isinf(s_g[~m]))
    if lay.n_img:
        assert_rel(isum_g.cpu().numpy(), isum_o, TOL[dt], "variation sums", abs_floor=1e-4)
    assert not status.cpu().numpy().any()


def _random_keep(lay, rng):
    """Every text token and a random subset of every image (fraction per image)."""
    keep, cu = [], [0]
    for b in range(lay.B):
        s0, s1 = int(lay.cu_seqlens[b]), int(lay.cu_seqlens[b + 1])
        take = np.ones(s1 - s0, dtype=bool)
        for i in range(int(lay.cu_img[b]), int(lay.cu_img[b + 1])):
            st, n = int(lay.img_start[i]) - s0, int(lay.img_len[i])
            take[st:st + n] = rng.random(n) < rng.choice([0.0, 0.1, 0.5, 1.0])
        keep.extend((s0 + np.flatnonzero(take)).tolist())
        cu.append(len(keep))
    return np.array(keep, np.int32), np.array(cu, np.int32)


@pytest.mark.parametrize("seed", range(12))
def test_random_layout_update(seed):
    rng = np.random.default_rng(4000 + seed)
    lay = _random_layout(rng)
    keep, cu = _random_keep(lay, rng)
    say(f"[random layout update] seed {seed}: B={lay.B} images={lay.n_img} kept={len(keep)}")
    dl = A.DeviceLayout(lay)
    keep_d = np.zeros(max(1, len(keep)), np.int32)      # (an empty list still gets an entry)
    keep_d[:len(keep)] = keep
    got = A.pruned_layout(dl, torch.from_numpy(keep_d).cuda(), torch.from_numpy(cu).cuda())
    ref = O.pruned_layout(lay, keep, cu, np.zeros(lay.B, np.int32))
    for n in ("cu_seqlens", "img_start", "img_len", "cu_img", "text_pos", "cu_text"):
        assert got[n].cpu().numpy().tolist() == getattr(ref, n).tolist(), n
