"""The whole layer at the size limits the header states: one image of
AVTP_MAX_IMAGE_LEN tokens, and AVTP_MAX_IMAGES images in one batch.

Each runs avtp_score, then avtp_budget_select_compact (the bench's step), and
checks against the oracle: scores and image sums within the bf16 tolerance,
budgets bit-exact on the GPU's image sums, the selection bit-exact on the
GPU's scores and budgets, the compaction bit-exact, and, for the single image
(whose budget is its keep total whatever the sums), the kept set equal to the
oracle chain's outside the threshold band."""
import numpy as np
import pytest
import torch

from gpu_util import TOL, assert_rel, kept_sets_match, need_gpu, say, to_dev, to_host_bits
from oracle import avtp_oracle as O
from paper_2608_26806_amd import avtp as A
from paper_2608_26806_amd.workloads import build_layout, f32_to_bf16_bits

pytestmark = pytest.mark.gpu

MAX_IMAGE_LEN = 1 << 20   # AVTP_MAX_IMAGE_LEN
MAX_IMAGES = 8192         # AVTP_MAX_IMAGES


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    need_gpu()
    A.lib()


def _layer(lay, rng, Hq=4, Hkv=2, d=64, width=16):
    q32 = rng.standard_normal((lay.T_tot, Hq, d)).astype(np.float32)
    k32 = rng.standard_normal((lay.N_tok, Hkv, d)).astype(np.float32)
    qb, kb = f32_to_bf16_bits(q32), f32_to_bf16_bits(k32)
    hid = f32_to_bf16_bits(rng.standard_normal((lay.N_tok, width)).astype(np.float32))
    dl = A.DeviceLayout(lay)
    status = torch.zeros(lay.B, dtype=torch.int32, device="cuda")
    s_g, isum_g = A.score_attn(dl, to_dev(qb, "bf16"), to_dev(kb, "bf16"), d ** -0.5,
                               status=status)
    hid_d = to_dev(hid, "bf16")
    out = torch.empty((dl.N_out, width), dtype=torch.bfloat16, device="cuda")
    bud_g, keep_g, cu_g = A.budget_select_compact(dl, isum_g, s_g, [(hid_d, out, 0)], 1.0, 50,
                                                  950, 0, status=status)
    torch.cuda.synchronize()
    assert not status.cpu().numpy().any()
    g = {"s": s_g.cpu().numpy(), "isum": isum_g.cpu().numpy(), "bud": bud_g.cpu().numpy(),
         "keep": keep_g.cpu().numpy(), "cu": cu_g.cpu().numpy(), "hid": to_host_bits(out)}
    s_o, isum_o, _, _ = O.attn_scores(lay, qb, kb, Hq, Hkv, d ** -0.5, "bf16")
    vis = lay.visual_mask()
    assert_rel(g["s"][vis], s_o[vis], TOL["bf16"], "scores")
    assert_rel(g["isum"], isum_o, TOL["bf16"], "image sums")
    assert np.array_equal(g["bud"], O.budget(lay, g["isum"], 1.0, 50, 950, 0))
    keep_s, cu_s = O.select(lay, g["s"], g["bud"])
    assert np.array_equal(g["keep"], keep_s) and np.array_equal(g["cu"], cu_s)
    assert np.array_equal(g["hid"], O.compact(g["keep"], hid))
    return g, s_o, isum_o


def test_longest_image():
    rng = np.random.default_rng(20)
    lay = build_layout([[MAX_IMAGE_LEN]], 2, 6, 10)
    say(f"[limits] one image of {MAX_IMAGE_LEN} tokens, N_tok={lay.N_tok}")
    g, s_o, isum_o = _layer(lay, rng)
    bud_o = O.budget(lay, isum_o.astype(np.float32), 1.0, 50, 950, 0)
    assert np.array_equal(g["bud"], bud_o)   # one image: its budget is the keep total
    keep_o, _ = O.select(lay, s_o.astype(np.float32), bud_o)
    kept_sets_match(lay, g["keep"], keep_o, s_o, bud_o, TOL["bf16"])


def test_most_images():
    rng = np.random.default_rng(21)
    seqs = [[int(x) for x in rng.integers(2, 10, size=64)] for _ in range(MAX_IMAGES // 64)]
    lay = build_layout(seqs, 1, 2, 50)
    assert lay.n_img == MAX_IMAGES
    say(f"[limits] {lay.n_img} images in {lay.B} sequences, N_tok={lay.N_tok}")
    _layer(lay, rng)
