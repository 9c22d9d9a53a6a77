"""avtp_score_noalloc (the score call that allocates nothing, for callers that
cannot allocate) against avtp_score with a caller workspace: identical
kernels, so scores and image sums must match bit for bit.  Two calls in a
row through the C ABI, the second on a smaller layout, so the library's
per-GPU scratch is reused with the first call's contents still in it; then
the oracle's tolerance on the second, and avtp_score once more."""
import numpy as np
import pytest
import torch

from gpu_util import TOL, assert_rel, need_gpu, say, to_dev
from oracle import avtp_oracle as O
from paper_2608_26806_amd import avtp as A
from paper_2608_26806_amd.workloads import make_workload

pytestmark = pytest.mark.gpu


def _run_both(wl):
    lay = wl.layout
    dl = A.DeviceLayout(lay)
    q, k = to_dev(wl.q_text, wl.dtype), to_dev(wl.k, wl.dtype)
    need = A.score_workspace_bytes(dl, A.SCORE_ATTN, A.dtype_code(q), wl.Hq, wl.Hkv, wl.d)
    assert 0 < need <= A.NOALLOC_MAX_WORKSPACE
    st_ref = torch.zeros(lay.B, dtype=torch.int32, device="cuda")
    s_ref, isum_ref = A.score_attn(dl, q, k, wl.softmax_scale, status=st_ref)
    # outputs start as garbage: every visual and text position must be written
    s_na = torch.full((lay.N_tok,), float("nan"), dtype=torch.float32, device="cuda")
    isum_na = torch.full((max(1, lay.n_img),), -7.0, dtype=torch.float32, device="cuda")
    st_na = torch.zeros(lay.B, dtype=torch.int32, device="cuda")
    A.score_attn_noalloc(dl, q, k, wl.softmax_scale, s_na, isum_na, status=st_na)
    torch.cuda.synchronize()
    assert torch.equal(s_na.view(torch.int32), s_ref.view(torch.int32)), "scores differ"
    assert torch.equal(isum_na[: lay.n_img].view(torch.int32), isum_ref.view(torch.int32)), \
        "image sums differ"
    assert torch.equal(st_na, st_ref) and not st_na.any()
    return s_na.cpu().numpy(), isum_na[: lay.n_img].cpu().numpy()


def test_noalloc_matches_workspace_call_twice_then_smaller():
    need_gpu()
    A.lib()
    big = make_workload(5, payload=False)
    say("[noalloc] config 5 (7.6 MiB of scratch)")
    _run_both(big)
    say("[noalloc] config 5 again")
    _run_both(big)
    small = make_workload(2, payload=False)
    say("[noalloc] config 2 after config 5 (smaller, same scratch)")
    s_g, isum_g = _run_both(small)
    lay = small.layout
    s_o, isum_o, _, _ = O.attn_scores(lay, small.q_text, small.k, small.Hq, small.Hkv,
                                      small.softmax_scale, small.dtype)
    vis = lay.visual_mask()
    assert_rel(s_g[vis], s_o[vis], TOL["bf16"], "scores (noalloc)")
    assert_rel(isum_g, isum_o, TOL["bf16"], "image sums (noalloc)")
    # the workspace call still works after the scratch calls
    dl = A.DeviceLayout(lay)
    s2, _ = A.score_attn(dl, to_dev(small.q_text, "bf16"), to_dev(small.k, "bf16"),
                         small.softmax_scale)
    assert np.array_equal(s2.cpu().numpy().view(np.int32), s_g.view(np.int32))
