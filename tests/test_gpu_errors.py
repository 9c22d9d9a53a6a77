"""Error reporting through the C ABI on the GPU.

A failed HIP call that the caller made before entering the library (here
hipSetDevice on a device that does not exist, an error on the host that
touches no GPU state) leaves its error for hipGetLastError().  The library's
calls must still succeed and report only their own launches, and must leave
no error behind."""
import ctypes

import numpy as np
import pytest
import torch

from gpu_util import need_gpu, say
from oracle import avtp_oracle as O
from paper_2608_26806_amd import avtp as A
from paper_2608_26806_amd.workloads import make_workload

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    need_gpu()
    A.lib()


def _hip():
    return ctypes.CDLL("libamdhip64.so")


def test_calls_after_a_failed_caller_hip_call_succeed():
    wl = make_workload(2, payload=True)
    lay = wl.layout
    dl = A.DeviceLayout(lay)
    dev = lambda x: torch.from_numpy(np.ascontiguousarray(x).view(np.int16)).view(torch.bfloat16).cuda()
    q, k = dev(wl.q_text), dev(wl.k)
    hip = _hip()
    torch.cuda.synchronize()

    def stale():
        assert hip.hipSetDevice(999) != 0          # fails on the host; the error stays pending

    say("[errors] score, budget, select, budget+select+compact after a failed hipSetDevice")
    stale()
    scores, isum = A.score_attn(dl, q, k, wl.softmax_scale)
    stale()
    bud = A.budget(dl, isum, wl.alpha, wl.lo_permille, wl.hi_permille, wl.floor_abs)
    stale()
    keep, cu = A.select(dl, scores, bud)
    stale()
    bud2, keep2, cu2 = A.budget_select_compact(dl, isum, scores, [], wl.alpha, wl.lo_permille,
                                               wl.hi_permille, wl.floor_abs)
    torch.cuda.synchronize()
    assert hip.hipGetLastError() == 0               # the library leaves no error behind
    assert torch.equal(bud, bud2) and torch.equal(keep, keep2) and torch.equal(cu, cu2)
    g = bud.cpu().numpy()
    assert np.array_equal(g, O.budget(lay, isum.cpu().numpy(), wl.alpha, wl.lo_permille,
                                      wl.hi_permille, wl.floor_abs))


def test_binding_rejects_short_buffers_wrong_dtypes_and_small_destinations():
    # checked in the binding before the call: a kernel would otherwise read or
    # write past the end of a short buffer
    wl = make_workload(2)
    dl = A.DeviceLayout(wl.layout)
    isum = torch.rand(dl.n_img, device="cuda")
    scores = torch.rand(dl.N_tok, device="cuda")
    bud = A.budget(dl, isum, 1.0)
    say("[errors] binding argument checks")
    with pytest.raises(ValueError, match="at least"):
        A.select(dl, scores[: dl.N_tok - 1], bud)
    with pytest.raises(TypeError, match="float32"):
        A.budget(dl, isum.double(), 1.0)
    with pytest.raises(ValueError, match="contiguous"):
        A.select(dl, torch.rand(dl.N_tok, 2, device="cuda")[:, 0], bud)
    keep, _ = A.select(dl, scores, bud)
    src = torch.rand(dl.N_tok, 16, device="cuda")
    with pytest.raises(ValueError, match="destination rows"):
        A.compact(dl, keep, [(src, torch.empty(dl.N_out - 1, 16, device="cuda"))])
    with pytest.raises(TypeError, match="differ"):
        A.compact(dl, keep, [(src, torch.empty(dl.N_out, 16, device="cuda", dtype=torch.float16))])
    with pytest.raises(ValueError, match="rows differ"):
        A.compact(dl, keep, [(src, torch.empty(dl.N_out, 8, device="cuda"))])
    out = torch.empty(dl.N_out, 16, device="cuda")
    A.compact(dl, keep, [(src, out)])                   # the well-formed call still runs
    torch.cuda.synchronize()
    assert torch.equal(out, src[keep.long()])
