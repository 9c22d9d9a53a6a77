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
