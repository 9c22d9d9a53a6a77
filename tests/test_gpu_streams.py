"""Concurrent calls: the header promises that calls on different streams with
different buffers may run concurrently (the library keeps no global mutable
state outside the allocation-free score call).  Two host threads, each on its
own stream with its own buffers, run the whole layer (score, then budget +
select + compact) on two different workloads several times; every output
must equal, bit for bit, the same layer run alone on the default stream."""
import threading

import numpy as np
import pytest
import torch

from gpu_util import need_gpu, say, to_dev, to_host_bits
from paper_2608_26806_amd import avtp as A
from paper_2608_26806_amd.workloads import make_workload

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    need_gpu()
    A.lib()


class _Layer:
    def __init__(self, cfg):
        wl = make_workload(cfg, payload=True)
        self.wl, lay = wl, wl.layout
        self.dl = A.DeviceLayout(lay)
        self.q, self.k = to_dev(wl.q_text, wl.dtype), to_dev(wl.k, wl.dtype)
        hid = to_dev(wl.hidden_states, wl.dtype)
        self.ws = A.alloc_workspace(A.score_workspace_bytes(self.dl, A.SCORE_ATTN,
                                                            A.dtype_code(self.q), wl.Hq, wl.Hkv,
                                                            wl.d))
        self.out_h = torch.empty((self.dl.N_out, hid.shape[1]), dtype=hid.dtype, device="cuda")
        self.pairs = A.TensorSet([(hid, self.out_h, 0)])
        self.scores = torch.empty(lay.N_tok, device="cuda")
        self.isum = torch.empty(max(1, lay.n_img), device="cuda")
        self.bud = torch.empty(max(1, lay.n_img), dtype=torch.int32, device="cuda")
        self.keep = torch.empty(max(1, self.dl.N_out), dtype=torch.int32, device="cuda")
        self.cu = torch.empty(lay.B + 1, dtype=torch.int32, device="cuda")

    def step(self, stream=None):
        wl = self.wl
        A.score_attn(self.dl, self.q, self.k, wl.softmax_scale, scores=self.scores,
                     img_sum=self.isum, ws=self.ws, stream=stream)
        A.budget_select_compact(self.dl, self.isum, self.scores, self.pairs, wl.alpha,
                                wl.lo_permille, wl.hi_permille, wl.floor_abs, budget_out=self.bud,
                                keep_idx=self.keep, cu_out=self.cu, stream=stream)

    def outputs(self):
        return [to_host_bits(t) for t in (self.scores, self.isum, self.bud, self.keep, self.cu,
                                          self.out_h)]


def test_two_threads_two_streams_match_the_sequential_run():
    layers = [_Layer(2), _Layer(3)]
    say("[streams] configs 2 and 3, sequential reference")
    ref = []
    for lyr in layers:
        lyr.step()
        torch.cuda.synchronize()
        ref.append(lyr.outputs())
    streams = [torch.cuda.Stream() for _ in layers]   # default priority
    errors = []

    def run(i):
        try:
            with torch.cuda.stream(streams[i]):
                for _ in range(5):
                    layers[i].step()
            streams[i].synchronize()
        except Exception as e:                          # reported by the main thread
            errors.append(e)

    for lyr in layers:                                  # outputs overwritten before the run
        for t in (lyr.scores, lyr.isum, lyr.out_h):
            t.fill_(float("nan"))
    torch.cuda.synchronize()
    say("[streams] two threads, one stream each")
    threads = [threading.Thread(target=run, args=(i,)) for i in range(len(layers))]
    for t in threads:
        t.start()
    for t in threads:
        t.join(timeout=120)
    assert not any(t.is_alive() for t in threads)
    assert not errors, errors
    torch.cuda.synchronize()
    for lyr, r in zip(layers, ref):
        for got, want in zip(lyr.outputs(), r):
            assert np.array_equal(got, want)
