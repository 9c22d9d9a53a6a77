"""The layer step captured in a HIP graph and replayed.

The step (avtp_score, then avtp_budget_select_compact; or the same with
avtp_score_noalloc) is captured with torch.cuda.graph: the C ABI calls
enqueue their kernels on torch's current stream, which is the capture stream,
and they allocate nothing and enqueue no memset, so they can be captured.
Each replay follows eager work that overwrites every output, and each
replay's outputs (scores, image sums, budgets, kept indices, cu_out, the
compacted hidden states, position ids, K and V, status) must equal the eager
step's bit for bit.  The binding's prepared calls (arguments marshalled once,
as the bench's timed step issues them) are checked the same way."""
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


def _setup(cfg):
    wl = make_workload(cfg, payload=True)
    lay = wl.layout
    dl = A.DeviceLayout(lay)
    q, k, v = to_dev(wl.q_text, wl.dtype), to_dev(wl.k, wl.dtype), to_dev(wl.v, wl.dtype)
    hid = to_dev(wl.hidden_states, wl.dtype)
    pos = torch.from_numpy(wl.pos).cuda()
    ws = A.alloc_workspace(A.score_workspace_bytes(dl, A.SCORE_ATTN, A.dtype_code(q), wl.Hq,
                                                   wl.Hkv, wl.d))
    out = {"scores": torch.empty(lay.N_tok, dtype=torch.float32, device="cuda"),
           "isum": torch.empty(max(1, lay.n_img), dtype=torch.float32, device="cuda"),
           "bud": torch.empty(max(1, lay.n_img), dtype=torch.int32, device="cuda"),
           "keep": torch.empty(max(1, lay.N_out), dtype=torch.int32, device="cuda"),
           "cu_out": torch.empty(lay.B + 1, dtype=torch.int32, device="cuda"),
           "status": torch.zeros(lay.B, dtype=torch.int32, device="cuda")}
    pairs = []
    for i, (src, tdim) in enumerate([(hid, 0), (pos, 1), (k, 0), (v, 0)]):
        shape = list(src.shape)
        shape[tdim] = lay.N_out
        dst = torch.empty(shape, dtype=src.dtype, device="cuda")
        out[f"t{i}"] = dst
        pairs.append((src, dst, tdim))
    tset = A.TensorSet(pairs)
    return wl, dl, q, k, ws, out, tset


def _step(wl, dl, q, k, ws, out, tset, noalloc):
    if noalloc:
        A.score_attn_noalloc(dl, q, k, wl.softmax_scale, out["scores"], out["isum"],
                             status=out["status"])
    else:
        A.score_attn(dl, q, k, wl.softmax_scale, scores=out["scores"], img_sum=out["isum"],
                     status=out["status"], ws=ws)
    A.budget_select_compact(dl, out["isum"], out["scores"], tset, wl.alpha, wl.lo_permille,
                            wl.hi_permille, wl.floor_abs, budget_out=out["bud"],
                            keep_idx=out["keep"], cu_out=out["cu_out"], status=out["status"])


def _scramble(out):
    # eager work between replays: every output overwritten
    for name, t in out.items():
        if name == "status":
            t.zero_()
        elif t.is_floating_point():
            t.fill_(float("nan"))
        else:
            t.fill_(-3)


@pytest.mark.parametrize("cfg,noalloc", [(1, False), (2, False), (3, False), (2, True)])
def test_graph_replays_equal_the_eager_step(cfg, noalloc):
    wl, dl, q, k, ws, out, tset = _setup(cfg)
    say(f"[graph] config {cfg} noalloc={noalloc}")
    _scramble(out)
    _step(wl, dl, q, k, ws, out, tset, noalloc)          # eager (also the first no-alloc call)
    torch.cuda.synchronize()
    ref = {n: to_host_bits(t) for n, t in out.items()}
    assert not out["status"].any()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):                         # a warm-up call off the default stream
        _step(wl, dl, q, k, ws, out, tset, noalloc)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        _step(wl, dl, q, k, ws, out, tset, noalloc)
    torch.cuda.synchronize()
    for r in range(3):
        _scramble(out)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for n, t in out.items():
            assert np.array_equal(to_host_bits(t), ref[n]), (r, n)


def test_prepared_calls_equal_the_plain_calls():
    # the binding's prepared calls (arguments marshalled once), issued twice,
    # against the plain calls on the same inputs
    wl, dl, q, k, ws, out, tset = _setup(2)
    say("[prepared] config 2")
    _scramble(out)
    _step(wl, dl, q, k, ws, out, tset, False)
    torch.cuda.synchronize()
    ref = {n: to_host_bits(t) for n, t in out.items()}
    calls = [A.prepare_score_attn(dl, q, k, wl.softmax_scale, out["scores"], out["isum"], ws,
                                  status=out["status"]),
             A.prepare_budget_select_compact(dl, out["isum"], out["scores"], tset, out["bud"],
                                             out["keep"], out["cu_out"], wl.alpha, wl.lo_permille,
                                             wl.hi_permille, wl.floor_abs, status=out["status"])]
    for r in range(2):
        _scramble(out)
        for c in calls:
            c()
        torch.cuda.synchronize()
        for n, t in out.items():
            assert np.array_equal(to_host_bits(t), ref[n]), (r, n)
