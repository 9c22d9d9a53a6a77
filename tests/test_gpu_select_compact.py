"""GPU parity of avtp_select_compact (selection and compaction in one launch)
against the oracle and against avtp_select followed by avtp_compact: kept
indices, cu_out and every compacted tensor bit-exact."""
import numpy as np
import pytest
import torch

from gpu_util import need_gpu, say, to_dev, to_host_bits
from oracle import avtp_oracle as O
from paper_2608_26806_amd import avtp as A
from paper_2608_26806_amd.workloads import build_layout, make_workload

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    need_gpu()
    A.lib()


LAYOUTS = {
    "mixed": ([[300, 1, 57], [], [129, 64, 2], [700]], 4, 9),
    "big_image": ([[0, 5], [9000, 3], [], [50, 0, 7]], 0, 6),   # an image past the LDS key cache
    "text_only": ([[], []], 0, 5),
}


def _scores(lay, pattern, rng):
    s = np.full(lay.N_tok, np.inf, np.float32)
    for i in range(lay.n_img):
        st, n = int(lay.img_start[i]), int(lay.img_len[i])
        if pattern == "random":
            v = rng.standard_normal(n).astype(np.float32)
        elif pattern == "ties":
            v = (rng.integers(0, 4, size=n) / 8).astype(np.float32)
        else:
            v = rng.choice(np.array([np.nan, -0.0, 0.0, -np.inf, 1e-30, -1e-30, 3.0], np.float32), n)
        s[st:st + n] = v
    return s


@pytest.mark.parametrize("pattern", ["random", "ties", "special"])
@pytest.mark.parametrize("name", sorted(LAYOUTS))
def test_fused_matches_oracle(name, pattern):
    imgs, pre, tail = LAYOUTS[name]
    lay0 = build_layout(imgs, pre, tail, 50)
    rng = np.random.default_rng(len(name) * 7 + len(pattern))
    s = _scores(lay0, pattern, rng)
    budgets = np.array([int(rng.integers(0, n + 1)) for n in lay0.img_len], np.int32)
    arrays = {nm: getattr(lay0, nm) for nm in A.DeviceLayout.NAMES}
    arrays["keep_total"] = [int(budgets[lay0.cu_img[b]:lay0.cu_img[b + 1]].sum()) for b in range(lay0.B)]
    dl = A.DeviceLayout(arrays)
    say(f"[select_compact] layout={name} pattern={pattern}")
    N, n_out = lay0.N_tok, dl.N_out
    hid = torch.randn(N, 64, device="cuda").to(torch.bfloat16)
    pos = torch.randint(0, 1 << 40, (3, N), dtype=torch.int64, device="cuda")
    odd = torch.randint(0, 255, (N, 3), dtype=torch.uint8, device="cuda")
    kv = torch.randn(N, 2, 16, device="cuda").to(torch.bfloat16)
    kv_hm = kv.transpose(0, 1).contiguous()                      # head-major planes
    outs = [torch.empty((n_out, 64), dtype=torch.bfloat16, device="cuda"),
            torch.empty((3, n_out), dtype=torch.int64, device="cuda"),
            torch.empty((n_out, 3), dtype=torch.uint8, device="cuda"),
            torch.empty((2, n_out, 16), dtype=torch.bfloat16, device="cuda")]
    pairs = [(hid, outs[0], 0), (pos, outs[1], 1), (odd, outs[2], 0), (kv_hm, outs[3], 1)]
    keep, cu = A.select_compact(dl, torch.from_numpy(s).cuda(), torch.from_numpy(budgets).cuda(), pairs)
    torch.cuda.synchronize()
    keep_o, cu_o = O.select(lay0, s, budgets)
    assert keep.cpu().numpy().tolist() == keep_o.tolist()
    assert cu.cpu().numpy().tolist() == cu_o.tolist()
    idx = torch.from_numpy(keep_o.astype(np.int64)).cuda()
    assert torch.equal(outs[0], hid[idx])
    assert torch.equal(outs[1], pos[:, idx])
    assert torch.equal(outs[2], odd[idx])
    assert torch.equal(outs[3], kv_hm[:, idx])


@pytest.mark.parametrize("cfg", [2, 3])
def test_fused_equals_separate_calls(cfg):
    wl = make_workload(cfg, payload=True)
    lay = wl.layout
    dl = A.DeviceLayout(lay)
    say(f"[select_compact] config {cfg}")
    rng = np.random.default_rng(cfg)
    s = rng.random(lay.N_tok).astype(np.float32)
    bud = O.budget(lay, np.array([s[a:a + n].sum() for a, n in zip(lay.img_start, lay.img_len)],
                                 np.float32), 1.0)
    sd, bd = torch.from_numpy(s).cuda(), torch.from_numpy(bud).cuda()
    hid = to_dev(wl.hidden_states, wl.dtype)
    pos = torch.from_numpy(wl.pos).cuda()
    kd, vd = to_dev(wl.k, wl.dtype), to_dev(wl.v, wl.dtype)
    srcs = [(hid, 0), (pos, 1), (kd, 0), (vd, 0)]
    keep_a, cu_a = A.select(dl, sd, bd)
    outs_a = A.compact_new(dl, keep_a, srcs)
    outs_b = []
    pairs = []
    for src, tdim in srcs:
        shape = list(src.shape)
        shape[tdim] = dl.N_out
        dst = torch.empty(shape, dtype=src.dtype, device="cuda")
        outs_b.append(dst)
        pairs.append((src, dst, tdim))
    keep_b, cu_b = A.select_compact(dl, sd, bd, pairs)
    torch.cuda.synchronize()
    assert torch.equal(keep_a, keep_b) and torch.equal(cu_a, cu_b)
    for x, y in zip(outs_a, outs_b):
        assert np.array_equal(to_host_bits(x), to_host_bits(y))


def test_fused_budgets_over_keep_total_flag_and_stay_in_bounds():
    # budgets that sum past keep_total: keep_idx is written up to its capacity
    # (and the overflow flagged) exactly as avtp_select does; rows are copied
    # only below n_out, so outputs sized for n_out are never overrun
    lay = build_layout([[40, 30], [25]], 2, 3, 50)
    rng = np.random.default_rng(5)
    s = rng.standard_normal(lay.N_tok).astype(np.float32)
    budgets = np.array([30, 20, 20], np.int32)                  # keep_total is 35 and 13;
    # sequence 0 writes entries [0, 57), sequence 1 [57, 82): past cap = n_out + 4 = 64
    dl = A.DeviceLayout(lay)
    n_out = dl.N_out
    cap = n_out + 4                                              # some spare entries in keep_idx
    say("[select_compact] over-full budgets")
    hid = torch.randn(lay.N_tok, 48, device="cuda")
    guard = torch.full((n_out + 8, 48), 7.0, device="cuda")     # rows past n_out must stay 7
    out = guard[:n_out]
    keep_f = torch.full((cap,), -1, dtype=torch.int32, device="cuda")
    st_f = torch.zeros(lay.B, dtype=torch.int32, device="cuda")
    keep_f, cu_f = A.select_compact(dl, torch.from_numpy(s).cuda(), torch.from_numpy(budgets).cuda(),
                                    [(hid, out, 0)], keep_idx=keep_f, status=st_f)
    keep_s = torch.full((cap,), -1, dtype=torch.int32, device="cuda")
    st_s = torch.zeros(lay.B, dtype=torch.int32, device="cuda")
    A.select(dl, torch.from_numpy(s).cuda(), torch.from_numpy(budgets).cuda(), keep_idx=keep_s,
             status=st_s)
    torch.cuda.synchronize()
    st = st_f.cpu().numpy()
    assert st.tolist() == st_s.cpu().numpy().tolist()
    assert st.tolist() == [0, A.FLAG_OUT_CAPACITY]               # only the second sequence overflows
    ks = keep_s.cpu().numpy()[:n_out]
    assert keep_f.cpu().numpy()[:n_out].tolist() == ks.tolist()
    assert torch.equal(out, hid[torch.from_numpy(ks.astype(np.int64)).cuda()])
    assert torch.all(guard[n_out:] == 7.0)
