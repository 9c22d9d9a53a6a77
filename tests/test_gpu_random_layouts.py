"""Seeded random layouts through budget, selection and compaction, against
the oracle: avtp_budget_select_compact (one call), avtp_budget, avtp_select,
avtp_compact (three calls) and avtp_budget then avtp_select_compact must all
give the oracle's budgets, kept indices, cu_out and compacted tensors bit for
bit.

The layouts mix what the fixed workloads do not: a random number of text rows
before every image (none included), empty and one-token images, images longer
than the selection keeps in LDS, sequences without images, up to 70 images
per sequence (above 64 the budget kernel runs first), keep totals anywhere
between their bounds, absolute floors, both budget modes, and scores with
exact ties, signed zeros, infinities and NaNs.  Some draws add a wide tensor
so that the compaction moves more than the one-launch limit."""
import numpy as np
import pytest
import torch

from gpu_util import need_gpu, say, to_host_bits
from oracle import avtp_oracle as O
from paper_2608_26806_amd import avtp as A
from paper_2608_26806_amd.workloads import Layout

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    need_gpu()
    A.lib()


def _random_layout(rng):
    cu_seqlens, img_start, img_len, cu_img, text_pos, cu_text = [0], [], [], [0], [], [0]
    pos = 0
    for _ in range(int(rng.integers(1, 7))):
        for _ in range(int(rng.choice([0, 1, 2, 5, 17, 40, 70]))):
            nt = int(rng.integers(0, 4))
            text_pos.extend(range(pos, pos + nt))
            pos += nt
            u = rng.random()
            n = (0 if u < 0.08 else 1 if u < 0.15 else int(rng.integers(4100, 6000)) if u < 0.19
                 else int(rng.integers(2, 700)))
            img_start.append(pos)
            img_len.append(n)
            pos += n
        nt = int(rng.integers(0, 6))
        if pos == cu_seqlens[-1] and nt == 0:
            nt = 1                                   # every sequence holds a token
        text_pos.extend(range(pos, pos + nt))
        pos += nt
        cu_seqlens.append(pos)
        cu_img.append(len(img_len))
        cu_text.append(len(text_pos))
    a = lambda v: np.asarray(v, dtype=np.int32)
    lay = Layout(a(cu_seqlens), a(img_start), a(img_len), a(cu_img), a(text_pos), a(cu_text),
                 np.zeros(len(cu_seqlens) - 1, np.int32))
    return lay


def _scores(rng, lay):
    s = rng.standard_normal(lay.N_tok).astype(np.float32)
    for i in range(lay.n_img):
        st, n = int(lay.img_start[i]), int(lay.img_len[i])
        u = rng.random()
        if u < 0.15:
            s[st:st + n] = np.float32(0.25)                        # one value: all ties
        elif u < 0.3:
            s[st:st + n] = np.round(s[st:st + n] * 2) / 2          # few distinct values
        elif u < 0.4 and n > 4:
            specials = np.array([np.nan, -0.0, 0.0, np.inf, -np.inf], np.float32)
            at = rng.integers(st, st + n, size=min(n, 8))
            s[at] = specials[rng.integers(0, len(specials), size=len(at))]
    return s


@pytest.mark.parametrize("seed", range(16))
def test_random_layout_one_call_and_three_calls(seed):
    rng = np.random.default_rng(1000 + seed)
    lay = _random_layout(rng)
    lo_pm, hi_pm = int(rng.choice([0, 50, 100])), int(rng.choice([900, 950, 1000]))
    fa = int(rng.choice([0, 3, 16]))
    alpha = float(rng.choice([0.0, 1.0, 2.5]))
    mode = O.BUDGET_RAW if rng.random() < 0.3 else O.BUDGET_PROPORTIONAL
    keeps = []
    for b in range(lay.B):
        ns = lay.img_len[lay.cu_img[b]:lay.cu_img[b + 1]]
        lo = sum(O.budget_bounds(int(x), lo_pm, hi_pm, fa)[0] for x in ns)
        hi = sum(O.budget_bounds(int(x), lo_pm, hi_pm, fa)[1] for x in ns)
        keeps.append(int(rng.integers(lo, hi + 1)))
    lay.keep_total[:] = keeps
    S = (rng.lognormal(0.0, 1.5, size=max(1, lay.n_img)) *
         np.maximum(1, np.append(lay.img_len, 0)[:max(1, lay.n_img)]) / 100).astype(np.float32)
    if lay.n_img and rng.random() < 0.2:
        S[int(rng.integers(0, lay.n_img))] = 0.0
    s = _scores(rng, lay)
    wide = rng.random() < 0.3
    say(f"[random layout] seed {seed}: B={lay.B} images={lay.n_img} N_tok={lay.N_tok} "
        f"T={lay.T_tot} N_out={lay.N_out} lo/hi={lo_pm}/{hi_pm} floor={fa} alpha={alpha} "
        f"mode={mode} wide={wide}")

    bud_o = O.budget(lay, S[:lay.n_img], alpha, lo_pm, hi_pm, fa, mode)
    keep_o, cu_o = O.select(lay, s, bud_o)

    dl = A.DeviceLayout(lay)
    S_d, s_d = torch.from_numpy(S).cuda(), torch.from_numpy(s).cuda()
    srcs = [(torch.randn(lay.N_tok, 24, device="cuda").to(torch.bfloat16), 0),
            (torch.randint(0, 1 << 40, (3, lay.N_tok), dtype=torch.int64, device="cuda"), 1)]
    if wide:
        srcs.append((torch.randn(lay.N_tok, 2048, device="cuda").to(torch.bfloat16), 0))
    idx = torch.from_numpy(keep_o.astype(np.int64)).cuda()
    want = [x.index_select(d, idx) for x, d in srcs]

    def outs():
        res = []
        for x, d in srcs:
            shape = list(x.shape)
            shape[d] = dl.N_out
            res.append(torch.full(shape, 7, dtype=x.dtype, device="cuda"))
        return res

    # one call
    out1 = outs()
    status = torch.zeros(lay.B, dtype=torch.int32, device="cuda")
    bud, keep, cu = A.budget_select_compact(dl, S_d, s_d, [(x, o, d) for (x, d), o in
                                                           zip(srcs, out1)],
                                            alpha, lo_pm, hi_pm, fa, mode, status=status)
    torch.cuda.synchronize()
    assert np.array_equal(bud.cpu().numpy(), bud_o)
    assert np.array_equal(keep.cpu().numpy()[:lay.N_out], keep_o)
    assert np.array_equal(cu.cpu().numpy(), cu_o)
    for o, w in zip(out1, want):
        assert np.array_equal(to_host_bits(o), to_host_bits(w))
    assert not status.cpu().numpy().any()

    # three calls
    out3 = outs()
    status.zero_()
    bud3 = A.budget(dl, S_d, alpha, lo_pm, hi_pm, fa, mode, status=status)
    keep3, cu3 = A.select(dl, s_d, bud3, status=status)
    A.compact(dl, keep3, A.TensorSet([(x, o, d) for (x, d), o in zip(srcs, out3)]))
    torch.cuda.synchronize()
    assert np.array_equal(bud3.cpu().numpy(), bud_o)
    assert np.array_equal(keep3.cpu().numpy()[:lay.N_out], keep_o)
    assert np.array_equal(cu3.cpu().numpy(), cu_o)
    for o, w in zip(out3, want):
        assert np.array_equal(to_host_bits(o), to_host_bits(w))
    assert not status.cpu().numpy().any()

    # selection and compaction in one call, given the budgets
    out2 = outs()
    keep2, cu2 = A.select_compact(dl, s_d, bud3, [(x, o, d) for (x, d), o in zip(srcs, out2)],
                                  status=status)
    torch.cuda.synchronize()
    assert np.array_equal(keep2.cpu().numpy()[:lay.N_out], keep_o)
    assert np.array_equal(cu2.cpu().numpy(), cu_o)
    for o, w in zip(out2, want):
        assert np.array_equal(to_host_bits(o), to_host_bits(w))
    assert not status.cpu().numpy().any()
