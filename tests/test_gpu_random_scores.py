"""Seeded random layouts through the attention score, against the oracle:
every row LSE (within the dtype's tolerance, absolute), every visual score and
every image sum (relative), both from the two-pass call and from pass 2 given
the oracle's LSE, and the no-text-after flag exactly on the sequences where
the oracle finds an image with no text row after it (its scores 0).

The layouts put a random number of text rows before every image and after the
last one (none included), with empty, one-token and ragged images and
sequences without images; the head grouping, head size and dtype vary too.
So the kernels' causal masks meet key tiles and stages that rows see in full,
in part or not at all, rows of one block spread over the whole sequence, and
pass 2's query split on most draws."""
import numpy as np
import pytest
import torch

from gpu_util import TOL, assert_rel, need_gpu, say, to_dev
from oracle import avtp_oracle as O
from paper_2608_26806_amd import avtp as A
from paper_2608_26806_amd.workloads import Layout, f32_to_bf16_bits

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    need_gpu()
    A.lib()


def _random_layout(rng):
    cu_seqlens, img_start, img_len, cu_img, text_pos, cu_text = [0], [], [], [0], [], [0]
    pos = 0
    for _ in range(int(rng.integers(1, 4))):
        for _ in range(int(rng.choice([0, 1, 2, 4, 6]))):
            nt = int(rng.integers(0, 6))
            text_pos.extend(range(pos, pos + nt))
            pos += nt
            u = rng.random()
            n = 0 if u < 0.05 else 1 if u < 0.1 else int(rng.integers(2, 600))
            img_start.append(pos)
            img_len.append(n)
            pos += n
        u = rng.random()
        nt = 0 if u < 0.25 else int(rng.integers(200, 400)) if u < 0.35 else int(rng.integers(1, 41))
        if pos == cu_seqlens[-1] and nt == 0:
            nt = 1                                   # every sequence holds a token
        text_pos.extend(range(pos, pos + nt))
        pos += nt
        cu_seqlens.append(pos)
        cu_img.append(len(img_len))
        cu_text.append(len(text_pos))
    a = lambda v: np.asarray(v, dtype=np.int32)
    return Layout(a(cu_seqlens), a(img_start), a(img_len), a(cu_img), a(text_pos), a(cu_text),
                  np.zeros(len(cu_seqlens) - 1, np.int32))


@pytest.mark.parametrize("seed", range(16))
def test_random_layout_scores(seed):
    rng = np.random.default_rng(2000 + seed)
    lay = _random_layout(rng)
    Hkv = int(rng.choice([1, 2]))
    Hq = Hkv * int(rng.choice([1, 2, 4, 7]))
    d = int(rng.choice([64, 128]))
    dt = "fp32" if rng.random() < 0.25 else "bf16"
    scale = d ** -0.5
    q32 = rng.standard_normal((lay.T_tot, Hq, d)).astype(np.float32)
    k32 = rng.standard_normal((lay.N_tok, Hkv, d)).astype(np.float32)
    k32[lay.visual_mask()] *= np.float32(rng.uniform(0.5, 2.0))
    q, k = (f32_to_bf16_bits(q32), f32_to_bf16_bits(k32)) if dt == "bf16" else (q32, k32)
    say(f"[random scores] seed {seed}: B={lay.B} images={lay.n_img} N_tok={lay.N_tok} "
        f"T={lay.T_tot} Hq={Hq} Hkv={Hkv} d={d} {dt}")
    s_o, isum_o, lse_o, empty = O.attn_scores(lay, q, k, Hq, Hkv, scale, dt)

    dl = A.DeviceLayout(lay)
    qd, kd = to_dev(q, dt), to_dev(k, dt)
    tol = TOL[dt]
    vis = lay.visual_mask()
    # which sequences hold an image with no text row after it
    flagged = {int(np.searchsorted(lay.cu_img, i, side="right") - 1) for i in empty}

    if lay.T_tot:
        lse_g = A.row_lse(dl, qd, kd, scale).cpu().numpy().astype(np.float64)
        assert_rel(lse_g, lse_o, 0.0, "row lse", abs_floor=tol)
    lse_sup = torch.from_numpy(np.ascontiguousarray(lse_o, dtype=np.float32)).cuda()
    for row_lse in (None, lse_sup):
        status = torch.zeros(lay.B, dtype=torch.int32, device="cuda")
        s_g, isum_g = A.score_attn(dl, qd, kd, scale, row_lse=row_lse, status=status)
        s_g, isum_g = s_g.cpu().numpy(), isum_g.cpu().numpy()
        what = "given lse" if row_lse is not None else "two passes"
        assert_rel(s_g[vis], s_o[vis], tol, f"scores ({what})", abs_floor=1e-30)
        assert np.all(np.isinf(s_g[~vis]) & (s_g[~vis] > 0))
        if lay.n_img:
            assert_rel(isum_g, isum_o, tol, f"image sums ({what})", abs_floor=1e-30)
        st = status.cpu().numpy()
        got = {b for b in range(lay.B) if st[b] & A.FLAG_NO_TEXT_AFTER}
        assert got == flagged, (got, flagged)
        assert not np.any(st & ~A.FLAG_NO_TEXT_AFTER)
        for i in empty:
            s0, n = int(lay.img_start[i]), int(lay.img_len[i])
            assert np.all(s_g[s0:s0 + n] == 0.0)


def test_batch_without_text_rows():
    # no text row anywhere: no query to read, every visual score 0 and every
    # sequence with a non-empty image flagged
    from paper_2608_26806_amd.workloads import build_layout
    lay = build_layout([[6, 0, 40], [], [300]], 0, 0, 50)   # the middle sequence is empty
    assert lay.T_tot == 0
    dl = A.DeviceLayout(lay)
    k = torch.randn(lay.N_tok, 2, 128, device="cuda").to(torch.bfloat16)
    q = torch.empty(0, 4, 128, device="cuda", dtype=torch.bfloat16)
    status = torch.zeros(lay.B, dtype=torch.int32, device="cuda")
    s_g, isum_g = A.score_attn(dl, q, k, 128 ** -0.5, status=status)
    assert A.row_lse(dl, q, k, 128 ** -0.5).numel() == 0
    torch.cuda.synchronize()
    s_g = s_g.cpu().numpy()
    vis = lay.visual_mask()
    assert np.all(s_g[vis] == 0.0) and np.all(np.isinf(s_g[~vis]))
    assert np.all(isum_g.cpu().numpy() == 0.0)
    s_o, isum_o, _, empty = O.attn_scores(lay, np.zeros((0, 4, 128), np.uint16),
                                          np.zeros((lay.N_tok, 2, 128), np.uint16), 4, 2,
                                          128 ** -0.5, "bf16")
    assert np.all(s_o[vis] == 0.0) and empty == {0, 2, 3}
    assert [int(x) for x in status.cpu().numpy()] == [A.FLAG_NO_TEXT_AFTER, 0, A.FLAG_NO_TEXT_AFTER]


def _large_random_layout(rng):
    """Up to 3 sequences of up to 11 images of up to 3,000 tokens, text between
    the images and up to 700 text rows after them."""
    cu_seqlens, img_start, img_len, cu_img, text_pos, cu_text = [0], [], [], [0], [], [0]
    pos = 0
    for _ in range(int(rng.integers(1, 4))):
        for _ in range(int(rng.integers(1, 12))):
            nt = int(rng.integers(0, 20))
            text_pos.extend(range(pos, pos + nt))
            pos += nt
            n = int(rng.integers(1, 3000))
            img_start.append(pos)
            img_len.append(n)
            pos += n
        nt = int(rng.integers(1, 700))
        text_pos.extend(range(pos, pos + nt))
        pos += nt
        cu_seqlens.append(pos)
        cu_img.append(len(img_len))
        cu_text.append(len(text_pos))
    a = lambda v: np.asarray(v, dtype=np.int32)
    return Layout(a(cu_seqlens), a(img_start), a(img_len), a(cu_img), a(text_pos), a(cu_text),
                  np.zeros(len(cu_seqlens) - 1, np.int32))


@pytest.mark.parametrize("seed", range(3))
def test_large_random_layout_scores(seed):
    # tens of thousands of tokens, hundreds to thousands of text rows and up
    # to 56 query heads: many key chunks, multi-stage query splits
    from concurrent.futures import ThreadPoolExecutor
    rng = np.random.default_rng(7000 + seed)
    lay = _large_random_layout(rng)
    Hkv = int(rng.choice([2, 4, 8]))
    Hq = Hkv * int(rng.choice([1, 4, 7]))
    d = 128
    q = f32_to_bf16_bits(rng.standard_normal((lay.T_tot, Hq, d)).astype(np.float32))
    k = f32_to_bf16_bits((rng.standard_normal((lay.N_tok, Hkv, d)) * 1.3).astype(np.float32))
    say(f"[large random scores] seed {seed}: B={lay.B} images={lay.n_img} N_tok={lay.N_tok} "
        f"T={lay.T_tot} Hq={Hq} Hkv={Hkv}")

    def one(b):
        return O.attn_scores(lay, q, k, Hq, Hkv, d ** -0.5, "bf16", seqs=[b])

    with ThreadPoolExecutor(max_workers=min(8, lay.B)) as ex:
        parts = list(ex.map(one, range(lay.B)))
    s_o, isum_o = np.full(lay.N_tok, np.inf), np.zeros(lay.n_img)
    lse_o = np.zeros((Hq, lay.T_tot))
    for b, (sb, ib, lb, _) in enumerate(parts):
        s0, s1 = int(lay.cu_seqlens[b]), int(lay.cu_seqlens[b + 1])
        i0, i1 = int(lay.cu_img[b]), int(lay.cu_img[b + 1])
        t0, t1 = int(lay.cu_text[b]), int(lay.cu_text[b + 1])
        s_o[s0:s1], isum_o[i0:i1], lse_o[:, t0:t1] = sb[s0:s1], ib[i0:i1], lb[:, t0:t1]
    dl = A.DeviceLayout(lay)
    qd, kd = to_dev(q, "bf16"), to_dev(k, "bf16")
    lse_g = A.row_lse(dl, qd, kd, d ** -0.5).cpu().numpy().astype(np.float64)
    s_g, isum_g = A.score_attn(dl, qd, kd, d ** -0.5)
    vis = lay.visual_mask()
    assert_rel(lse_g, lse_o, 0.0, "row lse", abs_floor=TOL["bf16"])
    assert_rel(s_g.cpu().numpy()[vis], s_o[vis], TOL["bf16"], "scores", abs_floor=1e-30)
    assert_rel(isum_g.cpu().numpy(), isum_o, TOL["bf16"], "image sums", abs_floor=1e-30)
