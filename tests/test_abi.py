"""The C ABI on the CPU: the library loads, exports every declared symbol, and
rejects bad arguments on the host before anything is launched.

Every call here fails validation, so no kernel is ever enqueued (there is no
GPU in this test); the device pointers of the layout are host memory that the
library never dereferences.
"""
import ctypes

import numpy as np
import pytest
import torch

from paper_2608_26806_amd import avtp as A
from paper_2608_26806_amd.workloads import build_layout


def _dl(lay=None, **patch):
    lay = lay or build_layout([[6, 4], [5]], 2, 3, 50)
    arrays = {n: np.array(getattr(lay, n)) for n in A.DeviceLayout.NAMES}
    arrays.update(patch)
    return A.DeviceLayout(arrays, host_only=True)


def _call_score(dl, d=128, Hq=4, Hkv=2, ws_bytes=None, dtype=A.BF16, scale=0.1):
    buf = torch.zeros(1 << 16, dtype=torch.uint8)
    p = ctypes.c_void_p(buf.data_ptr())
    n = buf.numel() if ws_bytes is None else ws_bytes
    return A.lib().avtp_score(None, dl.ref(), A.SCORE_ATTN, dtype, p, p, Hq, Hkv, d, scale, None,
                              None, None, 0, p, p, None, p, n)


def test_exports_every_declared_function():
    lib = A.lib()
    names = A.header_functions()
    assert {"avtp_score", "avtp_budget", "avtp_select", "avtp_compact"} <= set(names)
    for n in names:
        assert hasattr(lib, n), n
    assert lib.avtp_version() >> 16 == 1


def test_status_strings():
    for code in (0, -1, -2, -3, -4, -5):
        assert A.status_string(code).startswith("AVTP_")


def test_null_layout_and_bad_offsets():
    lib = A.lib()
    buf = torch.zeros(64, dtype=torch.uint8)
    p = ctypes.c_void_p(buf.data_ptr())
    assert lib.avtp_select(None, None, p, p, p, 100, p, None) == A.ERR_INVALID_ARG
    bad = _dl(cu_seqlens=np.array([1, 17, 25]))
    assert _call_score(bad) == A.ERR_INVALID_ARG


def test_overlapping_images_rejected():
    lay = build_layout([[6, 4]], 1, 2, 50)
    st = np.array(lay.img_start)
    st[1] = st[0] + 3                               # image 1 starts inside image 0
    assert _call_score(_dl(lay, img_start=st)) == A.ERR_INVALID_ARG


def test_text_inside_image_rejected():
    lay = build_layout([[6, 4]], 1, 2, 50)
    tp = np.array(lay.text_pos)
    tp[0] = lay.img_start[0] + 1
    tp.sort()
    assert _call_score(_dl(lay, text_pos=tp)) == A.ERR_INVALID_ARG


def test_uncovered_token_rejected():
    lay = build_layout([[6, 4]], 1, 2, 50)
    ln = np.array(lay.img_len)
    ln[1] -= 1                                      # the last image token belongs to nothing
    assert _call_score(_dl(lay, img_len=ln)) == A.ERR_INVALID_ARG


def test_head_and_dtype_checks():
    dl = _dl()
    assert _call_score(dl, d=96) == A.ERR_UNSUPPORTED
    assert _call_score(dl, Hq=6, Hkv=4) == A.ERR_INVALID_ARG
    assert _call_score(dl, dtype=7) == A.ERR_UNSUPPORTED
    assert _call_score(dl, scale=float("nan")) == A.ERR_INVALID_ARG


def test_workspace_checks():
    dl = _dl()
    need = A.score_workspace_bytes(dl, A.SCORE_ATTN, A.BF16, 4, 2, 128)
    assert need > 0
    assert _call_score(dl, ws_bytes=need - 1) == A.ERR_WORKSPACE
    bad = _dl(cu_seqlens=np.array([0, 5, 7]))
    assert A.score_workspace_bytes(bad, A.SCORE_ATTN, A.BF16, 4, 2, 128) == 0


def test_budget_infeasible_and_bad_alpha():
    lay = build_layout([[20, 20]], 0, 1, 50)
    buf = torch.zeros(64, dtype=torch.uint8)
    p = ctypes.c_void_p(buf.data_ptr())
    lib = A.lib()
    dl = _dl(lay, keep_total=np.array([39]))        # sum hi = 38 < 39
    assert lib.avtp_budget(None, dl.ref(), p, 0, 1.0, 50, 950, 0, p, None) == A.ERR_INFEASIBLE
    dl = _dl(lay, keep_total=np.array([10]))
    assert lib.avtp_budget(None, dl.ref(), p, 0, 1.0, 50, 950, 8, p, None) == A.ERR_INFEASIBLE
    assert lib.avtp_budget(None, dl.ref(), p, 0, -1.0, 50, 950, 0, p, None) == A.ERR_INVALID_ARG
    assert lib.avtp_budget(None, dl.ref(), p, 0, 1.0, 600, 500, 0, p, None) == A.ERR_INVALID_ARG
    assert lib.avtp_budget(None, dl.ref(), p, 5, 1.0, 50, 950, 0, p, None) == A.ERR_INVALID_ARG


def test_select_capacity_checked():
    dl = _dl()
    buf = torch.zeros(64, dtype=torch.uint8)
    p = ctypes.c_void_p(buf.data_ptr())
    assert A.lib().avtp_select(None, dl.ref(), p, p, p, dl.N_out - 1, p, None) == A.ERR_INVALID_ARG


def test_compact_descriptor_checks():
    dl = _dl()
    src = torch.zeros((dl.N_tok, 8), dtype=torch.float32)
    dst = torch.zeros((dl.N_out, 8), dtype=torch.float32)
    keep = torch.zeros(dl.N_out, dtype=torch.int32)
    lib = A.lib()
    d = A.tensor_desc(src, dst)
    arr = (A._Tensor * 9)(*([d] * 9))
    assert lib.avtp_compact(None, dl.ref(), ctypes.c_void_p(keep.data_ptr()), dl.N_out, arr, 9) \
        == A.ERR_UNSUPPORTED
    d.src_stride = 4                                  # stride below the row size
    arr = (A._Tensor * 1)(d)
    assert lib.avtp_compact(None, dl.ref(), ctypes.c_void_p(keep.data_ptr()), dl.N_out, arr, 1) \
        == A.ERR_INVALID_ARG
    d = A.tensor_desc(src, dst)
    arr = (A._Tensor * 1)(d)
    assert lib.avtp_compact(None, dl.ref(), ctypes.c_void_p(keep.data_ptr()), dl.N_out + 1, arr, 1) \
        == A.ERR_INVALID_ARG


def test_layout_limits():
    lay = build_layout([[1] * 257], 0, 1, 50)         # more images per sequence than supported
    assert _call_score(_dl(lay)) == A.ERR_UNSUPPORTED


def test_layer_selection_arguments_rejected_on_host():
    lib = A.lib()
    buf = torch.zeros(64, dtype=torch.uint8)
    p = ctypes.c_void_p(buf.data_ptr())
    assert lib.avtp_layer_select(None, None, 4, 3, 2, p, p) == A.ERR_INVALID_ARG   # no table
    assert lib.avtp_layer_select(None, p, 0, 3, 1, p, p) == A.ERR_INVALID_ARG      # L = 0
    assert lib.avtp_layer_select(None, p, 1025, 3, 1, p, p) == A.ERR_INVALID_ARG   # L > max
    assert lib.avtp_layer_select(None, p, 4, 0, 1, p, p) == A.ERR_INVALID_ARG      # N = 0
    assert lib.avtp_layer_select(None, p, 4, 3, 5, p, p) == A.ERR_INVALID_ARG      # k > L
    assert lib.avtp_layer_select(None, p, 4, 3, 0, p, p) == A.ERR_INVALID_ARG      # k = 0
    assert lib.avtp_layer_attention(None, None, p, p) == A.ERR_INVALID_ARG         # no layout
    assert lib.avtp_layer_attention(None, _dl().ref(), p, None) == A.ERR_INVALID_ARG


def test_pruned_layout_arguments_rejected_on_host():
    lib = A.lib()
    buf = torch.zeros(256, dtype=torch.uint8)
    p = ctypes.c_void_p(buf.data_ptr())
    dl = _dl()
    assert lib.avtp_pruned_layout(None, None, p, p, p, p, p, p, p, p) == A.ERR_INVALID_ARG
    assert lib.avtp_pruned_layout(None, dl.ref(), p, None, p, p, p, p, p, p) == A.ERR_INVALID_ARG
    assert lib.avtp_pruned_layout(None, dl.ref(), None, p, p, p, p, p, p, p) == A.ERR_INVALID_ARG
    assert lib.avtp_pruned_layout(None, dl.ref(), p, p, p, None, p, p, p, p) == A.ERR_INVALID_ARG
    assert lib.avtp_pruned_layout(None, dl.ref(), p, p, p, p, p, p, None, p) == A.ERR_INVALID_ARG


def test_select_compact_arguments_rejected_on_host():
    lib = A.lib()
    buf = torch.zeros(256, dtype=torch.uint8)
    p = ctypes.c_void_p(buf.data_ptr())
    dl = _dl()
    t = (A._Tensor * 1)()
    assert lib.avtp_select_compact(None, None, p, p, p, 100, p, None, t, 0) == A.ERR_INVALID_ARG
    assert lib.avtp_select_compact(None, dl.ref(), None, p, p, 100, p, None, t, 0) == A.ERR_INVALID_ARG
    assert lib.avtp_select_compact(None, dl.ref(), p, p, p, 1, p, None, t, 0) == A.ERR_INVALID_ARG  # capacity
    assert lib.avtp_select_compact(None, dl.ref(), p, p, p, 100, p, None, t, 9) == A.ERR_UNSUPPORTED
    assert lib.avtp_select_compact(None, dl.ref(), p, p, p, 100, p, None, t, 1) == A.ERR_INVALID_ARG  # null src


def test_budget_select_compact_arguments_rejected_on_host():
    """The one-call budget + selection + compaction checks the arguments of
    all three calls, feasibility included, before any launch."""
    lib = A.lib()
    buf = torch.zeros(256, dtype=torch.uint8)
    p = ctypes.c_void_p(buf.data_ptr())
    t = (A._Tensor * 1)()
    f = lib.avtp_budget_select_compact
    lay = build_layout([[20, 20]], 2, 1, 50)
    dl = _dl(lay)
    ok = (p, 0, 1.0, 50, 950, 0, p, p, p, 100, p, None, t, 0)   # img_sum .. n_tensors
    assert f(None, None, *ok) == A.ERR_INVALID_ARG
    assert f(None, _dl(lay, keep_total=np.array([39])).ref(), *ok) == A.ERR_INFEASIBLE  # sum hi 38
    assert f(None, _dl(lay, keep_total=np.array([10])).ref(),
             p, 0, 1.0, 50, 950, 8, *ok[6:]) == A.ERR_INFEASIBLE                      # floors 16
    bad = [(2, -1.0), (2, 33.0), (1, 5), (3, 960)]                 # alpha, mode, lo > hi
    for pos, val in bad:
        args = list(ok)
        args[pos] = val
        assert f(None, dl.ref(), *args) == A.ERR_INVALID_ARG, (pos, val)
    for pos in (0, 6, 7, 10):                                      # img_sum, scores, budget, cu_out
        args = list(ok)
        args[pos] = None
        assert f(None, dl.ref(), *args) == A.ERR_INVALID_ARG, pos
    args = list(ok)
    args[9] = dl.N_out - 1                                         # keep capacity
    assert f(None, dl.ref(), *args) == A.ERR_INVALID_ARG
    args = list(ok)
    args[13] = 9
    assert f(None, dl.ref(), *args) == A.ERR_UNSUPPORTED          # too many tensors
    args[13] = 1
    assert f(None, dl.ref(), *args) == A.ERR_INVALID_ARG          # null src


def test_score_rejects_sequences_past_the_32bit_offset_range():
    """The score kernels address a sequence's keys and text-row queries with
    32-bit byte offsets; longer sequences are rejected on the host."""
    lib = A.lib()
    buf = torch.zeros(1 << 16, dtype=torch.uint8)
    p = ctypes.c_void_p(buf.data_ptr())
    big = _dl(build_layout([[300000]], 0, 10, 10))    # 300,010 tokens

    def call(dl, Hq, Hkv, ws_bytes=1 << 16):
        return lib.avtp_score(None, dl.ref(), A.SCORE_ATTN, A.BF16, p, p, Hq, Hkv, 128, 0.1, None,
                              None, None, 0, p, p, None, p, ws_bytes)

    # keys: 300,010 * 64 heads * 256 B = 4.9 GB >= 4 GiB
    assert call(big, 64, 64) == A.ERR_UNSUPPORTED
    assert A.score_workspace_bytes(big, A.SCORE_ATTN, A.BF16, 64, 64, 128) == 0
    assert lib.avtp_row_lse(None, big.ref(), A.BF16, p, p, 64, 64, 128, 0.1, p, p, 1 << 16) \
        == A.ERR_UNSUPPORTED
    # 8 key heads: 614 MB, accepted (then the workspace is too small)
    assert A.score_workspace_bytes(big, A.SCORE_ATTN, A.BF16, 64, 8, 128) > (1 << 16)
    assert call(big, 64, 8) == A.ERR_WORKSPACE
    # text-row queries: 70,000 rows * 256 heads * 256 B = 4.6 GB
    text = _dl(build_layout([[16]], 0, 70000, 10))
    assert call(text, 256, 8) == A.ERR_UNSUPPORTED


def test_noalloc_rejects_oversize_and_bad_args_on_the_host():
    """avtp_score_noalloc checks every argument, and that the layout fits its
    scratch, before any HIP call (so this runs without a GPU)."""
    lib = A.lib()
    buf = torch.zeros(1 << 16, dtype=torch.uint8)
    p = ctypes.c_void_p(buf.data_ptr())
    # one 200k-token image, 64 key heads: the column-sum planes alone need 51 MB
    big = _dl(build_layout([[200000]], 0, 8, 10))
    need = A.score_workspace_bytes(big, A.SCORE_ATTN, A.BF16, 64, 64, 128)
    assert need > A.NOALLOC_MAX_WORKSPACE
    rc = lib.avtp_score_noalloc(None, big.ref(), A.SCORE_ATTN, A.BF16, p, p, 64, 64, 128, 0.1,
                                None, None, None, 0, p, p, None)
    assert rc == A.ERR_WORKSPACE
    small = _dl()
    for args, want in [((4, 2, 96), A.ERR_UNSUPPORTED), ((4, 3, 128), A.ERR_INVALID_ARG)]:
        Hq, Hkv, d = args
        rc = lib.avtp_score_noalloc(None, small.ref(), A.SCORE_ATTN, A.BF16, p, p, Hq, Hkv, d, 0.1,
                                    None, None, None, 0, p, p, None)
        assert rc == want
    rc = lib.avtp_score_noalloc(None, small.ref(), A.SCORE_ATTN, A.BF16, p, p, 4, 2, 128, 0.1,
                                None, None, None, 0, None, p, None)
    assert rc == A.ERR_INVALID_ARG


def test_binding_rejects_host_tensors_and_mismatched_shapes():
    # the binding checks what the C ABI cannot see in a bare pointer, before
    # calling it: a host tensor handed to a kernel would be read as device
    # memory (a raw stream handle keeps torch's GPU state out of this test)
    dl = _dl()
    raw = ctypes.c_void_p(0)
    with pytest.raises(ValueError, match="GPU tensor"):
        A.budget(dl, torch.zeros(dl.n_img), 1.0, stream=raw)
    with pytest.raises(ValueError, match="GPU tensor"):
        A.select(dl, torch.zeros(dl.N_tok), torch.zeros(dl.n_img, dtype=torch.int32), stream=raw)
    q = torch.zeros(dl.T_tot - 1, 4, 128, dtype=torch.bfloat16)     # one text row too few
    k = torch.zeros(dl.N_tok, 2, 128, dtype=torch.bfloat16)
    with pytest.raises(ValueError, match="text rows"):
        A.score_attn(dl, q, k, 0.1, scores=torch.zeros(dl.N_tok), img_sum=torch.zeros(dl.n_img),
                     ws=torch.zeros(1, dtype=torch.uint8), stream=raw)
    with pytest.raises(TypeError, match="dtype"):
        A.row_lse(dl, torch.zeros(dl.T_tot, 4, 128, dtype=torch.bfloat16), k.float(), 0.1,
                  out=torch.zeros(4, dl.T_tot),
                  ws=torch.zeros(1, dtype=torch.uint8), stream=raw)
    src = torch.zeros(dl.N_tok, 8)
    with pytest.raises(ValueError, match="on the GPU"):
        A.compact(dl, torch.zeros(dl.N_out, dtype=torch.int32), [(src, torch.zeros(dl.N_out, 8))],
                  stream=raw)


def test_row_lse_without_text_rows_needs_no_query_pointer():
    # a batch with no text rows: nothing is read or written through q_text and
    # row_lse_out (an empty tensor may have no address), and nothing is launched
    lay = build_layout([[6, 4], [5]], 0, 0, 50)
    assert lay.T_tot == 0
    dl = _dl(lay)
    buf = torch.zeros(1 << 16, dtype=torch.uint8)
    ws = ctypes.c_void_p((buf.data_ptr() + 255) // 256 * 256)
    k = ctypes.c_void_p(ws.value)
    rc = A.lib().avtp_row_lse(None, dl.ref(), A.BF16, None, k, 4, 2, 128, 0.1, None, ws,
                              buf.numel() - 256)
    assert rc == A.OK
    # with text rows the same null pointers are rejected
    assert A.lib().avtp_row_lse(None, _dl().ref(), A.BF16, None, k, 4, 2, 128, 0.1, None, ws,
                                buf.numel() - 256) == A.ERR_INVALID_ARG


def test_empty_layout_arrays_may_be_null():
    # arrays of length 0 need no address: the image arrays of a text-only
    # batch, text_pos of a batch without text rows, a compaction's destination
    # when no row is kept
    lib = A.lib()

    def layout(lay, null):
        dl = _dl(lay)
        for n in null:
            setattr(dl.st, n, None)
            setattr(dl.st, "h_" + n, None)
        return dl

    text_only = build_layout([[], []], 0, 3, 50)
    assert text_only.n_img == 0
    dl = layout(text_only, ("img_start", "img_len"))
    assert A.score_workspace_bytes(dl, A.SCORE_ATTN, A.BF16, 4, 2, 128) > 0
    images_only = build_layout([[7, 5]], 0, 0, 50)
    assert images_only.T_tot == 0
    dl = layout(images_only, ("text_pos",))
    assert A.score_workspace_bytes(dl, A.SCORE_ATTN, A.BF16, 4, 2, 128) > 0
    # the same nulls with arrays that are not empty are rejected
    assert A.score_workspace_bytes(layout(build_layout([[7]], 1, 1, 50), ("text_pos",)),
                                   A.SCORE_ATTN, A.BF16, 4, 2, 128) == 0
    assert A.score_workspace_bytes(layout(build_layout([[7]], 1, 1, 50), ("img_len",)),
                                   A.SCORE_ATTN, A.BF16, 4, 2, 128) == 0
    # nothing kept: nothing is copied and no destination is needed
    none_kept = build_layout([[6, 4]], 0, 0, 0)
    dl = _dl(none_kept)
    assert dl.N_out == 0
    buf = torch.zeros(64, dtype=torch.uint8)
    t = A._Tensor(buf.data_ptr(), None, 4, 4, 4, 1, 0, 0)
    assert lib.avtp_compact(None, dl.ref(), None, 0, ctypes.byref(t), 1) == A.OK
    t.src = None
    assert lib.avtp_compact(None, dl.ref(), None, 0, ctypes.byref(t), 1) == A.ERR_INVALID_ARG
