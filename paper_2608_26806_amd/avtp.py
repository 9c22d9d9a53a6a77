"""ctypes binding of libavtp.so (argument marshalling only).

Every step of the pruning layer runs in the library's HIP kernels; this module
turns torch tensors into device pointers, passes torch's current HIP stream,
and raises ``AvtpError`` on a non-zero status.  There is no fallback: if the
library is missing, loading it raises.
"""
from __future__ import annotations

import ctypes
import os
import re
from typing import Optional, Sequence

import numpy as np
import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
# AVTP_LIBRARY names another build of the same library (e.g. the host-sanitized
# one the CPU tests check the validation layer with)
LIB_PATH = os.environ.get("AVTP_LIBRARY") or os.path.join(_HERE, "libavtp.so")
HEADER_PATH = os.path.join(os.path.dirname(_HERE), "include", "avtp.h")

BF16, FP32 = 0, 1
SCORE_ATTN, SCORE_VARIATION = 0, 1
BUDGET_PROPORTIONAL, BUDGET_RAW = 0, 1
FLAG_NAN_SCORE, FLAG_NO_TEXT_AFTER, FLAG_INFEASIBLE, FLAG_OUT_CAPACITY = 1, 2, 4, 8
OK, ERR_INVALID_ARG, ERR_UNSUPPORTED, ERR_INFEASIBLE, ERR_WORKSPACE, ERR_HIP = 0, -1, -2, -3, -4, -5
NOALLOC_MAX_WORKSPACE = 16 << 20   # AVTP_NOALLOC_MAX_WORKSPACE of include/avtp.h

_i32p = ctypes.POINTER(ctypes.c_int32)


class _Layout(ctypes.Structure):
    _fields_ = [("B", ctypes.c_int32), ("n_img", ctypes.c_int32), ("N_tok", ctypes.c_int32),
                ("T_tot", ctypes.c_int32)] + \
               [(n, ctypes.c_void_p) for n in ("cu_seqlens", "img_start", "img_len", "cu_img",
                                                "text_pos", "cu_text", "keep_total")] + \
               [(n, ctypes.c_void_p) for n in ("h_cu_seqlens", "h_img_start", "h_img_len",
                                                "h_cu_img", "h_text_pos", "h_cu_text",
                                                "h_keep_total")]


class _Tensor(ctypes.Structure):
    _fields_ = [("src", ctypes.c_void_p), ("dst", ctypes.c_void_p), ("row_bytes", ctypes.c_int64),
                ("src_stride", ctypes.c_int64), ("dst_stride", ctypes.c_int64),
                ("planes", ctypes.c_int32), ("src_plane_stride", ctypes.c_int64),
                ("dst_plane_stride", ctypes.c_int64)]


class AvtpError(RuntimeError):
    def __init__(self, code: int, where: str):
        self.code = code
        super().__init__(f"{where}: {status_string(code)} ({code})")


_lib = None


def lib() -> ctypes.CDLL:
    """Load libavtp.so (raises if it was not built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing; build it with "
                               "`python -m paper_2608_26806_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        vp, c_int, c_float, sz = ctypes.c_void_p, ctypes.c_int, ctypes.c_float, ctypes.c_size_t
        LP = ctypes.POINTER(_Layout)
        L.avtp_score_workspace_size.argtypes = [LP, c_int, c_int, c_int, c_int, c_int]
        L.avtp_score_workspace_size.restype = sz
        L.avtp_score.argtypes = [vp, LP, c_int, c_int, vp, vp, c_int, c_int, c_int, c_float, vp, vp,
                                 vp, c_int, vp, vp, vp, vp, sz]
        L.avtp_row_lse.argtypes = [vp, LP, c_int, vp, vp, c_int, c_int, c_int, c_float, vp, vp, sz]
        L.avtp_score_noalloc.argtypes = [vp, LP, c_int, c_int, vp, vp, c_int, c_int, c_int, c_float,
                                         vp, vp, vp, c_int, vp, vp, vp]
        L.avtp_budget.argtypes = [vp, LP, vp, c_int, c_float, c_int, c_int, c_int, vp, vp]
        L.avtp_select.argtypes = [vp, LP, vp, vp, vp, ctypes.c_int64, vp, vp]
        L.avtp_compact.argtypes = [vp, LP, vp, ctypes.c_int64, ctypes.POINTER(_Tensor), c_int]
        L.avtp_pruned_layout.argtypes = [vp, LP, vp, vp, vp, vp, vp, vp, vp, vp]
        L.avtp_select_compact.argtypes = [vp, LP, vp, vp, vp, ctypes.c_int64, vp, vp,
                                          ctypes.POINTER(_Tensor), c_int]
        L.avtp_budget_select_compact.argtypes = [vp, LP, vp, c_int, ctypes.c_float, c_int, c_int,
                                                 c_int, vp, vp, vp, ctypes.c_int64, vp, vp,
                                                 ctypes.POINTER(_Tensor), c_int]
        L.avtp_layer_attention.argtypes = [vp, LP, vp, vp]
        L.avtp_layer_select.argtypes = [vp, vp, c_int, c_int, c_int, vp, vp]
        L.avtp_status_string.argtypes = [c_int]
        L.avtp_status_string.restype = ctypes.c_char_p
        L.avtp_version.restype = c_int
        for f in ("avtp_score", "avtp_score_noalloc", "avtp_row_lse", "avtp_budget", "avtp_select",
                  "avtp_compact",
                  "avtp_layer_attention", "avtp_layer_select", "avtp_pruned_layout",
                  "avtp_select_compact", "avtp_budget_select_compact"):
            getattr(L, f).restype = c_int
        _lib = L
    return _lib


def header_functions() -> list:
    """Names of the functions include/avtp.h declares."""
    text = open(HEADER_PATH).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(avtp_[a-z_]+)\s*\(", text)))


def status_string(code: int) -> str:
    return lib().avtp_status_string(int(code)).decode()


def _check(rc: int, where: str) -> None:
    if rc != OK:
        raise AvtpError(rc, where)


def _arg(t: Optional[torch.Tensor], name: str, numel: int = 0, dtype=None):
    """Device pointer of tensor argument ``name``, after the checks the C ABI
    cannot make (it receives bare pointers): on the GPU, contiguous, of the
    expected dtype and with at least ``numel`` elements, since a kernel would
    otherwise read or write a host tensor or a short buffer out of bounds.
    None passes through (optional arguments)."""
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError(f"{name}: a GPU tensor is needed, got one on {t.device}")
    if not t.is_contiguous():
        raise ValueError(f"{name}: a contiguous tensor is needed")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{name}: {dtype} is needed, got {t.dtype}")
    if t.numel() < numel:
        raise ValueError(f"{name}: at least {numel} elements are needed, got {t.numel()}")
    return ctypes.c_void_p(t.data_ptr())


def _check_qk(dl: "DeviceLayout", q_text: torch.Tensor, k: torch.Tensor) -> None:
    """q_text [T_tot, Hq, d] and k [N_tok, Hkv, d] of one dtype (more rows are
    allowed: the kernels read rows below T_tot and N_tok only)."""
    if q_text.dim() != 3 or k.dim() != 3 or q_text.shape[2] != k.shape[2]:
        raise ValueError("q_text must be [T_tot, Hq, d] and k [N_tok, Hkv, d]")
    if q_text.shape[0] < dl.T_tot or k.shape[0] < dl.N_tok:
        raise ValueError(f"q_text has {q_text.shape[0]} rows and k {k.shape[0]}; the layout has "
                         f"{dl.T_tot} text rows and {dl.N_tok} tokens")
    if q_text.dtype != k.dtype:
        raise TypeError(f"q_text ({q_text.dtype}) and k ({k.dtype}) differ in dtype")


def _stream(stream=None):
    """The HIP stream handle: torch's current stream by default; a torch
    stream, or a raw handle (ctypes.c_void_p) passed through as is."""
    if isinstance(stream, ctypes.c_void_p):
        return stream
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return BF16
    if t.dtype == torch.float32:
        return FP32
    raise TypeError(f"unsupported dtype {t.dtype}")


class DeviceLayout:
    """A packed batch layout with device arrays and their host mirrors.

    ``arrays`` maps cu_seqlens, img_start, img_len, cu_img, text_pos, cu_text,
    keep_total to int32 sequences (an object with those attributes works too).
    """

    NAMES = ("cu_seqlens", "img_start", "img_len", "cu_img", "text_pos", "cu_text", "keep_total")

    def __init__(self, arrays, device="cuda", host_only: bool = False):
        get = (lambda n: arrays[n]) if isinstance(arrays, dict) else (lambda n: getattr(arrays, n))
        self.host = {n: np.ascontiguousarray(np.asarray(get(n), dtype=np.int32)) for n in self.NAMES}
        h = self.host
        self.B = len(h["cu_seqlens"]) - 1
        self.n_img = len(h["img_len"])
        self.N_tok = int(h["cu_seqlens"][-1]) if self.B >= 0 and len(h["cu_seqlens"]) else 0
        self.T_tot = len(h["text_pos"])
        self.N_out = int(self.T_tot + int(np.sum(h["keep_total"], dtype=np.int64)))
        # one device buffer holds every array (a zero-length array still gets a valid pointer)
        offs, tot = {}, 0
        for n in self.NAMES:
            offs[n] = tot
            tot += max(1, len(h[n]))
        flat = np.zeros(tot, dtype=np.int32)
        for n in self.NAMES:
            flat[offs[n]:offs[n] + len(h[n])] = h[n]
        if host_only:
            self.dev = torch.from_numpy(flat)
        else:
            self.dev = torch.from_numpy(flat).to(device)
        base, es = self.dev.data_ptr(), 4
        self.st = _Layout(self.B, self.n_img, self.N_tok, self.T_tot,
                          *[base + es * offs[n] for n in self.NAMES],
                          *[h[n].ctypes.data for n in self.NAMES])

    def ref(self):
        return ctypes.byref(self.st)

    def device_array(self, name: str) -> torch.Tensor:
        h = self.host[name]
        off = self.st.__getattribute__(name) - self.dev.data_ptr()
        return self.dev[off // 4: off // 4 + len(h)]


# --------------------------------------------------------------------------- score
def score_workspace_bytes(dl: DeviceLayout, mode: int, dtype: int = BF16, Hq: int = 1,
                          Hkv: int = 1, d: int = 128) -> int:
    return int(lib().avtp_score_workspace_size(dl.ref(), mode, dtype, Hq, Hkv, d))


def alloc_workspace(nbytes: int, device="cuda") -> torch.Tensor:
    return torch.empty(max(1, nbytes), dtype=torch.uint8, device=device)


def row_lse(dl: DeviceLayout, q_text: torch.Tensor, k: torch.Tensor, softmax_scale: float,
            out: Optional[torch.Tensor] = None, ws: Optional[torch.Tensor] = None,
            stream=None) -> torch.Tensor:
    T, Hq, d = q_text.shape
    Hkv = k.shape[1]
    dt = dtype_code(q_text)
    if out is None:
        out = torch.empty((Hq, T), dtype=torch.float32, device=q_text.device)
    if ws is None:
        ws = alloc_workspace(score_workspace_bytes(dl, SCORE_ATTN, dt, Hq, Hkv, d), q_text.device)
    _check_qk(dl, q_text, k)
    _check(lib().avtp_row_lse(_stream(stream), dl.ref(), dt, _arg(q_text, "q_text"),
                              _arg(k, "k"), Hq, Hkv, d, float(softmax_scale),
                              _arg(out, "out", Hq * dl.T_tot, torch.float32),
                              _arg(ws, "ws", 0, torch.uint8), ws.numel()), "avtp_row_lse")
    return out


class Prepared:
    """One C ABI call with its arguments marshalled once: calling it issues the
    call again on the same buffers (for loops that repeat a call, where the
    per-call Python work would otherwise be a large part of a small layer's
    time).  It keeps the objects the arguments point into alive."""

    def __init__(self, fn, args: tuple, where: str, keep: tuple):
        self._fn, self._args, self._where, self._keep = fn, args, where, keep

    def __call__(self) -> None:
        rc = self._fn(*self._args)
        if rc != OK:
            raise AvtpError(rc, self._where)


def prepare_score_attn(dl: DeviceLayout, q_text: torch.Tensor, k: torch.Tensor,
                       softmax_scale: float, scores: torch.Tensor, img_sum: torch.Tensor,
                       ws: torch.Tensor, row_lse: Optional[torch.Tensor] = None,
                       status: Optional[torch.Tensor] = None, stream=None) -> Prepared:
    """avtp_score (attention mode) on fixed buffers, as a Prepared call."""
    T, Hq, d = q_text.shape
    _check_qk(dl, q_text, k)
    args = (_stream(stream), dl.ref(), SCORE_ATTN, dtype_code(q_text), _arg(q_text, "q_text"),
            _arg(k, "k"), Hq, k.shape[1], d, float(softmax_scale),
            _arg(row_lse, "row_lse", Hq * dl.T_tot, torch.float32), None, None, 0,
            _arg(scores, "scores", dl.N_tok, torch.float32),
            _arg(img_sum, "img_sum", dl.n_img, torch.float32),
            _arg(status, "status", dl.B, torch.int32), _arg(ws, "ws", 0, torch.uint8), ws.numel())
    return Prepared(lib().avtp_score, args, "avtp_score",
                    (dl, q_text, k, scores, img_sum, ws, row_lse, status, stream))


def prepare_budget_select_compact(dl: DeviceLayout, img_sum: torch.Tensor, scores: torch.Tensor,
                                  pairs, budget_out: torch.Tensor, keep_idx: torch.Tensor,
                                  cu_out: torch.Tensor, alpha: float = 1.0, lo_permille: int = 50,
                                  hi_permille: int = 950, floor_abs: int = 0,
                                  mode: int = BUDGET_PROPORTIONAL,
                                  status: Optional[torch.Tensor] = None, stream=None) -> Prepared:
    """avtp_budget_select_compact on fixed buffers, as a Prepared call."""
    ts = _tensor_set(pairs)
    _check_pairs(dl, ts, dl.N_out)
    args = (_stream(stream), dl.ref(), _arg(img_sum, "img_sum", dl.n_img, torch.float32), mode,
            float(alpha), lo_permille, hi_permille, floor_abs,
            _arg(scores, "scores", dl.N_tok, torch.float32),
            _arg(budget_out, "budget_out", dl.n_img, torch.int32),
            _arg(keep_idx, "keep_idx", 0, torch.int32), keep_idx.numel(),
            _arg(cu_out, "cu_out", dl.B + 1, torch.int32), _arg(status, "status", dl.B, torch.int32),
            ts.arr, ts.n)
    return Prepared(lib().avtp_budget_select_compact, args, "avtp_budget_select_compact",
                    (dl, img_sum, scores, ts, budget_out, keep_idx, cu_out, status, stream))


def score_attn(dl: DeviceLayout, q_text: torch.Tensor, k: torch.Tensor, softmax_scale: float,
               row_lse: Optional[torch.Tensor] = None, scores: Optional[torch.Tensor] = None,
               img_sum: Optional[torch.Tensor] = None, status: Optional[torch.Tensor] = None,
               ws: Optional[torch.Tensor] = None, stream=None):
    T, Hq, d = q_text.shape
    Hkv = k.shape[1]
    dt = dtype_code(q_text)
    dev = q_text.device
    if scores is None:
        scores = torch.empty(dl.N_tok, dtype=torch.float32, device=dev)
    if img_sum is None:
        img_sum = torch.empty(max(1, dl.n_img), dtype=torch.float32, device=dev)
    if ws is None:
        ws = alloc_workspace(score_workspace_bytes(dl, SCORE_ATTN, dt, Hq, Hkv, d), dev)
    _check_qk(dl, q_text, k)
    _check(lib().avtp_score(_stream(stream), dl.ref(), SCORE_ATTN, dt, _arg(q_text, "q_text"),
                            _arg(k, "k"), Hq, Hkv, d, float(softmax_scale),
                            _arg(row_lse, "row_lse", Hq * dl.T_tot, torch.float32), None, None, 0,
                            _arg(scores, "scores", dl.N_tok, torch.float32),
                            _arg(img_sum, "img_sum", dl.n_img, torch.float32),
                            _arg(status, "status", dl.B, torch.int32),
                            _arg(ws, "ws", 0, torch.uint8), ws.numel()),
           "avtp_score")
    return scores, img_sum[: dl.n_img]


def score_attn_noalloc(dl: DeviceLayout, q_text: torch.Tensor, k: torch.Tensor,
                       softmax_scale: float, scores: torch.Tensor, img_sum: torch.Tensor,
                       row_lse: Optional[torch.Tensor] = None,
                       status: Optional[torch.Tensor] = None, stream=None):
    """avtp_score_noalloc in attention mode: the caller passes the outputs; the
    library's own per-GPU scratch replaces the workspace."""
    T, Hq, d = q_text.shape
    Hkv = k.shape[1]
    _check_qk(dl, q_text, k)
    _check(lib().avtp_score_noalloc(_stream(stream), dl.ref(), SCORE_ATTN, dtype_code(q_text),
                                    _arg(q_text, "q_text"), _arg(k, "k"), Hq, Hkv, d,
                                    float(softmax_scale),
                                    _arg(row_lse, "row_lse", Hq * dl.T_tot, torch.float32), None,
                                    None, 0, _arg(scores, "scores", dl.N_tok, torch.float32),
                                    _arg(img_sum, "img_sum", dl.n_img, torch.float32),
                                    _arg(status, "status", dl.B, torch.int32)),
           "avtp_score_noalloc")
    return scores, img_sum[: dl.n_img]


def score_variation(dl: DeviceLayout, h_cur: torch.Tensor, h_prior: torch.Tensor,
                    scores: Optional[torch.Tensor] = None, img_sum: Optional[torch.Tensor] = None,
                    status: Optional[torch.Tensor] = None, stream=None):
    dev = h_cur.device
    hidden = h_cur.shape[-1]
    if scores is None:
        scores = torch.empty(dl.N_tok, dtype=torch.float32, device=dev)
    if img_sum is None:
        img_sum = torch.empty(max(1, dl.n_img), dtype=torch.float32, device=dev)
    ws = alloc_workspace(score_workspace_bytes(dl, SCORE_VARIATION), dev)
    if h_cur.shape != h_prior.shape or h_cur.dtype != h_prior.dtype or h_cur.shape[0] != dl.N_tok:
        raise ValueError("h_cur and h_prior must both be [N_tok, hidden] of one dtype")
    _check(lib().avtp_score(_stream(stream), dl.ref(), SCORE_VARIATION, dtype_code(h_cur), None,
                            None, 0, 0, 0, 1.0, None, _arg(h_cur, "h_cur"),
                            _arg(h_prior, "h_prior"), hidden,
                            _arg(scores, "scores", dl.N_tok, torch.float32),
                            _arg(img_sum, "img_sum", dl.n_img, torch.float32),
                            _arg(status, "status", dl.B, torch.int32),
                            _arg(ws, "ws", 0, torch.uint8), ws.numel()),
           "avtp_score")
    return scores, img_sum[: dl.n_img]


# --------------------------------------------------------------------------- budget
def budget(dl: DeviceLayout, img_sum: torch.Tensor, alpha: float = 1.0, lo_permille: int = 50,
           hi_permille: int = 950, floor_abs: int = 0, mode: int = BUDGET_PROPORTIONAL,
           out: Optional[torch.Tensor] = None, status: Optional[torch.Tensor] = None,
           stream=None) -> torch.Tensor:
    if out is None:
        out = torch.empty(max(1, dl.n_img), dtype=torch.int32, device=img_sum.device)
    _check(lib().avtp_budget(_stream(stream), dl.ref(),
                             _arg(img_sum, "img_sum", dl.n_img, torch.float32), mode, float(alpha),
                             lo_permille, hi_permille, floor_abs,
                             _arg(out, "out", dl.n_img, torch.int32),
                             _arg(status, "status", dl.B, torch.int32)),
           "avtp_budget")
    return out[: dl.n_img]


# --------------------------------------------------------------------------- select
def select(dl: DeviceLayout, scores: torch.Tensor, budget_: torch.Tensor,
           keep_idx: Optional[torch.Tensor] = None, cu_out: Optional[torch.Tensor] = None,
           status: Optional[torch.Tensor] = None, stream=None):
    dev = scores.device
    if keep_idx is None:
        keep_idx = torch.empty(max(1, dl.N_out), dtype=torch.int32, device=dev)
    if cu_out is None:
        cu_out = torch.empty(dl.B + 1, dtype=torch.int32, device=dev)
    _check(lib().avtp_select(_stream(stream), dl.ref(),
                             _arg(scores, "scores", dl.N_tok, torch.float32),
                             _arg(budget_, "budget", dl.n_img, torch.int32),
                             _arg(keep_idx, "keep_idx", 0, torch.int32), keep_idx.numel(),
                             _arg(cu_out, "cu_out", dl.B + 1, torch.int32),
                             _arg(status, "status", dl.B, torch.int32)),
           "avtp_select")
    return keep_idx[: dl.N_out], cu_out


# --------------------------------------------------------------------------- compact
def tensor_desc(src: torch.Tensor, dst: torch.Tensor, token_dim: int = 0) -> _Tensor:
    """Descriptor of a gather along ``token_dim`` (0: [N, ...]; 1: [P, N, ...])."""
    es = src.element_size()
    if token_dim == 0:
        row = src[0]
        if not row.is_contiguous() or not dst[0].is_contiguous():
            raise ValueError("rows must be contiguous")
        return _Tensor(src.data_ptr(), dst.data_ptr(), row.numel() * es, src.stride(0) * es,
                       dst.stride(0) * es, 1, 0, 0)
    if token_dim == 1:
        row = src[0, 0]
        if not row.is_contiguous() or not dst[0, 0].is_contiguous():
            raise ValueError("rows must be contiguous")
        return _Tensor(src.data_ptr(), dst.data_ptr(), row.numel() * es, src.stride(1) * es,
                       dst.stride(1) * es, src.shape[0], src.stride(0) * es, dst.stride(0) * es)
    raise ValueError("token_dim must be 0 or 1")


class TensorSet:
    """The descriptors of a compaction's (src, dst[, token_dim]) pairs, built
    once; pass it wherever pairs are taken to skip rebuilding them on every
    call (it keeps the tensors alive)."""

    def __init__(self, pairs: Sequence):
        self.pairs = list(pairs)
        descs = [tensor_desc(p[0], p[1], p[2] if len(p) > 2 else 0) for p in self.pairs]
        self.n = len(descs)
        self.arr = (_Tensor * max(1, self.n))(*descs)


def _tensor_set(pairs) -> TensorSet:
    return pairs if isinstance(pairs, TensorSet) else TensorSet(pairs)


def _check_pairs(dl: DeviceLayout, ts: TensorSet, n_out: int) -> None:
    """Every compaction pair on the GPU, source and destination of one dtype
    and row shape, with at least N_tok source rows and n_out destination rows
    along the token dimension (the kernels write every row below n_out)."""
    for p in ts.pairs:
        src, dst, td = p[0], p[1], (p[2] if len(p) > 2 else 0)
        if not (src.is_cuda and dst.is_cuda):
            raise ValueError("compaction tensors must be on the GPU")
        if src.dtype != dst.dtype:
            raise TypeError(f"compaction source ({src.dtype}) and destination ({dst.dtype}) differ")
        if src.shape[:td] + src.shape[td + 1:] != dst.shape[:td] + dst.shape[td + 1:]:
            raise ValueError(f"compaction rows differ: {tuple(src.shape)} -> {tuple(dst.shape)}")
        if src.shape[td] < dl.N_tok or dst.shape[td] < n_out:
            raise ValueError(f"compaction needs {dl.N_tok} source and {n_out} destination rows, "
                             f"got {src.shape[td]} and {dst.shape[td]}")


def compact(dl: DeviceLayout, keep_idx: torch.Tensor, pairs, n_out: Optional[int] = None,
            stream=None) -> None:
    """pairs: (src, dst) or (src, dst, token_dim) tuples, or a TensorSet of
    them; dst is written in place."""
    ts = _tensor_set(pairs)
    n = dl.N_out if n_out is None else int(n_out)
    _check_pairs(dl, ts, n)
    _check(lib().avtp_compact(_stream(stream), dl.ref(), _arg(keep_idx, "keep_idx", n, torch.int32),
                              n, ts.arr, ts.n),
           "avtp_compact")


def select_compact(dl: DeviceLayout, scores: torch.Tensor, budget_: torch.Tensor, pairs,
                   keep_idx: Optional[torch.Tensor] = None, cu_out: Optional[torch.Tensor] = None,
                   status: Optional[torch.Tensor] = None, stream=None):
    """avtp_select and avtp_compact in one launch; pairs as for compact."""
    dev = scores.device
    if keep_idx is None:
        keep_idx = torch.empty(max(1, dl.N_out), dtype=torch.int32, device=dev)
    if cu_out is None:
        cu_out = torch.empty(dl.B + 1, dtype=torch.int32, device=dev)
    ts = _tensor_set(pairs)
    _check_pairs(dl, ts, dl.N_out)
    _check(lib().avtp_select_compact(_stream(stream), dl.ref(),
                                     _arg(scores, "scores", dl.N_tok, torch.float32),
                                     _arg(budget_, "budget", dl.n_img, torch.int32),
                                     _arg(keep_idx, "keep_idx", 0, torch.int32), keep_idx.numel(),
                                     _arg(cu_out, "cu_out", dl.B + 1, torch.int32),
                                     _arg(status, "status", dl.B, torch.int32),
                                     ts.arr, ts.n), "avtp_select_compact")
    return keep_idx[: dl.N_out], cu_out


def budget_select_compact(dl: DeviceLayout, img_sum: torch.Tensor, scores: torch.Tensor,
                          pairs, alpha: float = 1.0, lo_permille: int = 50,
                          hi_permille: int = 950, floor_abs: int = 0,
                          mode: int = BUDGET_PROPORTIONAL, budget_out: Optional[torch.Tensor] = None,
                          keep_idx: Optional[torch.Tensor] = None,
                          cu_out: Optional[torch.Tensor] = None,
                          status: Optional[torch.Tensor] = None, stream=None):
    """avtp_budget followed by avtp_select_compact, in one call; pairs as for
    compact.  Returns (budget, keep_idx, cu_out)."""
    dev = scores.device
    if budget_out is None:
        budget_out = torch.empty(max(1, dl.n_img), dtype=torch.int32, device=dev)
    if keep_idx is None:
        keep_idx = torch.empty(max(1, dl.N_out), dtype=torch.int32, device=dev)
    if cu_out is None:
        cu_out = torch.empty(dl.B + 1, dtype=torch.int32, device=dev)
    ts = _tensor_set(pairs)
    _check_pairs(dl, ts, dl.N_out)
    _check(lib().avtp_budget_select_compact(
        _stream(stream), dl.ref(), _arg(img_sum, "img_sum", dl.n_img, torch.float32), mode,
        float(alpha), lo_permille, hi_permille, floor_abs,
        _arg(scores, "scores", dl.N_tok, torch.float32),
        _arg(budget_out, "budget_out", dl.n_img, torch.int32),
        _arg(keep_idx, "keep_idx", 0, torch.int32), keep_idx.numel(),
        _arg(cu_out, "cu_out", dl.B + 1, torch.int32), _arg(status, "status", dl.B, torch.int32),
        ts.arr, ts.n), "avtp_budget_select_compact")
    return budget_out[: dl.n_img], keep_idx[: dl.N_out], cu_out


def compact_new(dl: DeviceLayout, keep_idx: torch.Tensor, srcs: Sequence, stream=None):
    """Allocate outputs and compact (src, token_dim) pairs; returns the outputs."""
    outs, pairs = [], []
    for src, tdim in srcs:
        shape = list(src.shape)
        shape[tdim] = dl.N_out
        dst = torch.empty(shape, dtype=src.dtype, device=src.device)
        outs.append(dst)
        pairs.append((src, dst, tdim))
    compact(dl, keep_idx, pairs, stream=stream)
    return outs


# --------------------------------------------------------------------------- progressive pruning
def pruned_layout(dl: DeviceLayout, keep_idx: torch.Tensor, cu_out: torch.Tensor,
                  stream=None, out: Optional[dict] = None) -> dict:
    """Device arrays of the next pruning layer's layout (all but keep_total).
    out: the six int32 arrays to write (as returned by an earlier call on the
    same layout), else they are allocated."""
    dev = cu_out.device
    if out is None:
        out = {n: torch.empty(max(1, m), dtype=torch.int32, device=dev)
               for n, m in (("cu_seqlens", dl.B + 1), ("img_start", dl.n_img),
                            ("img_len", dl.n_img), ("cu_img", dl.B + 1), ("text_pos", dl.T_tot),
                            ("cu_text", dl.B + 1))}
    lens = {"cu_seqlens": dl.B + 1, "img_start": dl.n_img, "img_len": dl.n_img,
            "cu_img": dl.B + 1, "text_pos": dl.T_tot, "cu_text": dl.B + 1}
    _check(lib().avtp_pruned_layout(_stream(stream), dl.ref(),
                                    # (its length is cu_out[B], a device value)
                                    _arg(keep_idx, "keep_idx", 0, torch.int32),
                                    _arg(cu_out, "cu_out", dl.B + 1, torch.int32),
                                    *[_arg(out[n], n, lens[n], torch.int32)
                                      for n in ("cu_seqlens", "img_start", "img_len", "cu_img",
                                                "text_pos", "cu_text")]),
           "avtp_pruned_layout")
    return {n: t[: lens[n]] for n, t in out.items()}


# --------------------------------------------------------------------------- layer selection
def layer_attention(dl: DeviceLayout, img_sum: torch.Tensor, out: Optional[torch.Tensor] = None,
                    stream=None) -> torch.Tensor:
    """A [B] fp32: per sequence (sample), the sum of its image sums (one layer)."""
    if out is None:
        out = torch.empty(max(1, dl.B), dtype=torch.float32, device=img_sum.device)
    _check(lib().avtp_layer_attention(_stream(stream), dl.ref(),
                                      _arg(img_sum, "img_sum", dl.n_img, torch.float32),
                                      _arg(out, "out", dl.B, torch.float32)),
           "avtp_layer_attention")
    return out[: dl.B]


def layer_select(A: torch.Tensor, k: int, rank_sum: Optional[torch.Tensor] = None,
                 selected: Optional[torch.Tensor] = None, stream=None):
    """A [L, N] fp32 (layer, sample) -> (rank_sum [L] int32, selected [k] int32 ascending).
    The average rank R_l is rank_sum / N."""
    if A.dtype != torch.float32 or A.dim() != 2 or not A.is_contiguous():
        raise TypeError("A must be a contiguous [L, N] float32 tensor")
    L, N = A.shape
    if rank_sum is None:
        rank_sum = torch.empty(max(1, L), dtype=torch.int32, device=A.device)
    if selected is None:
        selected = torch.empty(max(1, k), dtype=torch.int32, device=A.device)
    _check(lib().avtp_layer_select(_stream(stream), _arg(A, "A", L * N, torch.float32), L, N,
                                   int(k), _arg(rank_sum, "rank_sum", L, torch.int32),
                                   _arg(selected, "selected", max(0, int(k)), torch.int32)),
           "avtp_layer_select")
    return rank_sum[:L], selected[:k]
