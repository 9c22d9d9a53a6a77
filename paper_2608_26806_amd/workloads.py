"""Seeded synthetic inputs for the AVTP pruning-layer operator.

This module only *draws* inputs: packed multi-image layouts, text queries,
keys, values, hidden states, position ids and keep totals.  It contains none
of the method's arithmetic (no scores, budgets, selection or compaction), so
both the CPU oracle and the HIP path can consume the very same tensors.

The shapes follow the three LVLMs the paper evaluates (LLaVA-OV-7B,
InternVL3.5-8B, Qwen3VL-8B; Experimental Setting) and the multi-image
benchmark regime it targets (many images, >8k visual tokens; Observations,
Table 1).  The benchmarks themselves are not available; these generators
stand in for them.

Packed ("THD") layout of one batch, all indices global token indices:
  * sequence b owns tokens [cu_seqlens[b], cu_seqlens[b+1]);
  * inside a sequence, each image is preceded by ``pre`` text tokens, and the
    remaining ``tail`` text tokens follow the last image;
  * image i covers [img_start[i], img_start[i] + img_len[i]), images of
    sequence b are cu_img[b] .. cu_img[b+1]-1 in ascending position order;
  * text token t (t in [cu_text[b], cu_text[b+1])) sits at text_pos[t].

Every tensor is drawn in float32 from ``numpy.random.default_rng`` (PCG64)
streams keyed by (1000 + config id, stream id), so optional tensors never
shift the others; bf16 tensors are then rounded to nearest-even bf16 and kept
as their uint16 bit patterns.
"""
from __future__ import annotations

import dataclasses
from typing import Optional

import numpy as np

# RNG stream ids: one independent stream per drawn quantity.
_S_LAYOUT, _S_SCALE, _S_SALIENT, _S_Q, _S_K, _S_V, _S_HID, _S_PRIOR, _S_NOISE = range(9)


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bfloat16 (nearest, ties to even); return uint16 bits."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32)
    out = np.empty(u.shape, dtype=np.uint16)
    flat_u = u.reshape(-1)
    flat_o = out.reshape(-1)
    step = 1 << 24
    for s in range(0, flat_u.size, step):
        c = flat_u[s:s + step]
        r = ((c >> 16) & 1) + np.uint32(0x7FFF)
        flat_o[s:s + step] = ((c + r) >> 16).astype(np.uint16)
    return out


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Exact widening of bfloat16 bit patterns to float32."""
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


@dataclasses.dataclass
class Layout:
    """Host description of one packed batch (all arrays int32)."""
    cu_seqlens: np.ndarray   # [B+1]
    img_start: np.ndarray    # [n_img] global token index of the image's first token
    img_len: np.ndarray      # [n_img]
    cu_img: np.ndarray       # [B+1]
    text_pos: np.ndarray     # [T_tot] global token index of each text token
    cu_text: np.ndarray      # [B+1]
    keep_total: np.ndarray   # [B] visual tokens kept per sequence

    @property
    def B(self) -> int:
        return len(self.cu_seqlens) - 1

    @property
    def n_img(self) -> int:
        return len(self.img_len)

    @property
    def N_tok(self) -> int:
        return int(self.cu_seqlens[-1])

    @property
    def T_tot(self) -> int:
        return len(self.text_pos)

    @property
    def N_out(self) -> int:
        """Rows after pruning: every text token plus each sequence's keep total."""
        return int(self.T_tot + int(np.sum(self.keep_total, dtype=np.int64)))

    def visual_mask(self) -> np.ndarray:
        m = np.zeros(self.N_tok, dtype=bool)
        for s, n in zip(self.img_start, self.img_len):
            m[s:s + n] = True
        return m


def build_layout(images_per_seq, pre: int, tail: int, keep_pct: int) -> Layout:
    """Pack sequences; ``images_per_seq[b]`` lists the token counts of b's images.

    keep_total[b] = round-half-up(keep_pct % of the sequence's visual tokens).
    """
    cu_seqlens, img_start, img_len, cu_img, text_pos, cu_text, keep = [0], [], [], [0], [], [0], []
    pos = 0
    for imgs in images_per_seq:
        for n in imgs:
            text_pos.extend(range(pos, pos + pre))
            pos += pre
            img_start.append(pos)
            img_len.append(int(n))
            pos += int(n)
        text_pos.extend(range(pos, pos + tail))
        pos += tail
        cu_seqlens.append(pos)
        cu_img.append(len(img_len))
        cu_text.append(len(text_pos))
        m = int(sum(int(n) for n in imgs))
        keep.append((keep_pct * m + 50) // 100)
    a = lambda v: np.asarray(v, dtype=np.int32)
    return Layout(a(cu_seqlens), a(img_start), a(img_len), a(cu_img), a(text_pos), a(cu_text), a(keep))


@dataclasses.dataclass
class Workload:
    name: str
    cfg: int
    dtype: str                 # "bf16" or "fp32": storage type of q/k/v/hidden
    layout: Layout
    Hq: int
    Hkv: int
    d: int
    hidden: int
    pos_planes: int
    softmax_scale: float
    alpha: float
    lo_permille: int
    hi_permille: int
    floor_abs: int
    salient: np.ndarray        # [N_tok] bool, tokens given extra text alignment
    q_text: np.ndarray         # [T_tot, Hq, d]   uint16 (bf16 bits) or float32
    k: np.ndarray              # [N_tok, Hkv, d]
    v: Optional[np.ndarray] = None        # [N_tok, Hkv, d]
    hidden_states: Optional[np.ndarray] = None  # [N_tok, hidden]
    pos: Optional[np.ndarray] = None      # [pos_planes, N_tok] int64
    h_prior: Optional[np.ndarray] = None  # [N_tok, hidden] (variation-mode inputs)
    h_cur: Optional[np.ndarray] = None    # [N_tok, hidden]

    def as_f32(self, name: str) -> np.ndarray:
        x = getattr(self, name)
        return bf16_bits_to_f32(x) if self.dtype == "bf16" else np.asarray(x, dtype=np.float32)


# ---------------------------------------------------------------------------
# configuration table (five workloads, smallest first)
# ---------------------------------------------------------------------------
CONFIGS = {
    1: dict(name="tiny-fp32 2x64 img + 16 text, 4/2 heads, d64", B=1, dtype="fp32", Hq=4, Hkv=2, d=64,
            hidden=256, pre=0, tail=16, keep=50, sigma=0.0, floor_abs=0, pos_planes=1),
    2: dict(name="llava-ov-7b 4x729 img, 64 text, 28/4 heads, d128", B=1, dtype="bf16", Hq=28, Hkv=4,
            d=128, hidden=3584, pre=4, tail=48, keep=25, sigma=0.5, floor_abs=0, pos_planes=1),
    3: dict(name="internvl3.5-8b 8x(256..1536) img, 96 text, 32/8 heads, d128, batch 2", B=2,
            dtype="bf16", Hq=32, Hkv=8, d=128, hidden=4096, pre=4, tail=64, keep=33, sigma=0.0,
            floor_abs=0, pos_planes=1),
    4: dict(name="qwen3vl-8b 16x(256..1280) img, 128 text, 32/8 heads, d128, batch 8", B=8,
            dtype="bf16", Hq=32, Hkv=8, d=128, hidden=4096, pre=4, tail=64, keep=33, sigma=0.75,
            floor_abs=0, pos_planes=3),
    5: dict(name="long multi-image 32x1024 img, 512 text, 32/8 heads, d128, batch 4", B=4,
            dtype="bf16", Hq=32, Hkv=8, d=128, hidden=4096, pre=4, tail=384, keep=10, sigma=0.0,
            floor_abs=16, pos_planes=1),
}


def _rng(cfg: int, stream: int, seed_offset: int = 0) -> np.random.Generator:
    return np.random.default_rng([1000 + cfg + seed_offset, stream])


def _image_sizes(cfg: int, B: int, rng: np.random.Generator):
    if cfg == 1:
        return [[64, 64] for _ in range(B)]
    if cfg == 2:
        return [[729] * 4 for _ in range(B)]
    if cfg == 3:
        return [[256 * int(u) for u in rng.integers(1, 7, size=8)] for _ in range(B)]
    if cfg == 4:
        return [[4 * int(u) for u in rng.integers(64, 321, size=16)] for _ in range(B)]
    if cfg == 5:
        return [[1024] * 32 for _ in range(B)]
    raise ValueError(cfg)


def _split_largest_remainder(total: int, weights) -> list:
    """Split an integer total in proportion to weights (input construction only)."""
    w = np.asarray(weights, dtype=np.float64)
    q = total * w / w.sum()
    base = np.floor(q).astype(np.int64)
    rem = q - base
    order = sorted(range(len(w)), key=lambda i: (-rem[i], i))
    for i in order[: total - int(base.sum())]:
        base[i] += 1
    return [int(x) for x in base]


def _salient_counts(cfg: int, imgs, rng: np.random.Generator):
    """Number of text-aligned tokens in each image of one sequence."""
    n = len(imgs)
    if cfg == 1:
        return [8, 0]
    if cfg in (2, 4):
        return [int(round(0.05 * m)) for m in imgs]
    if cfg == 3:
        frac = rng.uniform(0.01, 0.2, size=n)
        return [int(round(f * m)) for f, m in zip(frac, imgs)]
    if cfg == 5:
        total = int(round(0.05 * sum(imgs)))
        heavy = rng.choice(n, size=4, replace=False)
        heavy_share = _split_largest_remainder(int(round(0.7 * total)), [1.0] * 4)
        light = [i for i in range(n) if i not in set(heavy.tolist())]
        light_share = _split_largest_remainder(total - sum(heavy_share), [1.0] * len(light))
        counts = [0] * n
        for i, c in zip(heavy.tolist(), heavy_share):
            counts[i] = c
        for i, c in zip(light, light_share):
            counts[i] = c
        return [min(c, m) for c, m in zip(counts, imgs)]
    raise ValueError(cfg)


def _normal_f32(rng: np.random.Generator, shape) -> np.ndarray:
    return rng.standard_normal(size=shape, dtype=np.float32)


def _store(x: np.ndarray, dtype: str) -> np.ndarray:
    return f32_to_bf16_bits(x) if dtype == "bf16" else np.ascontiguousarray(x, dtype=np.float32)


def make_workload(cfg: int, *, payload: bool = True, variation: bool = False,
                  seed_offset: int = 0, batch: Optional[int] = None) -> Workload:
    """Draw configuration ``cfg`` (1..5).

    payload:   also draw V, hidden states and position ids (compaction inputs).
    variation: also draw h_prior and h_cur for the hidden-state-variation score.
    batch:     override the number of sequences (bounded samples of a workload).
    """
    c = dict(CONFIGS[cfg])
    B = c["B"] if batch is None else int(batch)
    Hq, Hkv, d, dtype = c["Hq"], c["Hkv"], c["d"], c["dtype"]
    G = Hq // Hkv
    imgs = _image_sizes(cfg, B, _rng(cfg, _S_LAYOUT, seed_offset))
    lay = build_layout(imgs, c["pre"], c["tail"], c["keep"])
    N, T = lay.N_tok, lay.T_tot

    # per-image log-normal key scale s_i = exp(sigma * xi_i)
    xi = _rng(cfg, _S_SCALE, seed_offset).standard_normal(lay.n_img)
    scale = np.exp(c["sigma"] * xi).astype(np.float32)

    # salient (text-aligned) tokens, chosen uniformly without replacement per image
    rs = _rng(cfg, _S_SALIENT, seed_offset)
    salient = np.zeros(N, dtype=bool)
    for b in range(B):
        i0, i1 = int(lay.cu_img[b]), int(lay.cu_img[b + 1])
        counts = _salient_counts(cfg, [int(x) for x in lay.img_len[i0:i1]], rs)
        for i, cnt in zip(range(i0, i1), counts):
            if cnt:
                sel = rs.choice(int(lay.img_len[i]), size=cnt, replace=False)
                salient[int(lay.img_start[i]) + sel] = True

    q32 = _normal_f32(_rng(cfg, _S_Q, seed_offset), (T, Hq, d))
    q_store = _store(q32, dtype)
    q_used = bf16_bits_to_f32(q_store) if dtype == "bf16" else q_store

    k32 = _normal_f32(_rng(cfg, _S_K, seed_offset), (N, Hkv, d))
    for i in range(lay.n_img):
        s0, n = int(lay.img_start[i]), int(lay.img_len[i])
        if scale[i] != 1.0:
            k32[s0:s0 + n] *= scale[i]
    # alignment: k_{j,g} += 2 sqrt(d) * normalised mean text query of group g (per sequence)
    for b in range(B):
        t0, t1 = int(lay.cu_text[b]), int(lay.cu_text[b + 1])
        s0, s1 = int(lay.cu_seqlens[b]), int(lay.cu_seqlens[b + 1])
        idx = np.nonzero(salient[s0:s1])[0] + s0
        if len(idx) == 0 or t1 == t0:
            continue
        qm = q_used[t0:t1].reshape(t1 - t0, Hkv, G, d).mean(axis=(0, 2))   # [Hkv, d]
        qm = qm / np.linalg.norm(qm, axis=-1, keepdims=True)
        k32[idx] += (2.0 * np.sqrt(d) * qm)[None].astype(np.float32)
    k_store = _store(k32, dtype)
    del k32

    wl = Workload(name=c["name"], cfg=cfg, dtype=dtype, layout=lay, Hq=Hq, Hkv=Hkv, d=d,
                  hidden=c["hidden"], pos_planes=c["pos_planes"], softmax_scale=1.0 / np.sqrt(d),
                  alpha=1.0, lo_permille=50, hi_permille=950, floor_abs=c["floor_abs"],
                  salient=salient, q_text=q_store, k=k_store)
    if payload:
        wl.v = _store(_normal_f32(_rng(cfg, _S_V, seed_offset), (N, Hkv, d)), dtype)
        wl.hidden_states = _draw_rows(_rng(cfg, _S_HID, seed_offset), N, c["hidden"], dtype)
        pos = np.empty((c["pos_planes"], N), dtype=np.int64)
        for b in range(B):
            s0, s1 = int(lay.cu_seqlens[b]), int(lay.cu_seqlens[b + 1])
            for r in range(c["pos_planes"]):
                pos[r, s0:s1] = np.arange(s1 - s0) + r * (s1 - s0)
        wl.pos = pos
    if variation:
        prior = _draw_rows(_rng(cfg, _S_PRIOR, seed_offset), N, c["hidden"], "fp32")
        gamma = np.where(salient, 0.5, 0.1).astype(np.float32)
        tok_scale = np.ones(N, dtype=np.float32)
        for i in range(lay.n_img):
            s0, n = int(lay.img_start[i]), int(lay.img_len[i])
            tok_scale[s0:s0 + n] = scale[i]
        rn = _rng(cfg, _S_NOISE, seed_offset)
        cur = np.empty_like(prior)
        step = max(1, (1 << 22) // c["hidden"])
        for s in range(0, N, step):
            e = min(N, s + step)
            noise = rn.standard_normal(size=(e - s, c["hidden"]), dtype=np.float32)
            cur[s:e] = prior[s:e] + (gamma[s:e] * tok_scale[s:e])[:, None] * noise
        wl.h_prior = _store(prior, dtype)
        wl.h_cur = _store(cur, dtype)
    return wl


def _draw_rows(rng: np.random.Generator, n: int, width: int, dtype: str) -> np.ndarray:
    out = np.empty((n, width), dtype=np.uint16 if dtype == "bf16" else np.float32)
    step = max(1, (1 << 22) // width)
    for s in range(0, n, step):
        e = min(n, s + step)
        out[s:e] = _store(rng.standard_normal(size=(e - s, width), dtype=np.float32), dtype)
    return out


def duplicate_key_rows(wl: Workload, src: int, dst) -> None:
    """Make the K rows of tokens ``dst`` bit-identical copies of token ``src``.

    Used to build exact score ties (the tokens then see identical logits).
    """
    for j in dst:
        wl.k[int(j)] = wl.k[int(src)]
