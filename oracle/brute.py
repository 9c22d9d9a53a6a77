"""Brute-force (loops only) versions of the oracle -- TEST INFRASTRUCTURE ONLY.

Pure-Python restatements, written straight from the definitions, used to pin
the vectorised oracle in ``avtp_oracle`` on tiny inputs (a handful of tokens
and heads).  Nothing here is vectorised or shared with ``avtp_oracle``.
"""
from __future__ import annotations

import itertools
import math
import struct


def bf16_to_float(bits: int) -> float:
    return struct.unpack("<f", struct.pack("<I", (int(bits) & 0xFFFF) << 16))[0]


def _val(x, dtype):
    return bf16_to_float(x) if dtype == "bf16" else float(x)


def attn_scores_loops(tokens, q_rows, k_rows, Hq, Hkv, scale, dtype="fp32"):
    """One sequence.

    tokens:  list of ("text", t) or ("img", i) in position order, t = text row
             index into q_rows, i = image id.
    q_rows:  q_rows[t][h] = list of d values.
    k_rows:  k_rows[j][g] = list of d values, j = position.
    Returns (scores by position: None for text, per-image sums dict).
    For every text row t at position p and head h the attention row is the
    softmax over every position <= p; s_j averages P[h, t, j] over the heads
    and over the text rows after j.
    """
    G = Hq // Hkv
    L = len(tokens)
    text_at = {p: tok[1] for p, tok in enumerate(tokens) if tok[0] == "text"}
    acc = [0.0] * L
    for p_t, t in text_at.items():
        for h in range(Hq):
            g = h // G
            z = []
            for j in range(p_t + 1):
                dot = 0.0
                for a, b in zip(q_rows[t][h], k_rows[j][g]):
                    dot += _val(a, dtype) * _val(b, dtype)
                z.append(scale * dot)
            m = max(z)
            den = sum(math.exp(x - m) for x in z)
            for j in range(p_t + 1):
                acc[j] += math.exp(z[j] - m) / den
    scores = [None] * L
    sums = {}
    for j, tok in enumerate(tokens):
        if tok[0] != "img":
            continue
        n_after = sum(1 for p in text_at if p > j)
        s = acc[j] / (Hq * n_after) if n_after else 0.0
        scores[j] = s
        sums[tok[1]] = sums.get(tok[1], 0.0) + s
    return scores, sums


def cosine_variation_loops(a, b, dtype="fp32"):
    """1 - <a,b> / max(|a||b|, 1e-8) for two rows given as lists."""
    x = [_val(v, dtype) for v in a]
    y = [_val(v, dtype) for v in b]
    dot = sum(u * v for u, v in zip(x, y))
    nx = math.sqrt(sum(u * u for u in x))
    ny = math.sqrt(sum(v * v for v in y))
    return 1.0 - dot / max(nx * ny, 1e-8)


def topk_sorted(scores, k):
    """Indices of the k best entries by (score desc, index asc), NaN last."""
    def key(j):
        s = scores[j]
        return (1, 0.0, j) if s != s else (0, -s, j)
    return sorted(range(len(scores)), key=key)[:k]


def min_dev_integer_budget(quota, lo, hi, K):
    """Enumerate every integer vector lo <= k <= hi with sum K and return the one
    minimising sum (k_i - quota_i)^2; among equal minimisers the
    lexicographically largest (the +1 goes to the lowest index)."""
    best = None
    for ks in itertools.product(*[range(a, b + 1) for a, b in zip(lo, hi)]):
        if sum(ks) != K:
            continue
        dev = sum((k - q) ** 2 for k, q in zip(ks, quota))
        cand = (dev, tuple(-k for k in ks))
        if best is None or cand < best[0]:
            best = (cand, ks)
    return None if best is None else list(best[1])
