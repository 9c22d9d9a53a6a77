"""CPU oracle for the AVTP pruning-layer operator -- TEST INFRASTRUCTURE ONLY.

Only the tests, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this module.  It shares no code with the HIP library
or its Python binding: it reads the seeded inputs (plain numpy arrays) and
computes, slowly and in float64, what the pruning layer computes, in the
order the paper states it.

Section references are to "Multi-Image Visual Token Pruning in Large Visual
Language Models" (AVTP):
  * problem statement: select a subsequence of the visual tokens (Method,
    Preliminary, "Visual Token Pruning");
  * attention that a layer pays to visual tokens (Sec. 3.3.2, the equation
    defining A_l as a sum of Attention(l, v_j); Fig. 2 caption: measured at
    first-token generation) -- evaluated here per visual token, see attn_*;
  * hidden-state-variation importance I = 1 - Sim(h^l, h^prior)
    (Sec. 3.3.1, the importance equation);
  * per-image mean importance and adaptive keep ratio
    r_i = r_base + alpha (I_i - I_avg) (Sec. 3.3.3, the two equations);
    alpha = 1.0 (Experimental Setting); per-image clamp at 5 % / 95 %
    (Appendix, effect of alpha).

Readings where the paper is silent are listed in the repository's design
notes and restated next to the code that takes them.

Inputs in bf16 are given as uint16 bit patterns and widened exactly; all
arithmetic is float64 except where a decision must be taken in the precision
the operator defines (the budget quantisation, see ``budget``).
"""
from __future__ import annotations

import math
from fractions import Fraction

import numpy as np

LN2 = math.log(2.0)


# ---------------------------------------------------------------------------
# input helpers
# ---------------------------------------------------------------------------
def widen(x: np.ndarray, dtype: str) -> np.ndarray:
    """bf16 bit patterns (uint16) or float32 -> float64, exactly."""
    if dtype == "bf16":
        return (np.asarray(x, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return np.asarray(x, dtype=np.float32).astype(np.float64)


def text_rows_after(layout, j: int) -> int:
    """|T_j|: text tokens of j's sequence at a later position than token j."""
    b = int(np.searchsorted(layout.cu_seqlens, j, side="right") - 1)
    t0, t1 = int(layout.cu_text[b]), int(layout.cu_text[b + 1])
    return int(np.sum(layout.text_pos[t0:t1] > j))


# ---------------------------------------------------------------------------
# O1: attention-to-visual-token score (Sec. 3.3.2 quantity, per token)
# ---------------------------------------------------------------------------
def _logits(qh: np.ndarray, kg: np.ndarray, scale: float, exact_dot: bool) -> np.ndarray:
    """z[t, j] = scale * <q_t, k_j>.

    exact_dot=True sums each dot product with the same reduction for every
    (t, j), so bit-identical key rows give bit-identical logits (needed for
    exact ties).  Otherwise a BLAS product is used (large inputs).
    """
    if exact_dot:
        z = (qh[:, None, :] * kg[None, :, :]).sum(axis=-1)
    else:
        z = qh @ kg.T
    return scale * z


def attn_row_lse(layout, q_text, k, Hq: int, Hkv: int, scale: float, dtype: str,
                 exact_dot: bool = False, seqs=None) -> np.ndarray:
    """Log-sum-exp of each text row's causal attention logits.

    For text row t (position p_t) and query head h, with key group
    g = h // (Hq / Hkv) (grouped-query attention shares one key head among
    Hq/Hkv consecutive query heads):
        lse[h, t] = log sum_{j in seq, j <= p_t} exp(scale * q_{t,h} . k_{j,g})
    The normaliser is the layer's real causal attention row over every
    earlier token, visual and text.  Returns float64 [Hq, T_tot] (natural log).
    Rows of sequences not in ``seqs`` are left NaN.
    """
    G = Hq // Hkv
    lse = np.full((Hq, layout.T_tot), np.nan)
    for b in (range(layout.B) if seqs is None else seqs):
        s0, s1 = int(layout.cu_seqlens[b]), int(layout.cu_seqlens[b + 1])
        t0, t1 = int(layout.cu_text[b]), int(layout.cu_text[b + 1])
        if t1 == t0:
            continue
        pos = layout.text_pos[t0:t1].astype(np.int64)
        keys_pos = np.arange(s0, s1)
        visible = keys_pos[None, :] <= pos[:, None]                 # [T_b, L_b]
        kb = widen(k[s0:s1], dtype)                                  # [L_b, Hkv, d]
        qb = widen(q_text[t0:t1], dtype)                             # [T_b, Hq, d]
        for h in range(Hq):
            z = _logits(qb[:, h, :], kb[:, h // G, :], scale, exact_dot)
            z = np.where(visible, z, -np.inf)
            m = z.max(axis=1, keepdims=True)
            lse[h, t0:t1] = (m + np.log(np.exp(z - m).sum(axis=1, keepdims=True)))[:, 0]
    return lse


def attn_scores(layout, q_text, k, Hq: int, Hkv: int, scale: float, dtype: str,
                exact_dot: bool = False, lse=None, seqs=None):
    """Per-visual-token attention score and per-image sums.

    For visual token j of image V_i, with T_j the text rows after j:
        P[h, t, j] = exp(scale * q_{t,h} . k_{j,g(h)} - lse[h, t])
        s_j = (1 / Hq) sum_h (1 / |T_j|) sum_{t in T_j} P[h, t, j]
        S_i = sum_{j in V_i} s_j
    i.e. the attention mass a text row pays to j, averaged over the rows that
    can see j and over all query heads.  Summing s_j over all visual tokens
    gives the layer's attention to visual tokens (Sec. 3.3.2).
    Text positions get +inf (they are never pruned).  If |T_j| = 0 the score
    is 0 and the image is reported in ``empty``.
    Returns (scores[N_tok] f64, img_sum[n_img] f64, lse[Hq, T_tot], empty set).
    """
    if lse is None:
        lse = attn_row_lse(layout, q_text, k, Hq, Hkv, scale, dtype, exact_dot, seqs)
    G = Hq // Hkv
    N = layout.N_tok
    colsum = np.zeros(N)
    scores = np.full(N, np.inf)
    for b in (range(layout.B) if seqs is None else seqs):
        s0, s1 = int(layout.cu_seqlens[b]), int(layout.cu_seqlens[b + 1])
        t0, t1 = int(layout.cu_text[b]), int(layout.cu_text[b + 1])
        if t1 == t0:
            continue
        pos = layout.text_pos[t0:t1].astype(np.int64)
        keys_pos = np.arange(s0, s1)
        visible = keys_pos[None, :] <= pos[:, None]
        kb = widen(k[s0:s1], dtype)
        qb = widen(q_text[t0:t1], dtype)
        acc = np.zeros(s1 - s0)
        for h in range(Hq):
            z = _logits(qb[:, h, :], kb[:, h // G, :], scale, exact_dot)
            p = np.where(visible, np.exp(z - lse[h, t0:t1][:, None]), 0.0)
            acc += p.sum(axis=0)
        colsum[s0:s1] = acc
    img_sum = np.zeros(layout.n_img)
    empty = set()
    bs = set(range(layout.B) if seqs is None else seqs)
    for b in bs:
        for i in range(int(layout.cu_img[b]), int(layout.cu_img[b + 1])):
            s0, n = int(layout.img_start[i]), int(layout.img_len[i])
            if n == 0:
                continue
            nt = text_rows_after(layout, s0)     # constant over an image: no text inside it
            if nt == 0:
                scores[s0:s0 + n] = 0.0
                empty.add(i)
            else:
                scores[s0:s0 + n] = colsum[s0:s0 + n] / (Hq * nt)
            img_sum[i] = scores[s0:s0 + n].sum()
    return scores, img_sum, lse, empty


def attn_score_one(layout, q_text, k, Hq: int, Hkv: int, scale: float, dtype: str,
                   lse: np.ndarray, j: int) -> float:
    """s_j for a single visual token, given the row LSE (sampled checks at full size)."""
    G = Hq // Hkv
    b = int(np.searchsorted(layout.cu_seqlens, j, side="right") - 1)
    t0, t1 = int(layout.cu_text[b]), int(layout.cu_text[b + 1])
    rows = [t for t in range(t0, t1) if int(layout.text_pos[t]) > j]
    if not rows:
        return 0.0
    kj = widen(k[j], dtype)                      # [Hkv, d]
    tot = 0.0
    for h in range(Hq):
        q = widen(q_text[rows, h, :], dtype)     # [R, d]
        z = scale * (q @ kj[h // G])
        tot += float(np.exp(z - lse[h, rows]).sum())
    return tot / (Hq * len(rows))


# ---------------------------------------------------------------------------
# O1': hidden-state-variation score (Sec. 3.3.1)
# ---------------------------------------------------------------------------
COS_EPS = 1e-8


def variation_scores(layout, h_cur, h_prior, dtype: str):
    """I_j = 1 - cos(h^l_j, h^prior_j) for visual tokens (Sec. 3.3.1).

    "Sim" is read as cosine similarity, with the usual guard
    cos = <a, b> / max(|a| |b|, 1e-8).  Text positions get +inf.
    Returns (scores[N_tok] f64, img_sum[n_img] f64).
    """
    N = layout.N_tok
    scores = np.full(N, np.inf)
    img_sum = np.zeros(layout.n_img)
    for i in range(layout.n_img):
        s0, n = int(layout.img_start[i]), int(layout.img_len[i])
        if n == 0:
            continue
        a = widen(h_cur[s0:s0 + n], dtype)
        p = widen(h_prior[s0:s0 + n], dtype)
        dot = (a * p).sum(axis=1)
        na = np.sqrt((a * a).sum(axis=1))
        npr = np.sqrt((p * p).sum(axis=1))
        scores[s0:s0 + n] = 1.0 - dot / np.maximum(na * npr, COS_EPS)
        img_sum[i] = scores[s0:s0 + n].sum()
    return scores, img_sum


# ---------------------------------------------------------------------------
# O2: per-image budgets (Sec. 3.3.3 + Appendix clamp)
# ---------------------------------------------------------------------------
WEIGHT_BITS = 28          # the largest weight becomes 2^28; the others keep their ratio to it
BUDGET_PROPORTIONAL = 0   # r_i in units where the mean importance equals r_base
BUDGET_RAW = 1            # r_i = r_base + alpha (I_i - I_avg) in raw score units


def budget_bounds(n: int, lo_permille: int, hi_permille: int, floor_abs: int):
    """Per-image keep bounds: ceil(lo n), floor(hi n), the absolute floor, and n."""
    lo = min(n, max((lo_permille * n + 999) // 1000, floor_abs))
    hi = max(lo, (hi_permille * n) // 1000)
    return lo, hi


def budget_weights(n_list, S_list, K: int, alpha: float, mode: int = BUDGET_PROPORTIONAL):
    """Integer weights W_i of one sequence (the only floating-point step).

    mean importance (Sec. 3.3.3): Ibar_i = S_i / n_i, Ibar_avg = S / M
    (token-weighted, so the ratios conserve the keep total before clamping).
    Quota q_i = r_i n_i = K w_i with
        proportional: r_i = r_base (1 + alpha (Ibar_i / Ibar_avg - 1))
                      -> w_i = (1 - alpha) n_i / M + alpha S_i / S
        raw:          r_i = r_base + alpha (Ibar_i - Ibar_avg)
                      -> w_i = n_i / M + alpha (S_i - n_i S / M) / K
    Negative w are clamped to 0.  Only the ratios of the weights matter to the
    water-filling (q_i = clamp(lam W_i, ...)), so they are measured against the
    largest one, w_max: W_i = max(1, rint((w_i / w_max) 2^28)).  This keeps
    every ratio of the rule (to 2^-28 of the largest weight) for weights of any
    size and bounds the integer stage's products; W_i >= 1 keeps every image in
    the water-filling.  If S is not positive and finite, every image gets its
    token share n_i / M.  Each operation is one IEEE float64 operation,
    evaluated left to right, no fused multiply-add.
    """
    alpha = float(np.float32(alpha))
    M = 0
    for n in n_list:
        M += int(n)
    S = 0.0
    for s in S_list:
        S = S + float(np.float32(s))
    good = math.isfinite(S) and S > 0.0
    ws = []
    for n, s in zip(n_list, S_list):
        s = float(np.float32(s))
        if int(n) == 0:
            ws.append(None)
            continue
        u = float(n) / float(M)
        if not good or not math.isfinite(s):
            w = u
        elif mode == BUDGET_PROPORTIONAL:
            w = (1.0 - alpha) * u + alpha * (s / S)
        else:
            w = u + alpha * ((s - u * S) / float(K)) if K > 0 else u
        if not (w > 0.0):
            w = 0.0
        ws.append(w)
    w_max = max([w for w in ws if w is not None], default=0.0)
    W = []
    for w in ws:
        if w is None:
            W.append(0)
        elif w_max > 0.0:
            W.append(max(1, int(round((w / w_max) * float(1 << WEIGHT_BITS)))))
        else:
            W.append(1)
    return W


def water_level(W, lo, hi, K: int):
    """Exact real quotas q*_i = clamp(lam W_i, lo_i, hi_i) with sum q* = K.

    f(lam) = sum_i clamp(lam W_i, lo_i, hi_i) is continuous and
    non-decreasing, linear between the breakpoints lo_i / W_i and hi_i / W_i;
    the segment that contains K is found by evaluating f at every breakpoint
    (exact rationals), then lam is solved on it.  Returns a list of Fractions.
    """
    idx = [i for i in range(len(W)) if W[i] > 0]
    if not idx:
        return [Fraction(0)] * len(W)

    def f(lam):
        return sum(min(max(lam * W[i], Fraction(lo[i])), Fraction(hi[i])) for i in idx)

    bps = sorted(set([Fraction(lo[i], W[i]) for i in idx] + [Fraction(hi[i], W[i]) for i in idx]))
    prev = None
    for bp in bps:
        if f(bp) >= K:
            break
        prev = bp
    else:
        raise ValueError("infeasible budget")
    hi_bp = bp
    lo_bp = prev if prev is not None else Fraction(0)
    # on [lo_bp, hi_bp] f is linear: f(lam) = f(lo_bp) + (lam - lo_bp) * slope
    flo, fhi = f(lo_bp), f(hi_bp)
    lam = hi_bp if fhi == flo else lo_bp + (K - flo) * (hi_bp - lo_bp) / (fhi - flo)
    q = [Fraction(0)] * len(W)
    for i in idx:
        q[i] = min(max(lam * W[i], Fraction(lo[i])), Fraction(hi[i]))
    return q


def largest_remainder(q, K: int):
    """Hamilton rounding: floor every quota, then +1 to the K - sum(floor)
    quotas with the largest fractional parts; equal parts go to the lowest
    image index."""
    k = [int(math.floor(x)) for x in q]
    rem = [x - ki for x, ki in zip(q, k)]
    extra = K - sum(k)
    order = sorted(range(len(q)), key=lambda i: (-rem[i], i))
    for i in order[:extra]:
        k[i] += 1
    return k


def budget(layout, img_sum, alpha: float, lo_permille: int = 50, hi_permille: int = 950,
           floor_abs: int = 0, mode: int = BUDGET_PROPORTIONAL, return_quota: bool = False):
    """Per-image keep counts k_i for every sequence; sum_i k_i = keep_total[b].

    img_sum is taken as float32 (the operator's score precision).  Raises
    ValueError when the bounds make keep_total unreachable.
    """
    out = np.zeros(layout.n_img, dtype=np.int32)
    quotas = [None] * layout.n_img
    for b in range(layout.B):
        i0, i1 = int(layout.cu_img[b]), int(layout.cu_img[b + 1])
        K = int(layout.keep_total[b])
        ns = [int(x) for x in layout.img_len[i0:i1]]
        if i1 == i0:
            if K != 0:
                raise ValueError("infeasible budget")
            continue
        bounds = [budget_bounds(n, lo_permille, hi_permille, floor_abs) for n in ns]
        lo = [x[0] for x in bounds]
        hi = [x[1] for x in bounds]
        if sum(lo) > K or K > sum(hi):
            raise ValueError("infeasible budget")
        W = budget_weights(ns, [img_sum[i] for i in range(i0, i1)], K, alpha, mode)
        q = water_level(W, lo, hi, K)
        ks = largest_remainder(q, K)
        out[i0:i1] = ks
        quotas[i0:i1] = q
    return (out, quotas) if return_quota else out


# ---------------------------------------------------------------------------
# O3: segmented top-k selection and the kept-index list
# ---------------------------------------------------------------------------
def select(layout, scores, budget_arr):
    """Keep, in every image, the budget_i highest-scoring tokens.

    Order inside an image: score descending, then token index ascending (the
    lowest index wins an exact tie; -0.0 equals +0.0; NaN ranks below every
    other value).  Text tokens are always kept.  Returns the kept global token
    indices of every sequence in ascending order, concatenated, and cu_out.
    """
    s = np.asarray(scores, dtype=np.float32)
    keep = []
    cu_out = [0]
    for b in range(layout.B):
        kept_b = [int(t) for t in layout.text_pos[int(layout.cu_text[b]):int(layout.cu_text[b + 1])]]
        for i in range(int(layout.cu_img[b]), int(layout.cu_img[b + 1])):
            s0, n = int(layout.img_start[i]), int(layout.img_len[i])
            key = lambda j: (0 if not math.isnan(float(s[j])) else 1,
                             -float(s[j]) if not math.isnan(float(s[j])) else 0.0, j)
            order = sorted(range(s0, s0 + n), key=key)
            kept_b.extend(order[:int(budget_arr[i])])
        kept_b.sort()
        keep.extend(kept_b)
        cu_out.append(len(keep))
    return np.asarray(keep, dtype=np.int32), np.asarray(cu_out, dtype=np.int32)


# ---------------------------------------------------------------------------
# O4: stable compaction
# ---------------------------------------------------------------------------
def compact(keep_idx, x: np.ndarray, axis: int = 0) -> np.ndarray:
    """out[r] = x[keep_idx[r]] along the token axis; values are copied unchanged
    (position ids keep their original values)."""
    return np.take(x, np.asarray(keep_idx, dtype=np.int64), axis=axis)


# ---------------------------------------------------------------------------
# O5: architecture-aware pruning-layer selection (Sec. 3.3.2)
# ---------------------------------------------------------------------------
def layer_attention(layout, img_sum) -> np.ndarray:
    """A^(b) of one layer for every sequence (sample) b: the attention the layer
    pays to all visual tokens of the sample (Sec. 3.3.2, the A_l equation).

    With the per-token attention score s_j of ``attn_scores`` standing for
    Attention(l, v_j), the sum over the sample's visual tokens equals the sum of
    its per-image sums S_i.  Summed exactly (math.fsum) from the float32 S_i."""
    cu = np.asarray(layout.cu_img, dtype=np.int64)
    s = np.asarray(img_sum, dtype=np.float64)
    return np.array([math.fsum(s[cu[b]:cu[b + 1]].tolist()) for b in range(len(cu) - 1)],
                    dtype=np.float64)


def layer_ranks(A) -> np.ndarray:
    """Rank(A_l^(i)) of Sec. 3.3.2 for A [L, N] (layer l, sample i): within each
    sample the layers are ranked by attention, rank 1 = the largest.

    Readings: equal values rank the lower layer index first, so every sample's
    ranks are a permutation of 1..L; NaN counts as the smallest value; -0.0
    equals +0.0."""
    A = np.asarray(A, dtype=np.float64)
    L, N = A.shape
    ranks = np.zeros((L, N), dtype=np.int64)
    for i in range(N):
        v = [-math.inf if math.isnan(x) else float(x) for x in A[:, i]]
        order = sorted(range(L), key=lambda l: (-v[l], l))
        for r, l in enumerate(order):
            ranks[l, i] = r + 1
    return ranks


def layer_select(A, k: int):
    """R_l = (1/N) sum_i Rank(A_l^(i)) and the k pruning layers with the highest
    average attention, i.e. the smallest average rank (Sec. 3.3.2, the R_l
    equation and the top-k rule).

    Returns (rank_sum [L] int64 = N R_l exactly, R [L] float64, selected: the k
    chosen layer indices in ascending order).  Equal rank sums choose the lower
    layer index."""
    ranks = layer_ranks(A)
    L, N = ranks.shape
    rank_sum = ranks.sum(axis=1)
    order = sorted(range(L), key=lambda l: (int(rank_sum[l]), l))
    return rank_sum, rank_sum / float(N), sorted(order[:k])


# ---------------------------------------------------------------------------
# O6: progressive pruning across layers (Sec. 3.3.1, Sec. 3.3.2)
# ---------------------------------------------------------------------------
def pruned_layout(layout, keep_idx, cu_out, keep_total_next):
    """The packed layout of the kept tokens, for the next pruning layer.

    Pruning keeps a subsequence of every sequence (Method, "Visual Token
    Pruning"), so the kept tokens of sequence b, in their original order,
    become sequence b of the next layer: kept token r of the batch gets index
    r.  An image keeps its kept tokens (its start is the new index of its
    first kept token, or where it would be if it kept none); every text token
    is kept.  keep_total_next is the next layer's keep totals (the schedule is
    the caller's).  Returns an object with the layout's array attributes."""
    from types import SimpleNamespace
    keep_idx = np.asarray(keep_idx, dtype=np.int64)
    cu_out = np.asarray(cu_out, dtype=np.int64)
    cu_img = np.asarray(layout.cu_img, dtype=np.int64)
    cu_text = np.asarray(layout.cu_text, dtype=np.int64)
    img_start, img_len, text_pos = [], [], []
    for b in range(len(cu_out) - 1):
        kept = keep_idx[cu_out[b]:cu_out[b + 1]].tolist()
        new_index = {j: int(cu_out[b]) + r for r, j in enumerate(kept)}
        for i in range(cu_img[b], cu_img[b + 1]):
            s0, n = int(layout.img_start[i]), int(layout.img_len[i])
            img_start.append(int(cu_out[b]) + sum(1 for j in kept if j < s0))
            img_len.append(sum(1 for j in kept if s0 <= j < s0 + n))
        for t in range(cu_text[b], cu_text[b + 1]):
            text_pos.append(new_index[int(layout.text_pos[t])])
    a = lambda v: np.asarray(v, dtype=np.int32)
    return SimpleNamespace(cu_seqlens=a(cu_out), img_start=a(img_start), img_len=a(img_len),
                           cu_img=a(cu_img), text_pos=a(text_pos), cu_text=a(cu_text),
                           keep_total=a(keep_total_next), B=len(cu_out) - 1,
                           n_img=len(img_len), N_tok=int(cu_out[-1]), T_tot=len(text_pos))


def keep_totals(layout, keep_pct: int):
    """keep_total[b] = round-half-up(keep_pct % of sequence b's visual tokens)."""
    cu = np.asarray(layout.cu_img, dtype=np.int64)
    n = np.asarray(layout.img_len, dtype=np.int64)
    return np.array([(keep_pct * int(n[cu[b]:cu[b + 1]].sum()) + 50) // 100
                     for b in range(len(cu) - 1)], dtype=np.int32)


def progressive_step(layout, h_cur, h_prior, dtype: str, keep_pct_next: int, alpha: float = 1.0,
                     lo_permille: int = 50, hi_permille: int = 950, floor_abs: int = 0):
    """One pruning layer of the progressive schedule in VARIATION mode: the
    importance of each visual token against its embedding after the previous
    pruning (h_prior, Sec. 3.3.1), per-image budgets, per-image top-k, and the
    kept tokens' hidden states, which are both this layer's output and the
    next pruning layer's h_prior.  Returns (next layout, kept h_cur, keep_idx,
    budgets, scores)."""
    s, isum = variation_scores(layout, h_cur, h_prior, dtype)
    bud = budget(layout, np.asarray(isum, dtype=np.float32), alpha, lo_permille, hi_permille,
                 floor_abs)
    keep, cu_out = select(layout, np.asarray(s, dtype=np.float32), bud)
    h_next = compact(keep, h_cur)
    nxt = pruned_layout(layout, keep, cu_out, np.zeros(len(cu_out) - 1, dtype=np.int32))
    nxt.keep_total = keep_totals(nxt, keep_pct_next)
    return nxt, h_next, keep, bud, s
