"""Progressive pruning across layers (Sec. 3.3.2: pruning at the selected
layers with a progressive schedule; Sec. 3.3.1: each pruning layer scores a
token by how far its hidden state moved since the previous pruning).

The caller runs its model and stops at each pruning layer with that layer's
hidden states; ``ProgressivePruner.step`` then prunes in VARIATION mode:

    score (1 - cos(h_cur, h_prior))  ->  budget  ->  select  ->  compact

compacting h_cur together with the caller's other per-token tensors (position
ids, the layer's K and V), and turns the kept tokens into the next layer's
layout.  The compacted h_cur is both the layer's output and the next pruning
layer's h_prior.  Every step runs in libavtp.so; this module only sequences
the calls, copies the new layout's small index arrays to the host (one
synchronisation per pruning layer, for launch sizing) and applies the
caller's keep schedule to them.
"""
from __future__ import annotations

from typing import Sequence

import numpy as np
import torch

from . import avtp as A


def keep_totals(img_len: np.ndarray, cu_img: np.ndarray, keep_pct: int) -> np.ndarray:
    """keep_total[b] = round-half-up(keep_pct % of sequence b's visual tokens)."""
    return np.array([(keep_pct * int(np.sum(img_len[cu_img[b]:cu_img[b + 1]], dtype=np.int64)) + 50)
                     // 100 for b in range(len(cu_img) - 1)], dtype=np.int32)


class ProgressivePruner:
    """State of a progressive schedule: the current layout and h_prior.

    dl: layout of the batch at the first pruning layer (its keep_total is that
    layer's keep totals); h_prior: the embeddings before any pruning
    [N_tok, hidden] (the LLM's input embeddings, Sec. 3.3.1).
    """

    def __init__(self, dl: A.DeviceLayout, h_prior: torch.Tensor, alpha: float = 1.0,
                 lo_permille: int = 50, hi_permille: int = 950, floor_abs: int = 0,
                 mode: int = A.BUDGET_PROPORTIONAL):
        self.dl = dl
        self.h_prior = h_prior
        self.alpha, self.lo, self.hi, self.floor, self.mode = alpha, lo_permille, hi_permille, \
            floor_abs, mode

    def step(self, h_cur: torch.Tensor, others: Sequence = (), keep_pct_next: int = 50,
             status: torch.Tensor = None):
        """Prune at one layer.  others: (tensor, token_dim) pairs compacted with
        h_cur.  Returns (h_out, [compacted others], keep_idx, budget, scores, img_sum);
        afterwards self.dl is the next layer's layout (keep totals from
        keep_pct_next) and self.h_prior is h_out."""
        dl = self.dl
        scores, isum = A.score_variation(dl, h_cur, self.h_prior, status=status)
        bud = A.budget(dl, isum, self.alpha, self.lo, self.hi, self.floor, mode=self.mode,
                       status=status)
        keep, cu_out = A.select(dl, scores, bud, status=status)
        outs = A.compact_new(dl, keep, [(h_cur, 0), *others])
        arrays = A.pruned_layout(dl, keep, cu_out)
        host = {n: t.cpu().numpy() for n, t in arrays.items()}     # one sync per pruning layer
        host["keep_total"] = keep_totals(host["img_len"], host["cu_img"], keep_pct_next)
        self.dl = A.DeviceLayout(host, device=h_cur.device)
        self.h_prior = outs[0]
        return outs[0], outs[1:], keep[: dl.N_out], bud, scores, isum
