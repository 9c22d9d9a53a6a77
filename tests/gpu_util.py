"""Helpers shared by the GPU tests (no test functions here)."""
from __future__ import annotations

import sys

import numpy as np
import pytest
import torch

from paper_2608_26806_amd import avtp as A

TOL = {"bf16": 2e-3, "fp32": 1e-5}        # relative tolerance on scores / image sums


def need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")


def say(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


def to_dev(x: np.ndarray, dtype: str) -> torch.Tensor:
    """Seeded host tensor -> device tensor of the workload's storage type."""
    if dtype == "bf16":
        return torch.from_numpy(np.ascontiguousarray(x).view(np.int16)).view(torch.bfloat16).cuda()
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).cuda()


def to_host_bits(t: torch.Tensor) -> np.ndarray:
    """Device tensor -> numpy array of its raw bits (for bit-exact compares)."""
    t = t.detach().contiguous().cpu()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()


def assert_rel(gpu: np.ndarray, ref: np.ndarray, tol: float, what: str, abs_floor: float = 0.0):
    gpu = np.asarray(gpu, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert gpu.shape == ref.shape, what
    err = np.abs(gpu - ref)
    bound = tol * np.abs(ref) + abs_floor
    bad = ~(err <= bound)
    if bad.any():
        i = int(np.argmax(np.where(bad, err / np.maximum(bound, 1e-300), 0)))
        raise AssertionError(f"{what}: {int(bad.sum())}/{bad.size} outside tol {tol} "
                             f"(worst at {i}: gpu {gpu.flat[i]!r} ref {ref.flat[i]!r})")


def kept_sets_match(layout, keep_gpu, keep_ref, scores_ref, budget_ref, tol):
    """Kept visual sets per image may differ only in tokens whose oracle score
    lies within ``tol`` (relative) of the image's k-th largest oracle score."""
    g, r = set(int(x) for x in keep_gpu), set(int(x) for x in keep_ref)
    diff = g ^ r
    for j in diff:
        i = int(np.searchsorted(layout.img_start, j, side="right") - 1)
        s0, n = int(layout.img_start[i]), int(layout.img_len[i])
        assert s0 <= j < s0 + n, f"text token {j} differs"
        k = int(budget_ref[i])
        vals = np.sort(scores_ref[s0:s0 + n])[::-1]
        theta = vals[k - 1] if k > 0 else vals[0]
        assert abs(scores_ref[j] - theta) <= tol * abs(theta), \
            f"token {j} (score {scores_ref[j]}) is not near the threshold {theta} of image {i}"
    return len(diff)


def budget_cases():
    """(image lengths, image sums, alpha, floor_abs, mode) of one sequence each:
    1-32 images with empty images, zero sums and both modes, then sequences of
    33 to 256 images."""
    from oracle import avtp_oracle as O

    rng = np.random.default_rng(77)
    cases = []
    for t in range(40):
        m = int(rng.integers(1, 33))
        n = [int(x) for x in rng.integers(1, 1600, size=m)]
        if t % 7 == 0:
            n[0] = 0 if m > 1 else n[0]                 # an empty image
        alpha = [0.0, 1.0, 2.0, 5.0][t % 4]
        floor_abs = [0, 16, 3][t % 3]
        mode = O.BUDGET_RAW if t % 5 == 4 else O.BUDGET_PROPORTIONAL
        S = (rng.lognormal(0.0, 1.0 + (t % 3), size=m) * np.array(n) / 100).astype(np.float32)
        if t % 11 == 3:
            S[:] = 0.0                                  # no importance at all
        if t % 13 == 5:
            S[int(rng.integers(0, m))] = 0.0
        cases.append((n, S, alpha, floor_abs, mode))
    # more images per sequence than 32: the kernel splits each breakpoint's
    # sum over 4 threads up to 32 images, over 2 up to 64, and not above
    for t, m in enumerate([33, 48, 64, 65, 100, 128, 129, 200, 256]):
        n = [int(x) for x in rng.integers(1, 400, size=m)]
        alpha = [1.0, 2.0, 0.0][t % 3]
        floor_abs = [0, 16][t % 2]
        mode = O.BUDGET_RAW if t % 4 == 3 else O.BUDGET_PROPORTIONAL
        S = (rng.lognormal(0.0, 2.0, size=m) * np.array(n) / 100).astype(np.float32)
        cases.append((n, S, alpha, floor_abs, mode))
    return cases
