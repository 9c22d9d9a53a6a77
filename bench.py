#!/usr/bin/env python3
"""Benchmark of the AVTP pruning layer on one MI355X.

One step = one pruning layer over one batch, the four calls of the C ABI on
one stream: avtp_score (row statistics + column-sum passes), avtp_budget,
avtp_select and avtp_compact of hidden states, position ids and the layer's K
and V.  Inputs are seeded synthetic tensors already resident in HBM.

    python bench.py [--steps K] [--warmup W] [--config 5] [--no-cpu-baseline]
                    [--no-per-config]

Prints one JSON line.  ``value`` is visual tokens processed per second for
the whole layer on the headline workload (config 5); ``roofline`` describes
the dominant kernel (timed live with HIP events on the stream the library
launches on); ``cpu_baseline`` times the float64 CPU oracle on a bounded
sample of the same workload.  ``per_config`` repeats the layer measurement
on the other four workloads (time per layer, visual tokens per second, MFMA
fraction of both score passes, HBM fraction of selection + compaction, the
fused selection + compaction against the two calls) with an oracle time for
each (median of 3 runs for configs 1-3 and one run for config 4 on all host
cores, and one single-thread run for configs 1-2).
"""
from __future__ import annotations

import argparse
import ctypes
import json
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, HERE)

METRIC = ("µs per pruning layer + visual tokens scored/s; % MFMA peak (score), "
          "% HBM peak")
PEAK_BF16_TFLOPS = 2500.0      # dense bf16 MFMA, MI355X
PEAK_FP32_MFMA_TFLOPS = 157.3
PEAK_HBM_GBS = 8000.0


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", type=int, default=5, choices=[1, 2, 3, 4, 5])
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-per-config", action="store_true",
                    help="measure only the headline workload")
    ap.add_argument("--sustain-s", type=float, default=3.0, metavar="S",
                    help="after the timed steps, run each score pass back to back for S seconds and "
                         "report its steady-state time (0: off)")
    ap.add_argument("--sustain-only", action="store_true",
                    help="only the sustained loops of the headline workload (e.g. for power sampling)")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                    help="only run a plain device copy of MIB mebibytes (counter calibration)")
    return ap.parse_args()


def source_digest(path):
    import hashlib
    return hashlib.sha256(open(path, "rb").read()).hexdigest()[:16]


def measured_traffic(kernel, workload, src_path):
    """HBM bytes per launch of `kernel` on `workload` from the committed counter
    summary (profiles/hbm_traffic.txt), or None if absent or taken on other source.

    Each line: kernel workload fetch_kib=F write_kib=W copy_read=R copy_write=C src=SHA
    where R and C are FETCH_SIZE / WRITE_SIZE divided by the true bytes of a plain copy.
    """
    path = os.path.join(HERE, "profiles", "hbm_traffic.txt")
    if not os.path.exists(path):
        return None
    want = source_digest(src_path)
    for line in open(path):
        f = line.split()
        if len(f) < 3 or f[0] != kernel or f[1] != workload:
            continue
        kv = dict(x.split("=", 1) for x in f[2:] if "=" in x)
        if kv.get("src") != want:
            return None
        return (float(kv["fetch_kib"]) * 1024 / float(kv["copy_read"])
                + float(kv["write_kib"]) * 1024 / float(kv["copy_write"]))
    return None


def time_sustained(st, seconds: float) -> dict:
    """Each score pass run back to back for `seconds` (after the timed steps):
    the steady-state time per call once the GPU's power controller has
    settled (the first tens of ms of a run are a transient).  Pass 1 is
    avtp_row_lse; pass 2 is avtp_score given that LSE (pass 2, LSE
    conversion, finalize).  Reported beside the timed steps, never as
    `value`."""
    import torch

    from paper_2608_26806_amd import avtp as A

    dl, q, k, lse, ws, wl = st["dl"], st["q"], st["k"], st["lse"], st["ws"], st["wl"]
    scores, isum = st["scores"], st["isum"]
    out = {}
    for name, fn in [("pass1_us", lambda: A.row_lse(dl, q, k, wl.softmax_scale, out=lse, ws=ws)),
                     ("pass2_us", lambda: A.score_attn(dl, q, k, wl.softmax_scale, row_lse=lse,
                                                       scores=scores, img_sum=isum, ws=ws))]:
        fn()
        torch.cuda.synchronize()
        n, t0 = 0, time.perf_counter()
        while time.perf_counter() - t0 < seconds:
            for _ in range(20):
                fn()
            torch.cuda.synchronize()
            n += 20
        out[name] = (time.perf_counter() - t0) / n * 1e6
        out[name.replace("_us", "_calls")] = n
    return out


def time_layer_selection(dl, isum, stream, dev, reps: int = 50) -> dict:
    """Median times of the calibration calls of Sec. 3.3.2 (not part of a pruning
    layer's step): the per-sample attention of one layer on this workload's image
    sums, and the ranking of a 36-layer x 400-sample table (100 samples from each
    of 4 benchmarks, a 36-layer model), k = 4."""
    import torch

    from paper_2608_26806_amd import avtp as A

    rng = np.random.default_rng(36400)
    table = torch.from_numpy(rng.standard_normal((36, 400)).astype(np.float32)).to(dev)
    a_out = torch.empty(max(1, dl.B), dtype=torch.float32, device=dev)
    rs = torch.empty(36, dtype=torch.int32, device=dev)
    sel = torch.empty(4, dtype=torch.int32, device=dev)
    res = {}
    for name, fn in [("layer_attention_us", lambda: A.layer_attention(dl, isum, out=a_out)),
                     ("layer_select_us_36x400_k4", lambda: A.layer_select(table, 4, rs, sel))]:
        fn()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(2 * reps)]
        for r in range(reps):
            ev[2 * r].record(stream)
            fn()
            ev[2 * r + 1].record(stream)
        torch.cuda.synchronize()
        res[name] = float(np.median([ev[2 * r].elapsed_time(ev[2 * r + 1]) for r in range(reps)])) * 1e3
    return res


def time_variation_and_progressive(dl, lay, hid, keep, cu_out, stream, dev, reps: int = 20) -> dict:
    """The VARIATION score (Sec. 3.3.1, row a4) on this workload's hidden states
    with a synthetic h_prior (h + 0.1 N(0,1), seeded), against the HBM roofline
    (2 x hidden x element bytes per visual token); the next-layer layout
    update; and one whole progressive pruning step (score, budget, select,
    compaction of the hidden states, layout update, and the host copy of the
    new layout's index arrays)."""
    import torch

    from paper_2608_26806_amd import avtp as A
    from paper_2608_26806_amd.progressive import ProgressivePruner

    g = torch.Generator(device=dev)
    g.manual_seed(3311)
    h_prior = (hid.float() + 0.1 * torch.randn(hid.shape, generator=g, device=dev)).to(hid.dtype)
    M = int(lay.img_len.sum())
    alg = 2.0 * M * hid.shape[1] * hid.element_size()
    sc = torch.empty(lay.N_tok, dtype=torch.float32, device=dev)
    isum = torch.empty(max(1, lay.n_img), dtype=torch.float32, device=dev)

    def timed(fn):
        fn()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(2 * reps)]
        for r in range(reps):
            ev[2 * r].record(stream)
            fn()
            ev[2 * r + 1].record(stream)
        torch.cuda.synchronize()
        return float(np.median([ev[2 * r].elapsed_time(ev[2 * r + 1]) for r in range(reps)])) * 1e3

    t_var = timed(lambda: A.score_variation(dl, hid, h_prior, scores=sc, img_sum=isum))
    lay_out = A.pruned_layout(dl, keep, cu_out)  # the outputs, allocated once
    t_lay = timed(lambda: A.pruned_layout(dl, keep, cu_out, out=lay_out))
    steps = []
    for _ in range(3):
        pr = ProgressivePruner(dl, h_prior)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        pr.step(hid, keep_pct_next=50)
        torch.cuda.synchronize()
        steps.append((time.perf_counter() - t0) * 1e6)
    gbs = alg / (t_var * 1e-6) / 1e9
    return {"variation_score": {"kernel": "variation_kernel (+ finalize)", "bound": "hbm",
                                "us": t_var, "alg_bytes": alg, "achieved": gbs,
                                "peak": PEAK_HBM_GBS, "unit": "GB/s", "frac": gbs / PEAK_HBM_GBS},
            "pruned_layout_us": t_lay,
            "progressive_step_us_wall": float(np.median(steps))}


def algorithmic_counts(lay, Hq, d, row_bytes_total):
    """Per-launch algorithmic work of each stage.

    pass 1: one q.k product per (head, text row, key at or before the row)
    pass 2: one per (head, text row, visual key before the row)
    compaction: each kept row read once and written once, plus its index.
    """
    vis = lay.visual_mask()
    p1 = p2 = 0
    for b in range(lay.B):
        s0 = int(lay.cu_seqlens[b])
        cum = np.cumsum(vis[s0:int(lay.cu_seqlens[b + 1])])
        for t in range(int(lay.cu_text[b]), int(lay.cu_text[b + 1])):
            p = int(lay.text_pos[t]) - s0
            p1 += p + 1
            p2 += int(cum[p])
    flops1 = 2.0 * d * Hq * p1
    flops2 = 2.0 * d * Hq * p2
    comp_bytes = 2.0 * lay.N_out * row_bytes_total + 4.0 * lay.N_out
    sel_bytes = 4.0 * lay.N_tok + 4.0 * lay.N_out + 8.0 * lay.n_img
    return flops1, flops2, comp_bytes, sel_bytes


def _oracle_threads():
    try:
        from threadpoolctl import threadpool_info
        return max([x.get("num_threads", 1) for x in threadpool_info()] or [1])
    except Exception:  # noqa: BLE001
        return os.cpu_count() or 1


def _oracle_layer(wl, seqs, keep_out=None):
    """The float64 oracle's four stages on sequences `seqs` of the workload:
    scores, budgets, selection and the compaction of those sequences' hidden
    states.  Returns (visual tokens, text rows) processed; if keep_out is a
    dict, it receives each sequence's oracle outputs (for the parity check,
    after the timing)."""
    from oracle import avtp_oracle as O
    from paper_2608_26806_amd.workloads import Layout
    lay = wl.layout
    m_tot = t_tot = 0
    for b in seqs:
        s, isum, _, _ = O.attn_scores(lay, wl.q_text, wl.k, wl.Hq, wl.Hkv, wl.softmax_scale,
                                      wl.dtype, exact_dot=(wl.cfg == 1), seqs=[b])
        i0, i1 = int(lay.cu_img[b]), int(lay.cu_img[b + 1])
        s0, s1 = int(lay.cu_seqlens[b]), int(lay.cu_seqlens[b + 1])
        ta, tb = int(lay.cu_text[b]), int(lay.cu_text[b + 1])
        sub = Layout(np.array([0, s1 - s0], np.int32), (lay.img_start[i0:i1] - s0).astype(np.int32),
                     lay.img_len[i0:i1].copy(), np.array([0, i1 - i0], np.int32),
                     (lay.text_pos[ta:tb] - s0).astype(np.int32), np.array([0, tb - ta], np.int32),
                     lay.keep_total[b:b + 1].copy())
        bud = O.budget(sub, isum[i0:i1].astype(np.float32), wl.alpha, wl.lo_permille,
                       wl.hi_permille, wl.floor_abs)
        keep, _ = O.select(sub, s[s0:s1].astype(np.float32), bud)
        hid = O.compact(keep, wl.hidden_states[s0:s1])
        m_tot += int(lay.img_len[i0:i1].sum())
        t_tot += tb - ta
        if keep_out is not None:
            keep_out[b] = {"scores": s[s0:s1], "isum": isum[i0:i1], "budget": bud, "keep": keep,
                           "hidden": hid, "sub": sub}
    return m_tot, t_tot


def parity_verdict(wl, gpu, orc):
    """The GPU layer's outputs against the oracle's on the sequences the oracle
    ran (gpu: host copies of scores, image sums, budgets, keep_idx, cu_out and
    the compacted hidden states).  Scores and image sums: largest relative
    error (tolerance 2e-3 for bf16, 1e-5 for fp32); budgets: equal to the
    oracle's on the oracle's own sums and on the GPU's; kept tokens: equal
    outside each image's threshold band; compaction: bit-exact given the
    GPU's kept indices."""
    from oracle import avtp_oracle as O
    lay = wl.layout
    tol = 2e-3 if wl.dtype == "bf16" else 1e-5
    err_s = err_i = 0.0
    bud_eq = bud_gpu_eq = comp_eq = True
    outside = 0
    for b, o in orc.items():
        s0, s1 = int(lay.cu_seqlens[b]), int(lay.cu_seqlens[b + 1])
        i0, i1 = int(lay.cu_img[b]), int(lay.cu_img[b + 1])
        sub = o["sub"]
        vis = sub.visual_mask()
        sg = gpu["scores"][s0:s1]
        err_s = max(err_s, float(np.max(np.abs(sg[vis] - o["scores"][vis]) / o["scores"][vis])))
        ig = gpu["isum"][i0:i1]
        err_i = max(err_i, float(np.max(np.abs(ig - o["isum"]) / o["isum"])))
        bg = gpu["budget"][i0:i1]
        bud_eq &= bool(np.array_equal(bg, o["budget"]))
        bud_gpu_eq &= bool(np.array_equal(bg, O.budget(sub, ig, wl.alpha, wl.lo_permille,
                                                       wl.hi_permille, wl.floor_abs)))
        kg = gpu["keep"][gpu["cu_out"][b]:gpu["cu_out"][b + 1]] - s0
        for j in set(kg.tolist()) ^ set(o["keep"].tolist()):
            i = int(np.searchsorted(sub.img_start, j, side="right") - 1)
            st, n = int(sub.img_start[i]), int(sub.img_len[i])
            k = int(o["budget"][i])
            theta = np.sort(o["scores"][st:st + n])[::-1][max(k - 1, 0)]
            outside += int(not (st <= j < st + n and abs(o["scores"][j] - theta) <= tol * theta))
        comp_eq &= bool(np.array_equal(gpu["hidden"][gpu["cu_out"][b]:gpu["cu_out"][b + 1]],
                                       wl.hidden_states[s0:s1][kg]))
    ok = err_s <= tol and err_i <= tol and bud_eq and bud_gpu_eq and outside == 0 and comp_eq
    return {"sequences": sorted(int(b) for b in orc), "tolerance": tol,
            "scores_max_rel_err": err_s, "img_sum_max_rel_err": err_i,
            "budgets_equal_oracle": bud_eq, "budgets_equal_on_gpu_sums": bud_gpu_eq,
            "kept_outside_threshold_band": outside, "compaction_bit_exact": comp_eq, "ok": ok}


def cpu_baseline(wl, nseq=3, keep_out=None):
    """The oracle on the first `nseq` sequences of the workload, all four stages."""
    lay = wl.layout
    nseq = min(nseq, lay.B)
    t0 = time.perf_counter()
    m_tot, t_tot = _oracle_layer(wl, range(nseq), keep_out)
    dt = time.perf_counter() - t0
    return {"value": m_tot / dt, "unit": "visual tokens/s", "cores": int(_oracle_threads()),
            "kind": "oracle",
            "sample": f"first {nseq} of {lay.B} sequences ({m_tot} visual tokens, {t_tot} text rows), "
                      f"all four stages, float64 numpy; {dt:.2f} s"}


def cpu_baseline_config(wl, runs, single_thread, keep_out=None):
    """The oracle on the whole workload: median of `runs` runs on all host
    cores, and (if asked) one run on one thread."""
    lay = wl.layout
    M = int(lay.img_len.sum())
    times = []
    for r in range(runs):
        t0 = time.perf_counter()
        _oracle_layer(wl, range(lay.B), keep_out if r == 0 else None)
        times.append(time.perf_counter() - t0)
    med = float(np.median(times))
    out = {"us_per_layer": med * 1e6, "visual_tokens_per_s": M / med, "cores": int(_oracle_threads()),
           "runs": runs, "kind": "oracle", "sample": "whole workload, all four stages"}
    if single_thread:
        from threadpoolctl import threadpool_limits
        with threadpool_limits(limits=1):
            t0 = time.perf_counter()
            _oracle_layer(wl, range(lay.B))
            t1 = time.perf_counter() - t0
        out["single_thread_us_per_layer"] = t1 * 1e6
        out["single_thread_visual_tokens_per_s"] = M / t1
    return out


def calibrate_copy(mib):
    """A plain device-to-device copy of a known size (reads and writes `mib` MiB),
    run under rocprofv3 to relate FETCH_SIZE / WRITE_SIZE to true bytes."""
    import torch
    n = mib * (1 << 20)
    src = torch.ones(n // 4, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"calibration_copy_bytes": n, "dispatches": 3}))


def _events(stream, fn, reps):
    """Median µs of `fn` over `reps` calls, HIP events on `stream`."""
    import torch
    fn()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2 * reps)]
    for r in range(reps):
        ev[2 * r].record(stream)
        fn()
        ev[2 * r + 1].record(stream)
    torch.cuda.synchronize()
    return float(np.median([ev[2 * r].elapsed_time(ev[2 * r + 1]) for r in range(reps)])) * 1e3


def measure_layer(wl, dev, steps, warmup):
    """Time the pruning layer of one workload; returns (report dict, state).

    The timed step is two calls of the C ABI: avtp_score in its plain
    two-pass form, then avtp_budget_select_compact (budgets, selection and
    the compaction of hidden states, position ids, K and V), each prepared
    once by the binding (arguments marshalled once); the `steps` steps are
    timed together, one HIP event pair around them.  Loops of
    their own, events between the calls, give the split between the two
    calls and the same layer as four calls (avtp_score, avtp_budget,
    avtp_select, avtp_compact) for the per-stage breakdown.  Pass 1 alone (avtp_row_lse: row statistics
    + LSE combine) is timed in a loop of its own; pass 2's time is the score
    call's minus pass 1's."""
    import torch

    from paper_2608_26806_amd import avtp as A

    lay = wl.layout

    def up(x):
        if wl.dtype == "bf16":
            return torch.from_numpy(np.ascontiguousarray(x).view(np.int16)).view(torch.bfloat16).to(dev)
        return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(dev)

    dl = A.DeviceLayout(lay, device=dev)
    q, k, v = up(wl.q_text), up(wl.k), up(wl.v)
    hid = up(wl.hidden_states)
    pos = torch.from_numpy(wl.pos).to(dev)
    dt = A.dtype_code(q)
    ws = A.alloc_workspace(A.score_workspace_bytes(dl, A.SCORE_ATTN, dt, wl.Hq, wl.Hkv, wl.d), dev)
    lse = torch.empty((wl.Hq, lay.T_tot), dtype=torch.float32, device=dev)
    scores = torch.empty(lay.N_tok, dtype=torch.float32, device=dev)
    isum = torch.empty(max(1, lay.n_img), dtype=torch.float32, device=dev)
    bud = torch.empty(max(1, lay.n_img), dtype=torch.int32, device=dev)
    keep = torch.empty(lay.N_out, dtype=torch.int32, device=dev)
    cu_out = torch.empty(lay.B + 1, dtype=torch.int32, device=dev)
    status = torch.zeros(lay.B, dtype=torch.int32, device=dev)
    pairs = []
    for src, tdim in [(hid, 0), (pos, 1), (k, 0), (v, 0)]:
        shape = list(src.shape)
        shape[tdim] = lay.N_out
        pairs.append((src, torch.empty(shape, dtype=src.dtype, device=dev), tdim))
    row_bytes_total = sum(p[0][0].numel() * p[0].element_size() if p[2] == 0 else
                          p[0].shape[0] * p[0][0, 0].numel() * p[0].element_size() for p in pairs)

    stream = torch.cuda.current_stream()
    sh = ctypes.c_void_p(stream.cuda_stream)  # the stream handle, looked up once
    tset = A.TensorSet(pairs)                 # the compaction's descriptors, built once
    score_call = lambda: A.score_attn(dl, q, k, wl.softmax_scale, scores=scores, img_sum=isum,
                                      status=status, ws=ws, stream=sh)
    bargs = (wl.alpha, wl.lo_permille, wl.hi_permille, wl.floor_abs)
    calls = [  # the timed step: the two calls with their arguments marshalled once
        A.prepare_score_attn(dl, q, k, wl.softmax_scale, scores, isum, ws, status=status, stream=sh),
        A.prepare_budget_select_compact(dl, isum, scores, tset, bud, keep, cu_out, *bargs,
                                        status=status, stream=sh),
    ]
    names = ["score", "budget", "select", "compact"]
    calls4 = [  # the same layer as four calls
        score_call,
        lambda: A.budget(dl, isum, *bargs, out=bud, status=status, stream=sh),
        lambda: A.select(dl, scores, bud, keep_idx=keep, cu_out=cu_out, status=status, stream=sh),
        lambda: A.compact(dl, keep, tset, stream=sh),
    ]

    def step(cs, ev=None):
        for j, c in enumerate(cs):
            if ev is not None:
                ev[j].record(stream)
            c()
        if ev is not None:
            ev[len(cs)].record(stream)

    def run(cs, n):
        """n steps of the calls cs, events between the calls; returns the
        per-call times (ms, one row per step), the step times and the wall
        time."""
        events = [[torch.cuda.Event(enable_timing=True) for _ in range(len(cs) + 1)]
                  for _ in range(n)]
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for i in range(n):
            step(cs, events[i])
        torch.cuda.synchronize()
        w = time.perf_counter() - t0
        per_ = np.array([[events[i][j].elapsed_time(events[i][j + 1]) for j in range(len(cs))]
                         for i in range(n)])
        return per_, np.array([events[i][0].elapsed_time(events[i][len(cs)]) for i in range(n)]), w

    for _ in range(warmup):
        step(calls)
    # the timed steps: one event pair around all of them (events between the
    # calls would add their own host time to every step)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    e0.record(stream)
    for _ in range(steps):
        step(calls)
    e1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_layer = e0.elapsed_time(e1) / steps
    per2, _, _ = run(calls, max(steps, 10))            # score / prune split, events between
    per, layer4_ms, _ = run(calls4, max(steps, 10))    # the four-call breakdown
    st = status.cpu().numpy()
    if st.any():
        print(f"warning: device status flags {st.tolist()}", file=sys.stderr)
    reps = max(steps, 10)
    t_p1 = _events(stream, lambda: A.row_lse(dl, q, k, wl.softmax_scale, out=lse, ws=ws, stream=sh),
                   reps) * 1e-3
    # the fused call and the two separate calls, timed the same way (events
    # around each call, or around the pair)
    fused_us = _events(stream, lambda: A.select_compact(dl, scores, bud, tset, keep_idx=keep,
                                                        cu_out=cu_out, status=status, stream=sh),
                       reps)

    def _sep():
        A.select(dl, scores, bud, keep_idx=keep, cu_out=cu_out, status=status, stream=sh)
        A.compact(dl, keep, tset, stream=sh)

    sep_us = _events(stream, _sep, reps)

    # the layer with the row LSE supplied by the caller (the layer's own
    # attention hands it over): pass 2 only, then budget, select, compact
    def _layer_lse():
        A.score_attn(dl, q, k, wl.softmax_scale, row_lse=lse, scores=scores, img_sum=isum,
                     status=status, ws=ws, stream=sh)
        calls[1]()

    lse_layer_us = _events(stream, _layer_lse, reps)

    # the same step captured once in a HIP graph and replayed (no host work
    # per call): what the layer costs the GPU alone, beside the eager steps
    side = torch.cuda.Stream()
    side.wait_stream(stream)
    with torch.cuda.stream(side):
        score_attn_cur = lambda: A.score_attn(dl, q, k, wl.softmax_scale, scores=scores,
                                              img_sum=isum, status=status, ws=ws)
        prune_cur = lambda: A.budget_select_compact(dl, isum, scores, tset, *bargs, budget_out=bud,
                                                    keep_idx=keep, cu_out=cu_out, status=status)
        score_attn_cur()
        prune_cur()
    stream.wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        score_attn_cur()
        prune_cur()
    torch.cuda.synchronize()
    graph.replay()
    g0, g1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    g0.record(stream)
    for _ in range(steps):  # back to back, as the timed steps
        graph.replay()
    g1.record(stream)
    torch.cuda.synchronize()
    graph_us = g0.elapsed_time(g1) / steps * 1e3
    del graph

    M = int(lay.img_len.sum())
    ms = {n: float(np.mean(per[:, j])) for j, n in enumerate(names)}
    ms_score = float(np.mean(per2[:, 0]))
    ms_prune = float(np.mean(per2[:, 1]))
    f1, f2, comp_bytes, sel_bytes = algorithmic_counts(lay, wl.Hq, wl.d, row_bytes_total)
    peak = PEAK_BF16_TFLOPS if wl.dtype == "bf16" else PEAK_FP32_MFMA_TFLOPS
    t_p2 = max(ms_score - t_p1, 1e-9)
    tf1 = f1 / (t_p1 * 1e-3) / 1e12
    tf2 = f2 / (t_p2 * 1e-3) / 1e12
    comp_gbs = comp_bytes / (ms["compact"] * 1e-3) / 1e9
    selcomp_gbs = (comp_bytes + sel_bytes) / ((ms["compact"] + ms["select"]) * 1e-3) / 1e9
    rep = {
        "workload": f"config {wl.cfg}: {wl.name}",
        "dtype": wl.dtype,
        "us_per_layer": ms_layer * 1e3,
        "visual_tokens_per_s": M / (ms_layer * 1e-3),
        "visual_tokens_scored_per_s": M / (ms_score * 1e-3),
        "us_per_call": {"score": ms_score * 1e3, "budget_select_compact": ms_prune * 1e3},
        "four_calls": {"us_per_layer": float(np.median(layer4_ms)) * 1e3,
                       "us_per_call": {n: ms[n] * 1e3 for n in names}},
        "score_passes": {
            "pass1_us": t_p1 * 1e3, "pass2_us": t_p2 * 1e3,
            "pass1_alg_gflop": f1 / 1e9, "pass1_tflops": tf1, "pass1_frac": tf1 / peak,
            "pass2_alg_gflop": f2 / 1e9, "pass2_tflops": tf2, "pass2_frac": tf2 / peak,
            "both_passes_frac": (f1 + f2) / (ms_score * 1e-3) / 1e12 / peak,
            "peak_tflops": peak},
        "roofline_compact": {"bound": "hbm", "achieved": comp_gbs, "peak": PEAK_HBM_GBS,
                             "unit": "GB/s", "frac": comp_gbs / PEAK_HBM_GBS,
                             "alg_bytes": comp_bytes},
        "select_plus_compact_hbm_frac": selcomp_gbs / PEAK_HBM_GBS,
        "layer_with_supplied_lse_us": lse_layer_us,
        "layer_graph_replay_us": graph_us,
        "select_compact_fused": {
            "us": fused_us,
            "hbm_frac": (comp_bytes + sel_bytes) / (fused_us * 1e-6) / 1e9 / PEAK_HBM_GBS,
            "separate_calls_us": sep_us},
    }
    torch.cuda.synchronize()
    host = {"scores": scores.cpu().numpy(), "isum": isum[:lay.n_img].cpu().numpy(),
            "budget": bud[:lay.n_img].cpu().numpy(), "keep": keep.cpu().numpy(),
            "cu_out": cu_out.cpu().numpy(), "hidden": _host_bits(pairs[0][1])}
    state = {"dl": dl, "isum": isum, "hid": hid, "keep": keep, "cu_out": cu_out, "stream": stream,
             "ms_layer": ms_layer, "wall": wall, "M": M, "t_p1": t_p1, "tf1": tf1, "peak": peak,
             "host": host, "q": q, "k": k, "lse": lse, "ws": ws, "wl": wl, "scores": scores,
             "f12": (f1, f2)}
    return rep, state


def _host_bits(t):
    """Device tensor -> numpy array of its raw bits (bf16 as uint16)."""
    import torch
    t = t.detach().contiguous().cpu()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()


def main():
    args = parse()
    if args.calibrate_copy:
        calibrate_copy(args.calibrate_copy)
        return
    if args.gpus != 1:
        print(json.dumps({"error": "runs on one GPU only; --gpus must be 1 (the path is per "
                                   "sequence and would shard over sequences across GPUs)"}))
        sys.exit(2)
    import torch
    from paper_2608_26806_amd import avtp as A
    from paper_2608_26806_amd.workloads import make_workload

    if not torch.cuda.is_available():
        print(json.dumps({"error": "no GPU visible"}))
        sys.exit(1)
    dev = torch.device("cuda:0")
    t_gen = time.perf_counter()
    wl = make_workload(args.config, payload=True)
    lay = wl.layout
    gen_s = time.perf_counter() - t_gen

    if args.sustain_only:
        dl = A.DeviceLayout(lay, device=dev)
        up = (lambda x: torch.from_numpy(np.ascontiguousarray(x).view(np.int16)).view(torch.bfloat16)
              .to(dev)) if wl.dtype == "bf16" else (lambda x: torch.from_numpy(
                  np.ascontiguousarray(x, dtype=np.float32)).to(dev))
        dt = A.BF16 if wl.dtype == "bf16" else A.FP32
        stt = {"dl": dl, "q": up(wl.q_text), "k": up(wl.k), "wl": wl,
               "lse": torch.empty((wl.Hq, lay.T_tot), dtype=torch.float32, device=dev),
               "ws": A.alloc_workspace(A.score_workspace_bytes(dl, A.SCORE_ATTN, dt, wl.Hq, wl.Hkv,
                                                               wl.d), dev),
               "scores": torch.empty(lay.N_tok, dtype=torch.float32, device=dev),
               "isum": torch.empty(max(1, lay.n_img), dtype=torch.float32, device=dev)}
        print(json.dumps({"workload": f"config {args.config}",
                          "sustained": time_sustained(stt, max(args.sustain_s, 1.0))}))
        return
    rep, stt = measure_layer(wl, dev, args.steps, args.warmup)
    sustained = None
    if args.sustain_s > 0:
        sustained = time_sustained(stt, args.sustain_s)
        f1, f2 = stt["f12"]
        pk = stt["peak"]
        sustained["pass1_frac"] = f1 / (sustained["pass1_us"] * 1e-6) / 1e12 / pk
        sustained["both_passes_frac"] = (f1 + f2) / ((sustained["pass1_us"] + sustained["pass2_us"])
                                                     * 1e-6) / 1e12 / pk
        sustained["seconds_per_pass"] = args.sustain_s
    layer_sel = time_layer_selection(stt["dl"], stt["isum"], stt["stream"], dev)
    var_prog = time_variation_and_progressive(stt["dl"], lay, stt["hid"], stt["keep"],
                                              stt["cu_out"], stt["stream"], dev)
    ms_layer = stt["ms_layer"]
    wall = stt["wall"]
    host5 = stt["host"]
    value = stt["M"] / (ms_layer * 1e-3)
    ach = stt["tf1"]
    peak = stt["peak"]
    del stt
    torch.cuda.empty_cache()

    out = {
        "metric": METRIC,
        "value": value,
        "unit": "visual tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_layer,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": wl.dtype,
        "data": "synthetic (seeded; shapes of the paper's LVLMs, no datasets or weights)",
        "config": {"workload": rep["workload"],
                   "batch": lay.B, "visual_tokens": int(lay.img_len.sum()), "text_rows": lay.T_tot,
                   "N_tok": lay.N_tok, "N_out": lay.N_out, "Hq": wl.Hq, "Hkv": wl.Hkv,
                   "head_dim": wl.d, "hidden": wl.hidden, "score_mode": "attn",
                   "parallelism": "none (1 GPU)"},
        "us_per_layer": rep["us_per_layer"],
        "us_per_call": rep["us_per_call"],
        "visual_tokens_scored_per_s": rep["visual_tokens_scored_per_s"],
        "roofline": {
            "kernel": "rowstats_kernel (pass 1: row statistics; timed with its lse combine)",
            "bound": "mfma", "achieved": ach, "peak": peak, "unit": "TFLOP/s",
            "frac": ach / peak,
            "traffic": measured_traffic("rowstats_kernel", f"config{args.config}",
                                        os.path.join(HERE, "paper_2608_26806_amd", "csrc",
                                                     "score_attn.hip"))},
        "score_passes": rep["score_passes"],
        "score_passes_sustained": sustained,
        "roofline_compact": rep["roofline_compact"],
        "select_plus_compact_hbm_frac": rep["select_plus_compact_hbm_frac"],
        "layer_with_supplied_lse_us": rep["layer_with_supplied_lse_us"],
        "layer_graph_replay_us": rep["layer_graph_replay_us"],
        "select_compact_fused": rep["select_compact_fused"],
        "layer_selection": layer_sel,
        "variation_and_progressive": var_prog,
        "wall_s_timed_region": wall,
        "input_generation_s": gen_s,
    }
    per = {}
    others = [] if args.no_per_config else [c for c in (1, 2, 3, 4) if c != args.config]
    wls, hosts = {}, {}
    for c in others:
        wc = make_workload(c, payload=True)
        r, stc = measure_layer(wc, dev, max(5, args.steps // 2), max(2, args.warmup))
        hosts[c] = stc["host"]
        del stc
        torch.cuda.empty_cache()
        per[str(c)] = r
        wls[c] = wc
    if not args.no_cpu_baseline:
        orc = {}
        out["cpu_baseline"] = cpu_baseline(wl, keep_out=orc)
        out["parity"] = parity_verdict(wl, host5, orc)
        for c, wc in wls.items():
            orc = {}
            per[str(c)]["cpu_baseline"] = cpu_baseline_config(wc, runs=3 if c <= 3 else 1,
                                                              single_thread=c <= 2, keep_out=orc)
            per[str(c)]["parity"] = parity_verdict(wc, hosts[c], orc)
    if per:
        out["per_config"] = per
    print(json.dumps(out))


if __name__ == "__main__":
    main()
