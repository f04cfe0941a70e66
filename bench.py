#!/usr/bin/env python3
"""Benchmark of the fused attention forward on one MI355X.

One step = one forward pass of the whole hot path (one kernel launch; in split mode the part kernel
and the merge kernel) over one batch of seeded synthetic input already resident in HBM. Prints ONE
JSON line:

* value      -- whole-job GEMM TFLOP/s: 2*B*Hq*Sq*Sk*(d_qk+d_v) (halved for causal) per step, over
                the wall-clock time of the timed steps (bracketed by device synchronisation)
* roofline   -- the step's achieved rate from HIP events around each launch on the launch stream,
                against the bf16 dense MFMA peak (TFLOP/s) or, for workloads whose operational
                intensity at HBM is below the ridge point (decode shapes), the HBM peak (GB/s of
                algorithmic bytes); HBM traffic from the committed rocprofv3 counter summary when it
                was taken on the current kernel source (default workload only)
* cpu_baseline -- the fp64 oracle timed on this host on a bounded sample of the same workload
* parity     -- a few seeded rows per head compared with the oracle (outside the timed region)

Default workload: the long-context GQA prefill, B1 Hq32 Hkv8 S131072 d128 causal (config 5, the
largest of the five configurations); ``--config N`` selects another. Split mode: ``--split N|auto``
with ``--workload decode-128k`` (and the other named decode shapes); ``--decode`` runs the
decode-shaped path (query heads of a group packed into 32-column blocks) on those shapes.

``--cold`` writes a 512 MiB buffer before every timed launch (outside the events around it), so each
launch starts with the 4 MB L2s and the 256 MB Infinity Cache holding none of its inputs; ``--ramp N``
prints the event time of each of N back-to-back launches from the first one on (clock and cache
warm-up). ``--ceilings`` runs the measured-ceiling microbenchmarks instead
(``paper_2609_21264_amd/ceilings.py``).

``--unfused`` times the layer-by-layer baseline (scores, mask + softmax, P V with S and P spilled to
HBM in bf16) on the same workload instead and prints one JSON line with each operator's HBM roofline
and the fused kernel's time on the same inputs (the paper's layer-by-layer vs. fused comparison).
"""

from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2516.6  # 256 CUs x 4096 dense bf16 FLOP/clk/CU x 2.4 GHz
PEAK_HBM_GBS = 8000.0      # HBM3E
# Device code whose measurements the committed profiles certify: every kernel and the headers they
# share (the host-side argument checks of fa_api.hip are not part of it).
KERNEL_SOURCES = ["paper_2609_21264_amd/csrc/fa_fwd_kernel.hip", "paper_2609_21264_amd/csrc/fa_decode_kernel.hip",
                  "paper_2609_21264_amd/csrc/fa_lbl_kernel.hip", "paper_2609_21264_amd/csrc/fa_internal.h",
                  "paper_2609_21264_amd/csrc/fa_device.h"]


def _code_tokens(text: str) -> str:
    """The source with its comments removed and every run of whitespace made one space: what the
    compiler sees, so that editing a comment does not orphan the profiles measured on that code."""
    out, i, n = [], 0, len(text)
    while i < n:
        c = text[i]
        if c in "\"'":  # string or character literal, copied through its closing quote
            j = i + 1
            while j < n and text[j] != c:
                j += 2 if text[j] == "\\" else 1
            out.append(text[i:j + 1])
            i = j + 1
        elif text.startswith("//", i):
            j = text.find("\n", i)
            i = n if j < 0 else j
        elif text.startswith("/*", i):
            j = text.find("*/", i + 2)
            out.append(" ")
            i = n if j < 0 else j + 2
        else:
            out.append(c)
            i += 1
    return " ".join("".join(out).split())


def kernel_source_hash() -> str:
    """sha256[:16] of the device sources' code (comments and layout ignored)."""
    h = hashlib.sha256()
    for rel in KERNEL_SOURCES:
        with open(os.path.join(ROOT, rel), encoding="utf-8") as f:
            h.update(_code_tokens(f.read()).encode())
        h.update(b"\0")
    return h.hexdigest()[:16]


def traffic_from_profile(config: int):
    """HBM bytes per launch from the committed counter summary, if it matches the current kernel."""
    path = os.path.join(ROOT, "profiles", f"fa_fwd_config{config}_hbm_traffic.txt")
    if not os.path.exists(path):
        return None
    fields = {}
    for line in open(path):
        m = re.match(r"^\s*([a-z0-9_]+)\s*[:=]\s*([0-9a-fA-Fx.eE+-]+)\s*$", line)
        if m:
            fields[m.group(1)] = m.group(2)
    if fields.get("kernel_source_sha256_16") != kernel_source_hash():
        return None
    try:
        return float(fields["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def blas_threads() -> int:
    """Threads NumPy's BLAS runs with (threadpoolctl when present, else OMP_NUM_THREADS, else 1)."""
    import numpy as np

    try:
        import threadpoolctl

        (np.ones((4, 4)) @ np.ones((4, 4)))  # loads the BLAS so that threadpoolctl sees it
        info = threadpoolctl.threadpool_info()
        if info:
            return max(i["num_threads"] for i in info)
    except Exception:
        pass
    try:
        return int(os.environ.get("OMP_NUM_THREADS", "1"))
    except ValueError:
        return 1


def cpu_baseline(w, q, k, v, budget_s: float):
    """Time the fp64 oracle on this host on a bounded sample of workload ``w``.

    Problems of at most 2^27 score elements per head are timed on whole heads (every query row);
    larger ones on the seeded 64-row subset of every head that the parity tests use (plus rows 0
    and Sq-1). Key/value groups (one K/V head and its query heads) are timed one after another until
    ``budget_s`` has elapsed. The oracle's time grows linearly with the rows it computes (each row
    is a full row of scores), so the time of the whole problem is the measured time scaled by
    (B*Hq*Sq) / rows timed; the value is the workload's metric FLOPs over that time.
    """
    import numpy as np

    import workloads as W
    from oracle import bf16_bits_to_f64, naive_attention_rows

    def f64(t):
        return bf16_bits_to_f64(t.contiguous().view(__import__("torch").int16).numpy())

    whole = w.Sq * w.Sk <= (1 << 27)
    rows = [np.arange(w.Sq)] * (w.B * w.Hq) if whole else W.sample_rows(w, n=64)
    G = w.group
    t_oracle, n_heads, n_rows = 0.0, 0, 0
    for b in range(w.B):
        for g in range(w.Hkv):
            rs = [rows[b * w.Hq + g * G + m] for m in range(G)]
            t0 = time.perf_counter()
            naive_attention_rows(lambda bb, hh, r: f64(q[b, g * G + hh][r]), lambda bb, gg: f64(k[b, g]),
                                 lambda bb, gg: f64(v[b, g]), 1, G, 1, w.Sq, w.scale, w.causal, rs)
            t_oracle += time.perf_counter() - t0
            n_heads += G
            n_rows += sum(len(r) for r in rs)
            if t_oracle >= budget_s:
                break
        if t_oracle >= budget_s:
            break
    total_rows = w.B * w.Hq * w.Sq
    t_full = t_oracle * total_rows / n_rows
    tflops = W.metric_flops(w) / t_full / 1e12
    what = "every row" if whole else f"{n_rows // n_heads}-row seeded subsets (64 rows + rows 0 and Sq-1)"
    return {"value": tflops, "unit": "TFLOP/s", "cores": blas_threads(), "kind": "oracle",
            "sample": f"{n_heads} of {w.B * w.Hq} query heads, {what}: {n_rows} rows in {t_oracle:.1f} s of fp64 "
                      f"NumPy, scaled x{total_rows / n_rows:.1f} to the whole problem ({t_full:.0f} s); metric FLOPs",
            "measured_s": round(t_oracle, 4), "rows_timed": n_rows, "extrapolated_s": round(t_full, 3),
            "host_cpu_count": os.cpu_count(),
            "host_cpus_usable": len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else None}


def parity_sample(w, q, k, v, o, lse, rows_per_head: int = 4):
    import numpy as np

    import workloads as W
    from oracle import bf16_bits_to_f64, naive_attention_rows

    def f64(t):
        return bf16_bits_to_f64(t.contiguous().view(__import__("torch").int16).numpy())

    rows = W.sample_rows(w, n=rows_per_head, seed_base=3000)
    res = naive_attention_rows(lambda b, h, r: f64(q[b, h][r]), lambda b, g: f64(k[b, g]),
                               lambda b, g: f64(v[b, g]), w.B, w.Hq, w.Hkv, w.Sq, w.scale, w.causal, rows)
    oc, lc = o.cpu(), lse.cpu()
    max_abs, lse_max, n, err_sum, n_el = 0.0, 0.0, 0, 0.0, 0
    for idx, (o_ref, l_ref) in enumerate(res):
        b, h = divmod(idx, w.Hq)
        r = rows[idx]
        og = f64(oc[b, h][r])
        err = np.abs(og - o_ref)
        max_abs = max(max_abs, float(err.max()) if err.size else 0.0)
        err_sum += float(err.sum())
        n_el += err.size
        fin = np.isfinite(l_ref)
        if fin.any():
            lse_max = max(lse_max, float(np.abs(lc[b, h][r].double().numpy()[fin] - l_ref[fin]).max()))
        n += len(r)
    mean_abs = err_sum / max(n_el, 1)
    return {"rows_checked": n, "max_abs": max_abs, "mean_abs": mean_abs, "lse_max_abs": lse_max,
            "pass": bool(max_abs <= 2e-2 and mean_abs <= 2e-3 and lse_max <= 1e-3)}


def paper_sweep():
    """Steady-state timing of the paper's shapes; one JSON line. For each shape: 0.3 s of warmup
    launches, then at least 20 launches and 0.2 s timed with events on the launch stream."""
    import torch

    import paper_2609_21264_amd as fa
    import workloads as W

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream(dev)
    rows = []
    for source, w, paper_us in W.PAPER_SWEEP:
        q, k, v = (x.to(dev) for x in W.make_inputs(w))
        o = torch.empty((w.B, w.Hq, w.Sq, w.dv), dtype=torch.bfloat16, device=dev)
        lse = torch.empty((w.B, w.Hq, w.Sq), dtype=torch.float32, device=dev)

        def step():
            st = fa.fa_fwd_ex(q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(), lse.data_ptr(), w.B, w.Hq,
                              w.Hkv, w.Sq, w.Sk, w.dqk, w.dv, w.scale, w.causal, stream.cuda_stream)
            if st != 0:
                raise fa.FaError(st)

        torch.cuda.synchronize()
        t_w, n_w = time.perf_counter(), 0
        while n_w < 10 or time.perf_counter() - t_w < 0.3:
            step()
            n_w += 1
            torch.cuda.synchronize()
        per = (time.perf_counter() - t_w) / n_w
        n = max(20, int(0.2 / per) + 1)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(n):
            step()
        e1.record(stream)
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / n
        ns_flops = W.metric_flops(w)
        paper_flops = W.paper_flops(w.Hq, w.Sq, w.Sk, w.dqk, w.dv, w.B)
        rows.append({"source": source, "shape": w.name, "H": w.Hq, "Hkv": w.Hkv, "S": w.Sq, "d": w.dqk,
                     "causal": w.causal, "ms": round(ms, 4),
                     "tflops_metric": round(ns_flops / (ms * 1e-3) / 1e12, 2),
                     "tflops_paper_convention": round(paper_flops / (ms * 1e-3) / 1e12, 2),
                     "paper_xdna2_ms": paper_us / 1e3, "speedup_vs_paper_xdna2": round(paper_us / 1e3 / ms, 1)})
        print(f"[sweep] {w.name}: {ms:.4f} ms, {rows[-1]['tflops_metric']} TFLOP/s", file=sys.stderr, flush=True)
        del q, k, v, o, lse
    print(json.dumps({"metric": "attention fwd on the paper's shapes, 1 MI355X", "unit": "ms / TFLOP/s",
                      "data": "synthetic", "dtype": "bf16", "n_gpus": 1,
                      "note": "tflops_metric halves causal FLOPs; tflops_paper_convention does not (the paper's "
                              "P_effGEMM); paper_xdna2_ms is the paper's measured latency on its NPU (context)",
                      "rows": rows}), flush=True)


def unfused_main(args, w):
    """The layer-by-layer path on workload w: each operator timed with HIP events on the launch stream
    (when the whole problem fits one spill buffer), the three-launch step timed by wall clock, and the
    fused kernel on the same inputs for the ratio. One JSON line."""
    import numpy as np
    import torch

    import paper_2609_21264_amd as fa
    import workloads as W
    from oracle import bf16_bits_to_f64, lbl_error_bound, naive_attention_rows

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    print(f"[bench] unfused, workload: {w.name}", file=sys.stderr, flush=True)
    q_cpu, k_cpu, v_cpu = W.make_inputs(w)
    q, k, v = q_cpu.to(dev), k_cpu.to(dev), v_cpu.to(dev)
    o = torch.empty((w.B, w.Hq, w.Sq, w.dv), dtype=torch.bfloat16, device=dev)
    lse = torch.empty((w.B, w.Hq, w.Sq), dtype=torch.float32, device=dev)
    handle = torch.cuda.current_stream(dev).cuda_stream
    stream = torch.cuda.current_stream(dev)
    full = fa.fa_lbl_workspace_bytes(w.B, w.Hq, w.Sq, w.Sk)
    cap = int(args.workspace_gib * (1 << 30))
    ws_bytes = min(full, cap)
    ws = torch.empty(max(ws_bytes, 16), dtype=torch.uint8, device=dev)
    one_chunk = ws_bytes >= full
    args_common = (w.B, w.Hq, w.Hkv, w.Sq, w.Sk)

    def ok(st):
        if st != 0:
            raise fa.FaError(st)

    def op_scores():
        ok(fa.fa_lbl_scores(q.data_ptr(), k.data_ptr(), ws.data_ptr(), *args_common, w.dqk, w.scale, w.causal,
                            handle))

    def op_softmax():
        ok(fa.fa_lbl_softmax(ws.data_ptr(), ws.data_ptr(), lse.data_ptr(), w.B, w.Hq, w.Sq, w.Sk, w.causal, handle))

    def op_pv():
        ok(fa.fa_lbl_pv(ws.data_ptr(), v.data_ptr(), o.data_ptr(), *args_common, w.dv, w.causal, handle))

    def step_unfused():
        ok(fa.fa_fwd_unfused(q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(), lse.data_ptr(), *args_common,
                             w.dqk, w.dv, w.scale, w.causal, ws.data_ptr(), ws_bytes, handle))

    def step_fused():
        ok(fa.fa_fwd_ex(q.data_ptr(), k.data_ptr(), v.data_ptr(), o_f.data_ptr(), None, *args_common, w.dqk, w.dv,
                        w.scale, w.causal, handle))

    o_f = torch.empty_like(o)

    def timed(fn, min_s=0.25, min_n=10, warm_s=0.3):
        t = time.perf_counter()
        nw = 0
        while nw < 3 or time.perf_counter() - t < warm_s:
            fn()
            nw += 1
            torch.cuda.synchronize()
        per = (time.perf_counter() - t) / nw
        n = max(min_n, int(min_s / max(per, 1e-6)) + 1)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(n):
            fn()
        torch.cuda.synchronize()
        return (time.perf_counter() - t0) / n, n, nw

    step_s, steps, warm = timed(step_unfused)
    print(f"[bench] unfused step {step_s * 1e3:.4f} ms ({steps} timed)", file=sys.stderr, flush=True)
    fused_s, _, _ = timed(step_fused)
    print(f"[bench] fused step {fused_s * 1e3:.4f} ms", file=sys.stderr, flush=True)

    kernels = None
    alg = W.unfused_algorithmic_bytes(w)
    if one_chunk:
        # Per operator: events around each launch on the launch stream, over the same number of steps.
        names = ("scores", "softmax", "pv")
        evs = {n: [] for n in names}
        for _ in range(3):
            op_scores(); op_softmax(); op_pv()
        torch.cuda.synchronize()
        for _ in range(steps):
            for n, fn in zip(names, (op_scores, op_softmax, op_pv)):
                a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                a.record(stream)
                fn()
                b.record(stream)
                evs[n].append((a, b))
        torch.cuda.synchronize()
        kernels = {}
        for n in names:
            ms = [a.elapsed_time(b) for a, b in evs[n]]
            avg = sum(ms) / len(ms)
            gbs = alg[n] / (avg / 1e3) / 1e9
            kernels[n] = {"ms": round(avg, 4), "algorithmic_bytes": alg[n], "achieved_gbs": round(gbs, 1),
                          "frac_of_hbm_peak": round(gbs / PEAK_HBM_GBS, 4)}
        # the output checked below comes from the composite call
        step_unfused()
        torch.cuda.synchronize()

    if args.copy_calibration > 0:
        n = args.copy_calibration * (1 << 20) // 4
        src = torch.ones(n, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(f"[bench] copy calibration: 3 x {args.copy_calibration} MiB device copies", file=sys.stderr, flush=True)
        del src, dst

    # Parity on sampled rows against exact attention, within the bound of the three bf16 roundings
    # plus fp32 slack (2^-12 max|V| on O, 2^-12 on LSE).
    def f64(t):
        return bf16_bits_to_f64(t.contiguous().view(torch.int16).numpy())

    rows = W.sample_rows(w, n=4, seed_base=3000)
    res = naive_attention_rows(lambda b, h, r: f64(q_cpu[b, h][r]), lambda b, g: f64(k_cpu[b, g]),
                               lambda b, g: f64(v_cpu[b, g]), w.B, w.Hq, w.Hkv, w.Sq, w.scale, w.causal, rows)
    oc, lc = o.cpu(), lse.cpu()
    worst, worst_lse, n_rows = 0.0, 0.0, 0
    for idx, (o_ref, l_ref) in enumerate(res):
        b, h = divmod(idx, w.Hq)
        g = h // w.group
        r = rows[idx]
        s = w.scale * (f64(q_cpu[b, h][r]) @ f64(k_cpu[b, g]).T)
        if w.causal:
            s = np.where(np.arange(w.Sk)[None, :] <= r[:, None] + (w.Sk - w.Sq), s, 0.0)
        m = np.abs(s).max(axis=1) if w.Sk else np.zeros(len(r))
        vmax = float(np.abs(f64(v_cpu[b, g])).max()) if w.Sk else 0.0
        bound = lbl_error_bound(m, vmax) + 2.0 ** -12 * vmax
        err = np.abs(f64(oc[b, h][r]) - o_ref).max(axis=1)
        worst = max(worst, float((err / np.maximum(bound, 1e-30)).max()))
        fin = np.isfinite(l_ref)
        if fin.any():
            lerr = np.abs(lc[b, h][r].double().numpy()[fin] - l_ref[fin]) / (2.0 ** -8 * m[fin] + 2.0 ** -12)
            worst_lse = max(worst_lse, float(lerr.max()))
        n_rows += len(r)
    parity = {"rows_checked": n_rows, "worst_o_err_over_bound": round(worst, 4),
              "worst_lse_err_over_bound": round(worst_lse, 4), "pass": bool(worst <= 1 and worst_lse <= 1)}
    print(f"[bench] parity sample: {parity}", file=sys.stderr, flush=True)

    flops = W.metric_flops(w)
    total = sum(alg.values())
    value = flops / step_s / 1e12
    dominant = max(kernels, key=lambda n: kernels[n]["ms"]) if kernels else None
    roof = None
    if kernels:
        kd = kernels[dominant]
        roof = {"bound": "hbm", "kernel": f"lbl_{dominant}_kernel", "achieved": kd["achieved_gbs"],
                "peak": PEAK_HBM_GBS, "unit": "GB/s", "frac": kd["frac_of_hbm_peak"], "traffic": None,
                "kernels": kernels}
    out = {
        "metric": "attention fwd GEMM TFLOP/s on 1 MI355X, unfused layer-by-layer path",
        "value": round(value, 3),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": steps,
        "warmup": warm,
        "ms_per_step": round(step_s * 1e3, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": w.name, "B": w.B, "Hq": w.Hq, "Hkv": w.Hkv, "Sq": w.Sq, "Sk": w.Sk,
                   "d_qk": w.dqk, "d_v": w.dv, "causal": w.causal, "path": "unfused",
                   "spill_buffer_bytes": ws_bytes, "chunks": "one" if one_chunk else "several"},
        "operational_intensity_flop_per_byte": round(flops / total, 2),
        "hbm_bound_tflops": round(PEAK_HBM_GBS * 1e9 * flops / total / 1e12, 1),
        "algorithmic_bytes_per_step": total,
        "roofline": roof,
        "fused": {"ms": round(fused_s * 1e3, 4), "tflops": round(flops / fused_s / 1e12, 3),
                  "algorithmic_bytes": W.algorithmic_bytes(w)},
        "fused_speedup": round(step_s / fused_s, 3),
        "parity": parity,
    }
    print(json.dumps(out), flush=True)


def ramp_main(args, w, step, stream):
    """Event times of ``args.ramp`` back-to-back launches from the very first one (no warmup): how
    many launches the GPU's clocks and caches take to settle. One JSON line."""
    import torch

    torch.cuda.synchronize()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.ramp)]
    for s, e in ev:
        s.record(stream)
        step()
        e.record(stream)
    torch.cuda.synchronize()
    ms = [s.elapsed_time(e) for s, e in ev]
    n = len(ms)
    windows = {}
    for lo, hi in ((0, 1), (1, 10), (10, 50), (50, 100), (100, 200), (200, 400), (400, 800), (800, n)):
        if lo < n and lo < hi:
            part = ms[lo:min(hi, n)]
            windows[f"{lo}-{min(hi, n) - 1}"] = round(sum(part) / len(part), 4)
    import workloads as W

    flops = W.metric_flops(w)
    tail = ms[n // 2:]
    print(json.dumps({"metric": "per-launch kernel time from a cold start (event pairs on the launch stream)",
                      "unit": "ms", "config": {"workload": w.name}, "launches": n,
                      "window_mean_ms": windows,
                      "first_launch_ms": round(ms[0], 4),
                      "second_half_mean_ms": round(sum(tail) / len(tail), 4),
                      "second_half_tflops": round(flops / (sum(tail) / len(tail) / 1e3) / 1e12, 1),
                      "ms": [round(x, 4) for x in ms]}), flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=-1,
                    help="timed steps; default: at least 20 and at least 0.25 s of launches")
    ap.add_argument("--warmup", type=int, default=-1,
                    help="untimed steps first; default: at least 10 and at least 0.5 s (the first tens of "
                         "milliseconds of back-to-back launches run slower while clocks and caches settle)")
    ap.add_argument("--config", type=int, default=5, choices=[1, 2, 3, 4, 5])
    ap.add_argument("--workload", default=None,
                    help="a named further workload instead of --config (split-mode shapes: "
                         "decode-128k, decode16-128k-causal, decode-b8-8k)")
    ap.add_argument("--shape", default=None, metavar="B,Hq,Hkv,Sq,Sk,d_qk,d_v,causal",
                    help="any other problem instead of --config, e.g. 1,32,8,16384,16384,128,128,1 (seeded "
                         "N(0,1) inputs, scale 1/sqrt(d_qk))")
    ap.add_argument("--paper-sweep", action="store_true",
                    help="time the paper's own shapes (Table 5 GPT-2 Small sweep and the 12 Table 6 models) "
                         "and print one JSON line with a row per shape, in both FLOP conventions")
    ap.add_argument("--split", default=None,
                    help="run split mode (fa_fwd_split) with this many key-range parts, or 'auto'")
    ap.add_argument("--decode", action="store_true",
                    help="run the decode-shaped path (fa_fwd_decode; parts from --split, default 'auto')")
    ap.add_argument("--unfused", action="store_true",
                    help="time the layer-by-layer baseline (three kernels, S and P spilled) instead, with the "
                         "fused kernel on the same inputs for comparison")
    ap.add_argument("--workspace-gib", type=float, default=64.0,
                    help="largest spill buffer for --unfused (bigger problems run in chunks)")
    ap.add_argument("--cpu-budget", type=float, default=12.0, help="seconds of oracle time for cpu_baseline")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cold", action="store_true",
                    help="write a 512 MiB buffer before each timed launch (outside its events): no input is "
                         "cache-resident when a launch starts; the value is then computed from the events")
    ap.add_argument("--ramp", type=int, default=0, metavar="N",
                    help="instead of the normal run: time N back-to-back launches from the very first one with "
                         "events and print their times (how long clocks and caches take to settle)")
    ap.add_argument("--ceilings", action="store_true",
                    help="run the measured-ceiling microbenchmarks (MFMA rate and clock, HBM streams through VGPR "
                         "and direct-to-LDS loads, LDS reads) and print one JSON line")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="after the timed steps, run 3 plain device-to-device copies of MIB MiB (a reference "
                         "kernel of known traffic for scaling rocprofv3 FETCH_SIZE / WRITE_SIZE)")
    args = ap.parse_args()

    if args.gpus != 1:
        print(f"bench.py measures one GPU only (got --gpus {args.gpus}): the fused attention kernel runs on a "
              "single MI355X and the library has no multi-GPU path.", file=sys.stderr)
        sys.exit(2)
    if args.paper_sweep:
        paper_sweep()
        return
    if args.ceilings:
        from paper_2609_21264_amd import ceilings

        ceilings.main()
        return

    import torch

    import paper_2609_21264_amd as fa
    import workloads as W

    if args.shape:
        B, Hq, Hkv, Sq, Sk, dqk, dv, causal = (int(x) for x in args.shape.split(","))
        w = W.small(f"B{B} Hq{Hq} Hkv{Hkv} Sq{Sq} Sk{Sk} dqk{dqk} dv{dv}" + (" causal" if causal else ""), B=B, Hq=Hq,
                    Hkv=Hkv, Sq=Sq, Sk=Sk, dqk=dqk, dv=dv, causal=bool(causal), seed=5000)
        args.workload = w.name  # no committed counter summary for it: traffic stays null
    else:
        w = W.EXTRA[args.workload] if args.workload else W.CONFIGS[args.config]
    if args.unfused:
        unfused_main(args, w)
        return
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    print(f"[bench] workload: {w.name}", file=sys.stderr, flush=True)
    q_cpu, k_cpu, v_cpu = W.make_inputs(w)
    q, k, v = q_cpu.to(dev), k_cpu.to(dev), v_cpu.to(dev)
    o = torch.empty((w.B, w.Hq, w.Sq, w.dv), dtype=torch.bfloat16, device=dev)
    lse = torch.empty((w.B, w.Hq, w.Sq), dtype=torch.float32, device=dev)
    stream = torch.cuda.current_stream(dev)
    handle = stream.cuda_stream

    n_split = 0
    if args.decode:
        n_split = (fa.fa_fwd_decode_parts(torch.cuda.get_device_properties(dev).multi_processor_count, w.B, w.Hq,
                                          w.Hkv, w.Sq, w.Sk)
                   if args.split in (None, "auto") else int(args.split))
        ws_bytes = fa.fa_fwd_split_workspace_bytes(w.B, w.Hq, w.Sq, w.dv, n_split)
        ws = torch.empty(max(ws_bytes, 1), dtype=torch.uint8, device=dev)  # allocated before timing
    elif args.split is not None:
        n_split = (fa.fa_fwd_split_parts(torch.cuda.get_device_properties(dev).multi_processor_count, w.B, w.Hq,
                                         w.Sq, w.Sk, w.dqk, w.dv, w.causal)
                   if args.split == "auto" else int(args.split))
        ws_bytes = fa.fa_fwd_split_workspace_bytes(w.B, w.Hq, w.Sq, w.dv, n_split)
        ws = torch.empty(max(ws_bytes, 1), dtype=torch.uint8, device=dev)  # allocated before timing

    def step():
        if args.decode:
            st = fa.fa_fwd_decode(q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(), lse.data_ptr(), w.B,
                                  w.Hq, w.Hkv, w.Sq, w.Sk, w.dqk, w.dv, w.scale, w.causal, n_split, ws.data_ptr(),
                                  ws_bytes, handle)
        elif n_split:
            st = fa.fa_fwd_split(q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(), lse.data_ptr(), w.B,
                                 w.Hq, w.Hkv, w.Sq, w.Sk, w.dqk, w.dv, w.scale, w.causal, n_split, ws.data_ptr(),
                                 ws_bytes, handle)
        else:
            st = fa.fa_fwd_ex(q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(), lse.data_ptr(), w.B, w.Hq,
                              w.Hkv, w.Sq, w.Sk, w.dqk, w.dv, w.scale, w.causal, handle)
        if st != 0:
            raise fa.FaError(st)

    if args.ramp > 0:
        ramp_main(args, w, step, stream)
        return

    flush = None
    if args.cold:
        flush = torch.empty(512 << 20, dtype=torch.uint8, device=dev)

    step_s = None  # wall time per step seen during warmup
    if args.warmup >= 0:
        for _ in range(args.warmup):
            step()
        torch.cuda.synchronize()
    else:
        # Warm up for a fixed time rather than a fixed count; the count done is what is reported.
        args.warmup = 0
        t_w = time.perf_counter()
        while args.warmup < 10 or time.perf_counter() - t_w < 0.5:
            for _ in range(max(1, min(64, args.warmup))):
                step()
                args.warmup += 1
            torch.cuda.synchronize()
        step_s = (time.perf_counter() - t_w) / args.warmup
    print(f"[bench] warmup done ({args.warmup} steps)", file=sys.stderr, flush=True)
    if args.steps < 0:
        if step_s is None:
            t_p = time.perf_counter()
            step()
            torch.cuda.synchronize()
            step_s = time.perf_counter() - t_p
        args.steps = max(20, int(0.25 / max(step_s, 1e-6)) + 1)

    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for s, e in ev:
        if flush is not None:
            flush.fill_(1)  # outside the event pair
        s.record(stream)
        step()
        e.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    launch_ms = [s.elapsed_time(e) for s, e in ev]
    print(f"[bench] timed {args.steps} steps in {wall:.4f} s", file=sys.stderr, flush=True)
    if flush is not None:
        # the wall clock includes the flushes: the whole-job rate comes from the launches' events
        wall = sum(launch_ms) / 1e3
        del flush

    flops = W.metric_flops(w)
    value = flops * args.steps / wall / 1e12
    avg_launch_s = sum(launch_ms) / len(launch_ms) / 1e3
    achieved = flops / avg_launch_s / 1e12
    traffic = traffic_from_profile(args.config) if not args.workload and not n_split and not args.cold else None
    kernel_name = ("fa_decode_kernel + fa_merge_kernel" if args.decode else
                   "fa_fwd_kernel (split) + fa_merge_kernel" if n_split else "fa_fwd_kernel")
    # Bound by operational intensity at HBM (metric FLOPs over algorithmic bytes) against the ridge
    # point of the two peaks.
    nbytes = W.algorithmic_bytes(w)
    hbm_bound = flops / nbytes < PEAK_BF16_TFLOPS * 1e12 / (PEAK_HBM_GBS * 1e9)
    if hbm_bound:
        ach_gbs = nbytes / avg_launch_s / 1e9
        roof = {"bound": "hbm", "achieved": round(ach_gbs, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                "frac": round(ach_gbs / PEAK_HBM_GBS, 4)}
    else:
        roof = {"bound": "mfma", "achieved": round(achieved, 3), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                "frac": round(achieved / PEAK_BF16_TFLOPS, 4)}

    if args.copy_calibration > 0:
        n = args.copy_calibration * (1 << 20) // 4
        src = torch.ones(n, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(f"[bench] copy calibration: 3 x {args.copy_calibration} MiB device copies", file=sys.stderr, flush=True)
        del src, dst

    parity = parity_sample(w, q_cpu, k_cpu, v_cpu, o, lse)
    print(f"[bench] parity sample: {parity}", file=sys.stderr, flush=True)
    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(w, q_cpu, k_cpu, v_cpu, args.cpu_budget)
        print(f"[bench] cpu baseline: {cpu}", file=sys.stderr, flush=True)

    out = {
        "metric": "attention fwd GEMM TFLOP/s on 1 MI355X; % of bf16 MFMA peak",
        "value": round(value, 3),
        "unit": "TFLOP/s",
        "pct_of_bf16_peak": round(100.0 * value / PEAK_BF16_TFLOPS, 2),
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(wall / args.steps * 1e3, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": w.name, "B": w.B, "Hq": w.Hq, "Hkv": w.Hkv, "Sq": w.Sq, "Sk": w.Sk,
                   "d_qk": w.dqk, "d_v": w.dv, "causal": w.causal, "scale": w.scale, "seed": w.seed,
                   "split": n_split or None, "path": "decode" if args.decode else ("split" if n_split else "fused"),
                   "caches": "cold (512 MiB written before each launch)" if args.cold else "warm"},
        "roofline": {**roof,
                     "traffic": traffic,
                     "kernel_ms": {"mean": round(sum(launch_ms) / len(launch_ms), 4),
                                   "median": round(sorted(launch_ms)[len(launch_ms) // 2], 4),
                                   "min": round(min(launch_ms), 4), "max": round(max(launch_ms), 4)},
                     "kernel": kernel_name,
                     "algorithmic_flops_per_launch": flops,
                     "algorithmic_bytes_per_launch": W.algorithmic_bytes(w)},
        "cpu_baseline": cpu,
        "parity": parity,
        "kernel_source": kernel_source_hash(),
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
