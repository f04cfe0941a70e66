"""Measured ceilings of the GPU for the fused attention forward's roofline (measurement only).

Runs the microbenchmarks of ``libfa_ceilings.so`` (``csrc/fa_ceilings.hip``) and prints one JSON
line: the bf16 MFMA rate with nothing else to do at one and two waves per SIMD, and the shader clock
the chip sustains meanwhile; the cycles an MFMA slot takes with the online softmax's VALU work
(exponentials, fmas) issued next to it (together the counterpart of the paper's instruction-count
compute ceiling, Sec. 5.2); HBM streaming reads through VGPRs and through direct-to-LDS buffer loads, 2 GiB each, far past
the 256 MB Infinity Cache (the per-level bandwidth ceilings of Sec. 5.2 / Table 2); and the LDS read
rate of the two read forms the fused kernel uses, in bytes per clock per CU.

Each kernel is timed with HIP events on the launch stream; the clock comes from the shader-clock and
real-time counters every wave stamps at its start and end (the real-time counter's rate is calibrated
against the events of the same launch). Every measurement runs ``repeats`` times back to back after a
warm-up and the fastest is reported, next to the nominal figure (the MFMA loop also reports the
last of 20 launches, when the clock has settled under sustained load).
"""

from __future__ import annotations

import ctypes
import json
import os
import sys

from . import build as _build

PEAK_BF16_TFLOPS = 2516.6  # 256 CUs x 4096 dense bf16 FLOP/clk/CU x 2.4 GHz
PEAK_HBM_GBS = 8000.0
NOMINAL_CLOCK_GHZ = 2.4
MFMA_FLOP = 2 * 32 * 32 * 16  # one v_mfma_f32_32x32x16_bf16
# (v_exp_f32, v_fma_f32) per MFMA slot of fa_ceil_mix (FA_CEIL_MIXES in fa_ceilings.hip)
MIXES = [(0, 0), (0, 2), (0, 4), (0, 6), (0, 8), (1, 0), (2, 0), (1, 2), (1, 3), (1, 4), (2, 2), (2, 4)]

_lib = None


def load() -> ctypes.CDLL:
    global _lib
    if _lib is not None:
        return _lib
    import torch  # noqa: F401  (maps torch's HIP runtime first)

    if not os.path.exists(_build.CEIL_LIB_PATH):
        raise ImportError(f"{_build.CEIL_LIB_PATH} is not built; run `python -m paper_2609_21264_amd.build`")
    lib = ctypes.CDLL(_build.CEIL_LIB_PATH)
    vp, i, sz = ctypes.c_void_p, ctypes.c_int, ctypes.c_size_t
    lib.fa_ceil_mfma.argtypes = [vp, vp, vp, i, i, i, vp]
    lib.fa_ceil_mix.argtypes = [vp, vp, vp, i, i, i, i, i, vp]
    lib.fa_ceil_read_vgpr.argtypes = [vp, sz, vp, vp, i, vp]
    lib.fa_ceil_read_lds.argtypes = [vp, sz, vp, i, vp]
    lib.fa_ceil_lds.argtypes = [vp, vp, i, i, i, vp]
    for f in (lib.fa_ceil_mfma, lib.fa_ceil_mix, lib.fa_ceil_read_vgpr, lib.fa_ceil_read_lds, lib.fa_ceil_lds):
        f.restype = i
    _lib = lib
    return lib


def _timed(launch, stamps, repeats: int):
    """Run ``launch`` once to warm up, then ``repeats`` times back to back with events; return, per
    timed run, (ms, shader clock GHz, real-time counter Hz), the clock from that run's stamps."""
    import torch

    stream = torch.cuda.current_stream()
    runs = []
    launch()
    torch.cuda.synchronize()
    for _ in range(repeats):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        st = launch()
        b.record(stream)
        torch.cuda.synchronize()
        if st != 0:
            raise RuntimeError(f"microbenchmark launch failed: hipError {st}")
        ms = a.elapsed_time(b)
        s = stamps.view(-1, 4).to(torch.float64).cpu()
        clk = s[:, 1] - s[:, 0]
        real = s[:, 3] - s[:, 2]
        span_real = float(s[:, 3].max() - s[:, 2].min())
        real_hz = span_real / (ms * 1e-3) if ms > 0 else float("nan")
        ghz = float((clk / real).median()) * real_hz / 1e9
        runs.append((ms, ghz, real_hz))
    return runs


def _best(runs):
    return min(runs, key=lambda r: r[0])


def main(repeats: int = 5) -> dict:
    import torch

    lib = load()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    props = torch.cuda.get_device_properties(dev)
    n_cu = props.multi_processor_count
    handle = torch.cuda.current_stream(dev).cuda_stream
    res = {"metric": "measured ceilings of one MI355X (microbenchmarks)", "device": props.name, "cus": n_cu}

    # bf16 MFMA rate, one workgroup per CU (96 KiB of LDS each), operands drawn N(0, 1) like the
    # attention inputs (the power draw, and so the clock, depends on the operand bits).
    g = torch.Generator(device="cpu").manual_seed(7)
    ops = torch.randn(1024, generator=g).to(torch.bfloat16).to(dev)
    for wpe in (1, 2):
        iters = 32768 // wpe  # ~8 ms per launch; 20 launches back to back reach the sustained clock
        waves = n_cu * 4 * wpe
        out = torch.empty(n_cu * 256 * wpe, dtype=torch.float32, device=dev)
        stamps = torch.zeros(waves * 4, dtype=torch.int64, device=dev)
        runs = _timed(lambda: lib.fa_ceil_mfma(ops.data_ptr(), out.data_ptr(), stamps.data_ptr(), wpe, n_cu, iters,
                                               handle), stamps, 20)
        flop = waves * iters * 16 * MFMA_FLOP
        ms, ghz, real_hz = _best(runs)
        last_ms, last_ghz, _ = runs[-1]
        tflops = flop / (ms * 1e-3) / 1e12
        last = flop / (last_ms * 1e-3) / 1e12
        res[f"mfma_bf16_{wpe}wave_per_simd"] = {
            "tflops": round(tflops, 1), "frac_of_nominal_peak": round(tflops / PEAK_BF16_TFLOPS, 4),
            "shader_clock_ghz": round(ghz, 3), "peak_at_that_clock_tflops": round(n_cu * 4096 * ghz / 1e3, 1),
            "last_of_20_tflops": round(last, 1), "last_of_20_clock_ghz": round(last_ghz, 3),
            "ms": round(ms, 3), "realtime_counter_mhz": round(real_hz / 1e6, 2)}
        print(f"[ceilings] mfma {wpe} wave/SIMD: best {tflops:.1f} TFLOP/s at {ghz:.3f} GHz, last {last:.1f} at "
              f"{last_ghz:.3f} GHz", file=sys.stderr, flush=True)

    # Issue cost of VALU work next to the MFMAs: shader cycles per slot (one MFMA plus n_exp
    # v_exp_f32 and n_fma v_fma_f32) per SIMD, at one and two waves per SIMD. An MFMA alone is 32
    # cycles of matrix-core work; a slot longer than that is bound by instruction issue.
    mix = {}
    for wpe in (1, 2):
        out = torch.empty(n_cu * 256 * wpe, dtype=torch.float32, device=dev)
        stamps = torch.zeros(n_cu * 4 * wpe * 4, dtype=torch.int64, device=dev)
        for ne, nf in MIXES:
            iters = 4096
            runs = _timed(lambda: lib.fa_ceil_mix(ops.data_ptr(), out.data_ptr(), stamps.data_ptr(), wpe, ne, nf, n_cu,
                                                  iters, handle), stamps, 3)
            # per workgroup (one CU, wpe waves per SIMD): first start to last end of its waves, over
            # the slots one SIMD runs (the waves of a SIMD do not share it evenly: one runs ahead)
            s_ = stamps.view(n_cu, 4 * wpe, 4).to(torch.float64).cpu()
            span = s_[:, :, 1].max(dim=1).values - s_[:, :, 0].min(dim=1).values
            cyc = float(span.median()) / (iters * 4 * wpe)
            mix[f"{wpe}wave_{ne}exp_{nf}fma"] = round(cyc, 2)
        print(f"[ceilings] mix {wpe} wave/SIMD: " + ", ".join(f"{k.split('_', 1)[1]} {v}" for k, v in mix.items()
                                                              if k.startswith(f"{wpe}wave")),
              file=sys.stderr, flush=True)
    res["mfma_valu_mix_cycles_per_slot_per_simd"] = mix

    # HBM streaming reads, 2 GiB (past the Infinity Cache).
    nbytes = 2 << 30
    src = torch.empty(nbytes, dtype=torch.uint8, device=dev)
    src.fill_(0x5a)
    sink = torch.zeros(16, dtype=torch.uint8, device=dev)
    n_wg = n_cu * 8
    stamps = torch.zeros(n_wg * 4 * 4, dtype=torch.int64, device=dev)
    ms, ghz, _ = _best(_timed(lambda: lib.fa_ceil_read_vgpr(src.data_ptr(), nbytes, sink.data_ptr(), stamps.data_ptr(),
                                                            n_wg, handle), stamps, repeats))
    gbs = nbytes / (ms * 1e-3) / 1e9
    res["hbm_read_vgpr"] = {"gbs": round(gbs, 1), "frac_of_nominal_peak": round(gbs / PEAK_HBM_GBS, 4),
                            "bytes": nbytes, "ms": round(ms, 3), "workgroups": n_wg}
    print(f"[ceilings] HBM read via VGPR: {gbs:.1f} GB/s", file=sys.stderr, flush=True)
    n_wg = n_cu * 2
    stamps = torch.zeros(n_wg * 4 * 4, dtype=torch.int64, device=dev)
    ms, ghz, _ = _best(_timed(lambda: lib.fa_ceil_read_lds(src.data_ptr(), nbytes, stamps.data_ptr(), n_wg, handle),
                              stamps, repeats))
    gbs = nbytes / (ms * 1e-3) / 1e9
    res["hbm_read_direct_to_lds"] = {"gbs": round(gbs, 1), "frac_of_nominal_peak": round(gbs / PEAK_HBM_GBS, 4),
                                     "bytes": nbytes, "ms": round(ms, 3), "workgroups": n_wg}
    print(f"[ceilings] HBM read direct to LDS: {gbs:.1f} GB/s", file=sys.stderr, flush=True)
    del src

    # LDS read rate (two 64 KiB workgroups per CU), in bytes per clock per CU at the measured clock.
    n_wg = n_cu * 2
    iters = 256
    out = torch.empty(n_wg * 256 * 4, dtype=torch.int32, device=dev)
    stamps = torch.zeros(n_wg * 4 * 4, dtype=torch.int64, device=dev)
    for tr, name, per_pass in ((0, "lds_read_b128", 64 * 1024), (1, "lds_read_b64_tr_b16", 128 * 512)):
        ms, ghz, _ = _best(_timed(lambda: lib.fa_ceil_lds(out.data_ptr(), stamps.data_ptr(), n_wg, iters, tr, handle),
                                  stamps, repeats))
        total = n_wg * 4 * iters * per_pass
        bpc = total / (ms * 1e-3) / (ghz * 1e9) / n_cu
        res[name] = {"bytes_per_clk_per_cu": round(bpc, 1), "tbs": round(total / (ms * 1e-3) / 1e12, 2),
                     "shader_clock_ghz": round(ghz, 3), "ms": round(ms, 3)}
        print(f"[ceilings] {name}: {bpc:.1f} B/clk/CU at {ghz:.3f} GHz", file=sys.stderr, flush=True)
    print(json.dumps(res), flush=True)
    return res


if __name__ == "__main__":
    main()
