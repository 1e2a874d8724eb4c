"""Benchmark of the DiT attention hot path on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload pixart]

One step = one pass of the whole hot path for one layer on the chosen
workload (default: Pixart 1024px, B=2 H=16 d=72, 4096 tokens):
  * the M PipeFusion patch steps in order (each call writes its fresh K/V
    slice into the layer's buffer and attends over the fresh/stale buffer),
  * the sequence-parallel share: chunk attention of the local query shard over
    each K/V chunk (O and LSE), then the LSE merge of the partials.
Inputs are synthetic (seeded N(0,1); stale K/V = fresh + N(0, 0.05^2)) and
resident in HBM before timing starts.  A clock pre-heat (whole steps for
--preheat-s seconds of wall time, 0.3 by default: a GPU that was idle runs
its first tens of milliseconds of work at lower clocks), then W untimed
steps, then K timed steps between synchronisations with events
only at the ends; then K more steps with HIP events around each run of
consecutive launches of one kernel give each kernel's average duration.
Prints ONE JSON line.

`value` is algorithmic attention FLOP/s (4*B*H*Nq*Nk*d per call) over the
whole step.  `roofline` refers to the kernel with the largest share of the
step's time: `achieved` and `frac` are timed with HIP events live in this
run; `traffic` (HBM bytes per launch) and `mfma_busy` come from rocprofv3
counter runs of the same kernel build, whose summaries `traffic_source` and
`counters_source` name, and are null for any other build.  `cpu_baseline`
times the fp64 oracle on a bounded row sample of the same workload on the
host's cores.  With the default pixart workload the line also carries
`flux_16k`: the same measurement of the Flux 2048px sequence-parallel share
(16896 tokens), the 16k-token configuration.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 matrix peak (published)
PEAK_F32_TFLOPS = 157.3     # MI355X fp32 vector peak (published)
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E (published)

# HBM traffic per call of the dominant kernel, in bytes: rocprofv3 --pmc
# FETCH_SIZE and WRITE_SIZE (KiB per dispatch, one counter per run), scaled by
# what the same counters read for kv_update_kernel copying a known size
# (FETCH x about 1.995, WRITE x 1.0).  Each entry holds the fingerprint of the
# kernel build it was taken on (sha256 prefix of the source and its compile
# flags); a different build reports null.
MEASURED_TRAFFIC = {
    ("pixart", "patch_attn"): {"bytes": (49251 + 13875) * 1024, "src": "8ea515cefb0f3f25"},
    ("sd3", "patch_attn"): {"bytes": (59123 + 9216) * 1024, "src": "8ea515cefb0f3f25"},
    # the partitioned sweep and its fix-up, one launch of each per call
    ("flux", "chunk_attn"): {"bytes": (139907 + 41225) * 1024, "src": "8ea515cefb0f3f25"},
    ("flux_ring", "chunk_attn"): {"bytes": (158643 + 41277) * 1024, "src": "8ea515cefb0f3f25"},
    ("cog", "patch_attn"): {"bytes": (259311 + 19744) * 1024, "src": "8ea515cefb0f3f25"},
    ("cog", "chunk_attn"): {"bytes": (133526 + 109990) * 1024, "src": "8ea515cefb0f3f25"},
}


TRAFFIC_FILES = {
    "pixart": "profiles/attn_patch_pixart_hbm_traffic.txt",
    "sd3": "profiles/attn_patch_sd3_hbm_traffic.txt",
    "flux": "profiles/attn_chunk_flux_hbm_traffic.txt",
    "flux_ring": "profiles/attn_chunk_flux_ring_hbm_traffic.txt",
    "cog": "profiles/attn_patch_cog_hbm_traffic.txt",
}


def traffic_of(workload: str, kind: str) -> dict:
    from paper_2411_01738_amd.build import kernel_fingerprint

    e = MEASURED_TRAFFIC.get((workload, kind))
    if e is None or kernel_fingerprint() != e["src"]:
        return {"traffic": None, "traffic_source": None}
    return {"traffic": e["bytes"], "traffic_source": TRAFFIC_FILES[workload]}


# Matrix-core counters of the dominant kernel from a rocprofv3 --pmc run of
# the same workload (SQ_VALU_MFMA_BUSY_CYCLES / (4 SIMDs x SQ_BUSY_CU_CYCLES):
# the fraction of the kernel's CU-busy time the matrix pipes worked), with the
# summary file and the kernel build's fingerprint; a different build reports
# nothing.
MEASURED_COUNTERS = {
    ("pixart", "patch_attn"): {"mfma_busy": 0.378, "file": "profiles/attn_patch_pixart_mfma_counters.txt",
                               "src": "8ea515cefb0f3f25"},
    ("sd3", "patch_attn"): {"mfma_busy": 0.353, "file": "profiles/attn_patch_sd3_mfma_counters.txt",
                            "src": "8ea515cefb0f3f25"},
    ("flux", "chunk_attn"): {"mfma_busy": 0.531, "file": "profiles/attn_chunk_flux_mfma_counters.txt",
                             "src": "8ea515cefb0f3f25"},
    ("cog", "patch_attn"): {"mfma_busy": 0.406, "file": "profiles/attn_patch_cog_mfma_counters.txt",
                            "src": "8ea515cefb0f3f25"},
    ("cog", "chunk_attn"): {"mfma_busy": 0.457, "file": "profiles/attn_patch_cog_mfma_counters.txt",
                            "src": "8ea515cefb0f3f25"},
}


def counters_of(workload: str, kind: str) -> dict:
    from paper_2411_01738_amd.build import kernel_fingerprint

    e = MEASURED_COUNTERS.get((workload, kind))
    if e is None or kernel_fingerprint() != e["src"]:
        return {"mfma_busy": None, "counters_source": None}
    return {"mfma_busy": e["mfma_busy"], "counters_source": e["file"]}


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=200)
    ap.add_argument("--preheat-s", type=float, default=0.3,
                    help="seconds of untimed whole steps before the warm-up steps (clock ramp)")
    ap.add_argument("--workload", default="pixart",
                    choices=["tiny", "pixart", "sd3", "flux", "cog", "sd3_ic", "sd3_ic_bal", "pixart_hybrid",
                             "pixart_stage",
                             "flux_ring"])
    ap.add_argument("--no-split", action="store_true",
                    help="never split a query tile's keys over several workgroups")
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="target CPU time of the oracle baseline sample (0 = skip)")
    ap.add_argument("--no-flux", action="store_true",
                    help="with the pixart workload, skip the Flux 16k-token SP share beside it")
    return ap.parse_args()


def cpu_baseline(w, t, target_s: float, one_thread: bool = True):
    """fp64 oracle on a bounded sample of the workload: whole calls of the step
    in order (patch steps, else chunk steps) until about target_s / 3 seconds
    have been spent; when one call alone would take far longer, an evenly
    spaced subset of its query rows.  Scaled to TFLOP/s of algorithmic work;
    the median of 3 such samples is reported.  With one_thread, the same is
    then run on one thread for a quarter of the time."""
    import numpy as np

    import oracle

    orc = oracle.get()
    jobs = []  # (description, nq_total, nk, run(rows), flops(rows))
    attn = lambda nq, nk: w.attn_flops(nq, nk)
    if w.hidden:
        kv = np.ascontiguousarray(np.stack([t.k_stale, t.v_stale]))
        ws = [t.extra[n] for n in ("wq", "wk", "wv", "wo")]
        C, HD = w.hidden, w.H * w.d
        for p, (off, ln) in enumerate(w.patches()):
            x = t.extra["x"][:, off:off + ln].copy()
            jobs.append((f"stage micro-step {p}", ln, w.N,
                         lambda rows, x=x, off=off: orc.stage_step(x, *ws, kv, off, rows=rows),
                         lambda n, ln=ln: attn(n, w.N) + 2.0 * w.B * C * HD * (3 * ln + n)))
    elif w.patches():
        kv = np.ascontiguousarray(np.stack([t.k_stale, t.v_stale]))
        for p, (ranges, qrows) in enumerate(w.patch_calls()):
            frows = np.concatenate([np.arange(o, o + n) for o, n in ranges])
            q = t.q[:, qrows].copy()
            fk = t.k_fresh[:, frows].copy()
            fv = t.v_fresh[:, frows].copy()
            jobs.append((f"patch step {p}", len(qrows), w.N,
                         lambda rows, q=q, ranges=ranges, fk=fk, fv=fv:
                         orc.patch_ranges(q, kv, ranges, fk, fv, rows=rows),
                         lambda n: attn(n, w.N)))
    else:
        q0, q1 = w.sp_q
        q = t.q[:, q0:q1].copy()
        for r, (s, e) in enumerate(w.sp_chunks):
            k = t.k_fresh[:, s:e].copy()
            v = t.v_fresh[:, s:e].copy()
            jobs.append((f"chunk {r}", q1 - q0, e - s,
                         lambda rows, k=k, v=v: orc.attention(q, k, v, rows=rows),
                         lambda n, nk=e - s: attn(n, nk)))

    def sample(budget_s):
        # calibrate the cost of one (query row x key) on a few rows of the
        # first call; the first probe also starts the oracle's thread pool
        desc0, nq0, nk0, run0, _ = jobs[0]
        probe = np.linspace(0, nq0 - 1, min(64, nq0)).astype(np.int64)
        run0(probe)
        t0 = time.perf_counter()
        run0(probe)
        per_unit = (time.perf_counter() - t0) / (len(probe) * nk0)
        # whole calls in step order, the step repeated if it is short, the
        # last call cut to an evenly spaced subset of its rows to stay near
        # the budget
        flops, spent, parts = 0.0, 0.0, []
        for rep in range(1000):
            for desc, nq, nk, run, flops_of in jobs:
                left = budget_s - spent
                if left <= 0.05 * budget_s:
                    break
                n = min(nq, max(1, int(left / (per_unit * nk))))
                rows = (np.arange(nq, dtype=np.int64) if n >= nq
                        else np.linspace(0, nq - 1, n).astype(np.int64))
                t0 = time.perf_counter()
                run(rows)
                dt = time.perf_counter() - t0
                spent += dt
                per_unit = dt / (len(rows) * nk)
                flops += flops_of(len(rows))
                parts.append(f"{desc} ({len(rows)}/{nq} rows)")
            else:
                continue
            break
        return flops, spent, parts

    runs = [sample(target_s / 3) for _ in range(3)]
    rates = [f / sp / 1e12 for f, sp, _ in runs]
    med = sorted(range(3), key=lambda i: rates[i])[1]
    flops, spent, parts = runs[med]
    threads = orc.num_threads()
    if len(parts) > 6:
        parts = parts[:3] + [f"... {len(parts) - 6} more calls ..."] + parts[-3:]
    out = {
        "value": rates[med],
        "unit": "TFLOP/s",
        "cores": threads,
        "kind": "oracle",
        "sample": "median of 3 samples, each: " + "; ".join(parts) +
                  f"; all {w.B * w.H} (batch, head) pairs, fp64, {spent:.1f} s",
        "samples_tflops": [round(r, 5) for r in rates],
        "cpu": cpu_model(),
    }
    if one_thread:
        orc.set_num_threads(1)
        try:
            flops1, spent1, _ = sample(target_s / 4)
        finally:
            orc.set_num_threads(threads)
        out["one_thread_value"] = flops1 / spent1 / 1e12
        out["one_thread_sample_s"] = round(spent1, 1)
    return out


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    import platform
    return platform.processor() or "unknown"


def measure(w, t, steps: int, warmup: int, split: bool, extra_timings: bool = True, preheat_s: float = 0.0):
    """Time one workload on the GPU: whole steps for `preheat_s` seconds and
    `warmup` more, all untimed, then exactly
    `steps` timed steps between synchronisations (events only at the two
    ends), then `steps` more with HIP events around each run of consecutive
    launches of one kernel.  Returns the step figures, per-kernel figures and
    the roofline of the kernel with the largest share of the step."""
    import torch

    from paper_2411_01738_amd import _lib
    from paper_2411_01738_amd.hotpath import HotPath

    hp = HotPath(w, t, split=split)
    stream = torch.cuda.current_stream()

    # each entry: (kind, callable, flops, bytes)
    calls = []
    patch_kind = "stage_step" if hp.stage is not None else "patch_attn"
    for p in range(len(hp.patch_q)):
        calls.append((patch_kind, lambda p=p: hp.patch_step(p), hp.patch_flops(p), 0.0))
    if hp.sp_q is not None:
        for r in range(len(hp.chunk_k)):
            calls.append(("chunk_attn", lambda r=r: hp.chunk_step(r), hp.chunk_flops(r), 0.0))
        if not w.sp_ring:
            calls.append(("lse_merge", hp.merge, 0.0, hp.merge_bytes()))

    # clock pre-heat: the GPU leaves its idle clocks during the first tens of
    # milliseconds of sustained work; untimed, before the warm-up steps
    t_end = time.perf_counter() + preheat_s
    while time.perf_counter() < t_end:
        for _ in range(10):
            hp.step()
        torch.cuda.synchronize()
    for _ in range(warmup):
        hp.step()
    torch.cuda.synchronize()

    # timed region: exactly K steps, events only at its two ends
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record(stream)
    for _ in range(steps):
        for _, fn, _, _ in calls:
            fn()
    end.record(stream)
    torch.cuda.synchronize()
    ms_per_step = start.elapsed_time(end) / steps

    # per-kernel durations: K more steps with HIP events on the launch stream
    # around each run of consecutive launches of one kernel (the M patch
    # steps, the chunk steps, the merge); an event pair costs the stream a few
    # microseconds, so it is kept out of the timed region above
    groups = []  # (kind, first call, end call)
    for i, (kind, _, _, _) in enumerate(calls):
        if groups and groups[-1][0] == kind:
            groups[-1][2] = i + 1
        else:
            groups.append([kind, i, i + 1])
    ev = [[(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in groups] for _ in range(steps)]
    torch.cuda.synchronize()
    for s_ in range(steps):
        for g, (_, a, b) in enumerate(groups):
            ev[s_][g][0].record(stream)
            for _, fn, _, _ in calls[a:b]:
                fn()
            ev[s_][g][1].record(stream)
    torch.cuda.synchronize()

    kinds = {}
    for g, (kind, a, b) in enumerate(groups):
        d = kinds.setdefault(kind, {"launches": 0, "ms": 0.0, "flops": 0.0, "bytes": 0.0, "per_step": []})
        for s_ in range(steps):
            ms = ev[s_][g][0].elapsed_time(ev[s_][g][1])
            d["ms"] += ms
            d["per_step"].append(ms * 1e3 / (b - a))
        d["launches"] += (b - a) * steps
        for _, _, flops, nbytes in calls[a:b]:
            d["flops"] += flops * steps
            d["bytes"] += nbytes * steps
    peak = PEAK_BF16_TFLOPS if w.dtype == "bf16" else PEAK_F32_TFLOPS
    kern = {}
    for kind, d in kinds.items():
        avg_us = d["ms"] * 1e3 / d["launches"]
        ps = sorted(d["per_step"])
        e = {"launches_per_step": d["launches"] // steps, "avg_us": round(avg_us, 3),
             "median_us": round(ps[len(ps) // 2], 3), "min_us": round(ps[0], 3)}
        if d["flops"]:
            tf = d["flops"] / (d["ms"] / 1e3) / 1e12
            e.update(tflops=round(tf, 2), frac_peak=round(tf / peak, 4))
        if d["bytes"]:
            gbs = d["bytes"] / (d["ms"] / 1e3) / 1e9
            e.update(gbs=round(gbs, 1), frac_hbm=round(gbs / PEAK_HBM_GBS, 4))
        kern[kind] = e

    # stand-alone K/V-slice update (the patch kernel does it fused): its GB/s.
    # Warm: back-to-back launches through the C ABI with the arguments
    # marshalled once (a launch takes less time than the binding's checks).
    # Cold: each launch after a 1 GiB write that evicts L2 and the MALL,
    # bracketed by its own events (which add about a microsecond).
    if extra_timings and w.patches():
        off, ln = w.patches()[0]
        L = _lib.lib()
        L.xdit_set_stream(stream.cuda_stream)
        upd = (hp.kv_buf.data_ptr(), off, ln, hp.patch_k[0].data_ptr(), hp.patch_v[0].data_ptr(),
               w.B, w.N, w.H, w.d, _lib.XDIT_BF16 if w.dtype == "bf16" else _lib.XDIT_F32)
        _lib.check(L.xdit_kv_update(*upd))
        reps = 200
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        a.record(stream)
        rcs = [L.xdit_kv_update(*upd) for _ in range(reps)]
        b.record(stream)
        torch.cuda.synchronize()
        for rc in rcs:
            _lib.check(rc)
        warm_us = a.elapsed_time(b) * 1e3 / reps
        flush = torch.empty(1 << 28, dtype=torch.float32, device="cuda")
        cold = []
        for _ in range(20):
            flush.fill_(1.0)
            a.record(stream)
            _lib.check(L.xdit_kv_update(*upd))
            b.record(stream)
            torch.cuda.synchronize()
            cold.append(a.elapsed_time(b) * 1e3)
        del flush
        cold_us = sorted(cold)[len(cold) // 2]
        nb = hp.update_bytes(0)
        kern["kv_update"] = {"avg_us": round(warm_us, 3), "gbs": round(nb / warm_us / 1e3, 1),
                             "frac_hbm": round(nb / warm_us / 1e3 / PEAK_HBM_GBS, 4),
                             "cold_median_us": round(cold_us, 3),
                             "cold_gbs": round(nb / cold_us / 1e3, 1),
                             "note": "outside the step: warm back-to-back, and cold after"
                                     " evicting L2/MALL"}

    # the merge is one launch per step, so its in-step events include their
    # own overhead; back-to-back launches through the C ABI give its duration
    if extra_timings and hp.sp_q is not None and not w.sp_ring:
        import ctypes

        L = _lib.lib()
        L.xdit_set_stream(stream.cuda_stream)
        n = len(hp.chunk_out)
        optrs = (ctypes.c_void_p * n)(*[o.data_ptr() for o in hp.chunk_out])
        lptrs = (ctypes.c_void_p * n)(*[x.data_ptr() for x in hp.chunk_lse])
        nq = w.sp_q[1] - w.sp_q[0]
        mrg = (optrs, lptrs, n, hp.sp_out.data_ptr(), hp.sp_lse.data_ptr(), w.B, nq, w.H, w.d,
               _lib.XDIT_BF16 if w.dtype == "bf16" else _lib.XDIT_F32)
        reps = 50
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        a.record(stream)
        rcs = [L.xdit_lse_merge(*mrg) for _ in range(reps)]
        b.record(stream)
        torch.cuda.synchronize()
        for rc in rcs:
            _lib.check(rc)
        us = a.elapsed_time(b) * 1e3 / reps
        # cold: each launch after a 1 GiB write that evicts L2 and the MALL
        flush = torch.empty(1 << 28, dtype=torch.float32, device="cuda")
        cold = []
        for _ in range(20):
            flush.fill_(1.0)
            a.record(stream)
            _lib.check(L.xdit_lse_merge(*mrg))
            b.record(stream)
            torch.cuda.synchronize()
            cold.append(a.elapsed_time(b) * 1e3)
        del flush
        cold_us = sorted(cold)[len(cold) // 2]
        kern["lse_merge"].update(back_to_back_us=round(us, 3),
                                 back_to_back_gbs=round(hp.merge_bytes() / us / 1e3, 1),
                                 cold_median_us=round(cold_us, 3),
                                 cold_gbs=round(hp.merge_bytes() / cold_us / 1e3, 1))

    step_flops = hp.step_flops()
    value = step_flops / (ms_per_step / 1e3) / 1e12

    dom = max(kinds, key=lambda k: kinds[k]["ms"])
    dd = kinds[dom]
    avg_s = dd["ms"] / 1e3 / dd["launches"]
    timing = ("HIP events on the launch stream around each run of launches of this kernel,"
              " over the K steps after the timed region; achieved = algorithmic work per launch"
              " / average launch duration")
    if dd["flops"]:
        per_launch = dd["flops"] / dd["launches"]
        achieved = per_launch / avg_s / 1e12
        # bf16 attention runs on the matrix cores; the f32 path is plain VALU code
        roof = {"kernel": dom, "bound": "mfma" if w.dtype == "bf16" else "alu",
                "achieved": round(achieved, 2), "peak": peak,
                "unit": "TFLOP/s", "frac": round(achieved / peak, 4)}
    else:
        per_launch = dd["bytes"] / dd["launches"]
        achieved = per_launch / avg_s / 1e9
        roof = {"kernel": dom, "bound": "hbm", "achieved": round(achieved, 1),
                "peak": PEAK_HBM_GBS, "unit": "GB/s", "frac": round(achieved / PEAK_HBM_GBS, 4)}
    roof.update(traffic_of(w.name, dom))
    roof["timing"] = timing
    roof.update(counters_of(w.name, dom))
    hp = None
    torch.cuda.empty_cache()
    return {"ms_per_step": ms_per_step, "value": value, "step_flops": step_flops, "kernels": kern,
            "roofline": roof}


DESC = {"tiny": "tiny fp32: B=1 H=2 d=64, 256 tokens, M=4 patch steps + 4-chunk SP share",
        "pixart": "pixart-1024px: B=2 H=16 d=72, 4096 tokens, M=4 patch steps"
                  " + 4-chunk SP share (Q 1024 rows)",
        "sd3": "sd3-1024px joint attention: B=2 H=24 d=64, 4096 image + 333 text tokens,"
               " M=8 patch steps",
        "flux": "flux-2048px SP share: B=1 H=24 d=128, Q 4224 rows x 4 chunks of 4224 + merge",
        "cog": "cogvideox video: B=1 H=48 d=64, 17550 video + 226 text tokens, M=16 patch"
               " steps + 8-chunk split (Q all rows) + merge",
        "sd3_ic": "sd3-1024px in-context: B=2 H=24 d=64, 4096 image + 333 text tokens,"
                  " M=8 patch steps, patch 0 carries the text (845 fresh rows and queries)",
        "sd3_ic_bal": "sd3-1024px in-context, balanced partition: B=2 H=24 d=64, 4096 image"
                      " + 333 text tokens, M=8 patch steps of 553-554 fresh rows (patch 0:"
                      " 220 image + 333 text)",
        "flux_ring": "flux-2048px SP share, ring form: B=1 H=24 d=128, Q 4224 rows, 4 chunks"
                     " of 4224 each merged into the running output as it arrives",
        "pixart_stage": "pixart-1024px stage micro-steps: B=2 H=16 d=72 hidden 1152, 4096"
                        " tokens, M=4 x (QKV projections, patch step, output projection);"
                        " value counts projection and attention FLOPs",
        "pixart_hybrid": "pixart-1024px PipeFusion x 2-way SP share: B=2 H=16 d=72,"
                         " 4096 tokens, M=4 patch steps of 1024 gathered fresh rows,"
                         " 512 local queries each"}


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only; --gpus {args.gpus} is not supported "
              "(this build has no multi-GPU path)", file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2411_01738_amd import _lib
    from paper_2411_01738_amd.inputs import WORKLOADS, generate

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    _lib.lib()  # fails loudly if the HIP library is missing
    torch.cuda.set_device(0)
    w = WORKLOADS[args.workload]
    t = generate(w)
    m = measure(w, t, args.steps, args.warmup, not args.no_split, preheat_s=args.preheat_s)

    # the 16k-token target configuration (Flux SP share) beside the headline
    # one, under the same clock: same K and W, its own per-kernel figures,
    # roofline and oracle sample
    flux = None
    if args.workload == "pixart" and not args.no_flux:
        wf = WORKLOADS["flux"]
        tf = generate(wf)
        mf = measure(wf, tf, args.steps, args.warmup, not args.no_split, extra_timings=True,
                     preheat_s=args.preheat_s)
        flux = {"workload": DESC["flux"], "value": round(mf["value"], 2), "unit": "TFLOP/s",
                "ms_per_step": round(mf["ms_per_step"], 4), "flops_per_step": mf["step_flops"],
                "kernels": mf["kernels"], "roofline": mf["roofline"]}
        if args.cpu_seconds > 0:
            flux["cpu_baseline"] = cpu_baseline(wf, tf, args.cpu_seconds * 0.6, one_thread=False)
        del tf

    cpu = None
    if args.cpu_seconds > 0:
        cpu = cpu_baseline(w, t, args.cpu_seconds)

    line = {
        "metric": "attention TFLOP/s (bf16) per patch/chunk step; merge GB/s",
        "value": round(m["value"], 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "preheat_s": args.preheat_s,
        "ms_per_step": round(m["ms_per_step"], 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic",
        "config": {"workload": DESC[w.name], "B": w.B, "H": w.H, "d": w.d, "tokens": w.N,
                   "patches": len(w.patches()), "sp_chunks": len(w.sp_chunks),
                   "flops_per_step": m["step_flops"]},
        "kernels": m["kernels"],
        "roofline": m["roofline"],
        "cpu_baseline": cpu,
    }
    if flux is not None:
        line["flux_16k"] = flux
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
