"""Benchmark of the DiT attention hot path on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload pixart]

One step = one pass of the whole hot path for one layer on the chosen
workload (default: Pixart 1024px, B=2 H=16 d=72, 4096 tokens):
  * the M PipeFusion patch steps in order (each call writes its fresh K/V
    slice into the layer's buffer and attends over the fresh/stale buffer),
  * the sequence-parallel share: chunk attention of the local query shard over
    each K/V chunk (O and LSE), then the LSE merge of the partials.
Inputs are synthetic (seeded N(0,1); stale K/V = fresh + N(0, 0.05^2)) and
resident in HBM before timing starts.  W untimed steps (the default lets the
GPU clocks settle), then K timed steps between synchronisations with events
only at the ends; then K more steps with HIP events around each run of
consecutive launches of one kernel give each kernel's average duration.
Prints ONE JSON line.

`value` is algorithmic attention FLOP/s (4*B*H*Nq*Nk*d per call) over the
whole step.  `roofline` refers to the kernel with the largest share of the
step's time.  `cpu_baseline` times the fp64 oracle on a bounded row sample of
the same workload on the host's cores.
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
    ("pixart", "patch_attn"): {"bytes": (49151 + 13875) * 1024, "src": "0ae64fdbe1062094"},
    ("sd3", "patch_attn"): {"bytes": (58953 + 9216) * 1024, "src": "0ae64fdbe1062094"},
    # the partitioned sweep and its fix-up, one launch of each per call
    ("flux", "chunk_attn"): {"bytes": (154455 + 41224) * 1024, "src": "0ae64fdbe1062094"},
    ("flux_ring", "chunk_attn"): {"bytes": (135360 + 25763) * 1024, "src": "0ae64fdbe1062094"},
    ("cog", "patch_attn"): {"bytes": (264983 + 19744) * 1024, "src": "0ae64fdbe1062094"},
    ("cog", "chunk_attn"): {"bytes": (133307 + 109989) * 1024, "src": "0ae64fdbe1062094"},
}


def traffic_of(workload: str, kind: str):
    from paper_2411_01738_amd.build import kernel_fingerprint

    e = MEASURED_TRAFFIC.get((workload, kind))
    if e is None:
        return None
    return e["bytes"] if kernel_fingerprint() == e["src"] else None


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=200)
    ap.add_argument("--workload", default="pixart",
                    choices=["tiny", "pixart", "sd3", "flux", "cog", "sd3_ic", "sd3_ic_bal", "pixart_hybrid",
                             "pixart_stage",
                             "flux_ring"])
    ap.add_argument("--no-split", action="store_true",
                    help="never split a query tile's keys over several workgroups")
    ap.add_argument("--cpu-seconds", type=float, default=15.0,
                    help="target CPU time of the oracle baseline sample (0 = skip)")
    return ap.parse_args()


def cpu_baseline(w, t, target_s: float):
    """fp64 oracle on a bounded sample of the workload: whole calls of the step
    in order (patch steps, else chunk steps) until about target_s seconds have
    been spent; when one call alone would take far longer, an evenly spaced
    subset of its query rows.  Scaled to TFLOP/s of algorithmic work.  The
    same is then run on one thread for a third of the time."""
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

    flops, spent, parts = sample(target_s)
    threads = orc.num_threads()
    orc.set_num_threads(1)
    try:
        flops1, spent1, _ = sample(target_s / 3)
    finally:
        orc.set_num_threads(threads)
    if len(parts) > 6:
        parts = parts[:3] + [f"... {len(parts) - 6} more calls ..."] + parts[-3:]
    return {
        "value": flops / spent / 1e12,
        "unit": "TFLOP/s",
        "cores": threads,
        "kind": "oracle",
        "sample": "; ".join(parts) + f"; all {w.B * w.H} (batch, head) pairs, fp64,"
                  f" {spent:.1f} s",
        "one_thread_value": flops1 / spent1 / 1e12,
        "one_thread_sample_s": round(spent1, 1),
    }


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only; --gpus {args.gpus} is not supported "
              "(this build has no multi-GPU path)", file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2411_01738_amd import _lib
    from paper_2411_01738_amd.hotpath import HotPath
    from paper_2411_01738_amd.inputs import WORKLOADS, generate

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    _lib.lib()  # fails loudly if the HIP library is missing
    torch.cuda.set_device(0)
    w = WORKLOADS[args.workload]
    t = generate(w)
    hp = HotPath(w, t, split=not args.no_split)
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

    for _ in range(args.warmup):
        hp.step()
    torch.cuda.synchronize()

    # timed region: exactly K steps, events only at its two ends
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record(stream)
    for _ in range(args.steps):
        for _, fn, _, _ in calls:
            fn()
    end.record(stream)
    torch.cuda.synchronize()
    ms_per_step = start.elapsed_time(end) / args.steps

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
           for _ in groups] for _ in range(args.steps)]
    torch.cuda.synchronize()
    for s in range(args.steps):
        for g, (_, a, b) in enumerate(groups):
            ev[s][g][0].record(stream)
            for _, fn, _, _ in calls[a:b]:
                fn()
            ev[s][g][1].record(stream)
    torch.cuda.synchronize()

    kinds = {}
    for g, (kind, a, b) in enumerate(groups):
        d = kinds.setdefault(kind, {"launches": 0, "ms": 0.0, "flops": 0.0, "bytes": 0.0, "per_step": []})
        for s in range(args.steps):
            ms = ev[s][g][0].elapsed_time(ev[s][g][1])
            d["ms"] += ms
            d["per_step"].append(ms * 1e3 / (b - a))
        d["launches"] += (b - a) * args.steps
        for _, _, flops, nbytes in calls[a:b]:
            d["flops"] += flops * args.steps
            d["bytes"] += nbytes * args.steps
    peak = PEAK_BF16_TFLOPS if w.dtype == "bf16" else PEAK_F32_TFLOPS
    kern = {}
    for kind, d in kinds.items():
        avg_us = d["ms"] * 1e3 / d["launches"]
        ps = sorted(d["per_step"])
        e = {"launches_per_step": d["launches"] // args.steps, "avg_us": round(avg_us, 3),
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
    if w.patches():
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
    if hp.sp_q is not None and not w.sp_ring:
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
    roof["traffic"] = traffic_of(w.name, dom)

    cpu = None
    if args.cpu_seconds > 0:
        cpu = cpu_baseline(w, t, args.cpu_seconds)

    desc = {"tiny": "tiny fp32: B=1 H=2 d=64, 256 tokens, M=4 patch steps + 4-chunk SP share",
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
                             " 512 local queries each"}[w.name]
    line = {
        "metric": "attention TFLOP/s (bf16) per patch/chunk step; merge GB/s",
        "value": round(value, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic",
        "config": {"workload": desc, "B": w.B, "H": w.H, "d": w.d, "tokens": w.N,
                   "patches": len(w.patches()), "sp_chunks": len(w.sp_chunks),
                   "flops_per_step": step_flops},
        "kernels": kern,
        "roofline": roof,
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
