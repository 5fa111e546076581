#!/usr/bin/env python3
"""Benchmark of one pipeline stage's hot path on one MI355X.

One step = every row of the hot path once, over one batch of synthetic input
resident in HBM (70B-class slice, four layers):
  per layer: pack + unpack of the boundary activation (forward) and of the
  activation gradient (backward, same mask key), each a batched launch over
  the four boundaries.  Each side evaluates the mask once: the sender packs
  from the key and keeps the kept positions, the receiver unpacks the
  values-only payload from the key and keeps its own; the backward pack and
  unpack read those lists;
  per weight matrix (3 per layer): anchor EMA + top-r SVD + filter
  (sc_build_prior), then the spectral correction of the masked gradient
  (sc_correct) with that prior.
The build's streaming phase (EMA and power passes) runs alone; the masking
runs on a second stream beside the build's Rayleigh-Ritz step and the
correction.  The same steps are also timed strictly one part after another
(components.serial_step) and with the prior built asynchronously
(components.async_step).

Prints one JSON line.  `value` is the algorithmic HBM bytes of the step
divided by the measured step time (GB/s); `roofline` reports the kernel that
took the most time, measured live with HIP events on its own stream (library
event timing); `cpu_baseline` times the CPU oracle on a bounded sample of the
same workload.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import platform
import subprocess
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "mask pack/unpack GB/s + spectral-correction TFLOP/s, % of HBM/MFMA peak"
PEAK_HBM = 8000.0          # GB/s
PEAK_BF16 = 2500.0         # TFLOP/s dense
PEAK_F32 = 157.3           # TFLOP/s (fp32 matrix and vector)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--config", type=int, default=5)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-probe", action="store_true",
                    help="run one plain copy kernel of known size (512 MiB in, 512 MiB out) before the "
                         "warmup, as the reference for scaling HBM byte counters")
    ap.add_argument("--cpu-seconds", type=float, default=20.0,
                    help="approximate budget of the CPU-oracle sample")
    ap.add_argument("--no-adamw", action="store_true",
                    help="skip the separate measurement of the corrected AdamW step")
    ap.add_argument("--no-bernoulli", action="store_true",
                    help="skip the separate measurement of the Bernoulli mask variant")
    ap.add_argument("--no-powersgd", action="store_true",
                    help="skip the separate measurement of the PowerSGD compressor")
    ap.add_argument("--no-async", action="store_true",
                    help="skip the second timed loop in which the anchor-prior build runs on its own "
                         "stream beside the masking and the correction")
    return ap.parse_args()


def touched_line_fraction(H: int, K: int, elem_bytes: int, line: int = 128) -> float:
    """Expected share of 128-byte lines of a row that hold >= 1 kept entry:
    1 - C(H - E, K) / C(H, K) with E elements per line."""
    E = line // elem_bytes
    if K > H - E:
        return 1.0
    lg = math.lgamma
    log_ratio = (lg(H - E + 1) - lg(K + 1) - lg(H - E - K + 1)) - (lg(H + 1) - lg(K + 1) - lg(H - K + 1))
    return 1.0 - math.exp(log_ratio)


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (asked for --gpus {args.gpus}): the library has no "
              "multi-GPU path (no collectives, no sharding), so N must be 1.", file=sys.stderr)
        return 2

    import torch
    import workloads
    import paper_2609_14339_amd as pk

    cfg = workloads.CONFIGS[args.config]
    act, gs = cfg.act, cfg.grad
    dev = torch.device("cuda")
    torch.cuda.set_device(0)
    stream = torch.cuda.current_stream()
    esz = 2 if act.dtype == torch.bfloat16 else 4
    gsz = 2 if gs.dtype == torch.bfloat16 else 4
    L = gs.layers
    keep = act.keep[0]
    H, rows = act.H, act.B * act.S
    K = pk.ac_keep_count(H, keep)
    scale = H / K
    r = gs.r[0]
    p, q = cfg.oversample, cfg.power_iters
    t0 = time.time()

    # ---------------- inputs, resident in HBM ----------------
    # the L boundaries' activations (and gradients) stacked [L, rows, H];
    # boundary l is keyed with layer l
    x_all = torch.empty(L, rows, H, dtype=act.dtype, device=dev)
    gx_all = torch.empty_like(x_all)
    keys = []
    for l in range(L):
        x_all[l] = workloads.activation(act, cfg.cid, l, 0, dev)
        gx_all[l] = workloads.activation(act, cfg.cid, l, 1, dev)
        keys.append(pk.make_key(B=act.B, S=act.S, H=H, **workloads.mask_key_fields(cfg.cid, layer=l)))
    xs, gxs = [x_all[l] for l in range(L)], [gx_all[l] for l in range(L)]
    vals = [torch.empty(L, rows, K, dtype=act.dtype, device=dev) for _ in range(2)]
    idx_s = torch.empty(L, rows, K, dtype=torch.int16, device=dev)      # the sender's kept positions
    idx_r = torch.empty_like(idx_s)                                      # the receiver's
    ys = [torch.empty(L, rows, H, dtype=act.dtype, device=dev) for _ in range(2)]
    mats = []
    nbuf = 2
    for l in range(L):
        for j, (m, n) in enumerate(gs.shapes):
            G_anc, G_mask = workloads.grad_pair_fast(gs, cfg.cid, l, j, dev)
            priors = [(torch.empty(m, r, device=dev), torch.empty(r, device=dev),
                       torch.empty(n, r, device=dev), torch.empty(r, device=dev)) for _ in range(nbuf)]
            ws = pk.workspace(m, n, r, p, gs.dtype)
            mats.append(dict(m=m, n=n, G_anc=G_anc, G_mask=G_mask,
                             M=torch.zeros(m, n, device=dev), out=priors[0], priors=priors,
                             Gp=torch.empty_like(G_mask), ws=ws,
                             cws=torch.empty(max(pk.sc_adamw_workspace_size(m, n, r, gs.dtype), 256),
                                             dtype=torch.uint8, device=dev)))
    # one batched call per phase over every matrix of the stage; with the
    # anchor prior built asynchronously (Sec. 3.2; Alg. 1 corrects with the
    # basis of the last anchor arrival), build b writes prior buffer b % 2
    # while the correction reads the other one
    build_items = [[dict(G_anc=mt["G_anc"], M=mt["M"], out=mt["priors"][b], ws=mt["ws"]) for mt in mats]
                   for b in range(nbuf)]
    corr_items = [[dict(G=mt["G_mask"], prior=(mt["priors"][b][0], mt["priors"][b][3], mt["priors"][b][2]),
                        out=mt["Gp"], ws=mt["cws"]) for mt in mats] for b in range(nbuf)]
    torch.cuda.synchronize()
    setup_s = time.time() - t0
    print(f"[bench] inputs ready in {setup_s:.1f} s; HBM in use "
          f"{torch.cuda.memory_allocated() / 2**30:.1f} GiB", file=sys.stderr, flush=True)

    if args.copy_probe:
        # torch.neg over 128 Mi floats: a plain elementwise kernel that reads
        # and writes exactly 512 MiB each
        src = torch.ones(1 << 27, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        torch.neg(src, out=dst)
        torch.cuda.synchronize()
        del src, dst

    ev = lambda: torch.cuda.Event(enable_timing=True)
    phase_ms = {"ac": 0.0, "build": 0.0, "correct": 0.0}
    # The timed step does every part once, each build with this step's
    # anchor gradient and each correction with the prior it built: the
    # subspace iteration of the build (EMA, power passes), then its
    # Rayleigh-Ritz step and the correction, with the masking (independent of
    # both) on a second stream beside them, after the streaming passes.  Two
    # more loops time the same work arranged otherwise:
    #   components.serial_step: masking, build, correction one after another
    #     on one stream;
    #   components.async_step: the build on a stream of its own beside the
    #     masking and a correction that uses the previous build's prior, as
    #     the method uses it (the prior is built asynchronously).
    # Every stream has the default priority.
    mode = ["overlap"]
    astream = torch.cuda.Stream()       # the asynchronous build
    side = torch.cuda.Stream()          # the overlapped step's masking
    n_steps_run = [0]
    built = {}      # step -> event after its build
    corrected = {}  # step -> event after its correction
    builders = {None: pk.sc_build_prior_batched, "sub": pk.sc_build_subspace_batched,
                "ritz": pk.sc_build_ritz_batched}

    def build(i, phase=None):
        bstream = astream if mode[0] == "async" else stream
        # correction i - 1 reads prior buffer (i - 2) % 2 = i % 2: it must be done
        if mode[0] == "async" and i - 1 in corrected:
            bstream.wait_event(corrected[i - 1])
        b0, b1 = ev(), ev()
        b0.record(bstream)
        with torch.cuda.stream(bstream):
            builders[phase](build_items[i % nbuf], r, workloads.BETA, workloads.TAU, p, q, seed=1000,
                            dtype=gs.dtype)
        b1.record(bstream)
        return b0, b1

    def masking():
        # forward: the sender packs from the key (keeping its index lists), the
        # receiver unpacks the values-only payload from the key (keeping its
        # own); backward: the receiver packs the gradient from its lists, the
        # sender unpacks it from its lists
        pk.ac_mask_pack_batched(x_all, K, keys[0], vals=vals[0], idx_out=idx_s)
        pk.ac_unpack_scatter_batched(vals[0], H, keys[0], scale, idx_out=idx_r, y=ys[0])
        pk.ac_mask_pack_batched(gx_all, K, keys[0], vals=vals[1], idx_in=idx_r)
        pk.ac_unpack_scatter_batched(vals[1], H, keys[0], scale, idx_in=idx_s, y=ys[1])

    def step(record: bool):
        i = n_steps_run[0]
        n_steps_run[0] += 1
        e0 = ev()
        e0.record(stream)
        if mode[0] == "overlap":
            s0, s1 = build(i, "sub")
            side.wait_event(s1)
            a0, a1 = ev(), ev()
            a0.record(side)
            with torch.cuda.stream(side):
                masking()
            a1.record(side)
            _, r1 = build(i, "ritz")
            bmark, b = (s0, r1), i % nbuf
        else:
            if mode[0] == "async":
                astream.wait_event(e0)
                bmark = build(i)
            a0, a1 = e0, ev()
            masking()
            a1.record(stream)
            if mode[0] == "serial":
                bmark, b = build(i), i % nbuf
            else:
                stream.wait_event(built[i - 1])            # the last finished anchor prior
                b = (i - 1) % nbuf
        built[i] = bmark[1]
        c0, c1 = ev(), ev()
        c0.record(stream)
        pk.sc_correct_batched(corr_items[b], r, workloads.ALPHA, dtype=gs.dtype)
        c1.record(stream)
        if mode[0] == "overlap":
            stream.wait_event(a1)                      # the next build streams M alone
        c = torch.cuda.Event()
        c.record(stream)
        corrected[i] = c
        return dict(ac=(a0, a1), build=bmark, correct=(c0, c1)) if record else None


    for _ in range(args.warmup):
        step(False)
    torch.cuda.synchronize()
    print(f"[bench] {args.warmup} warmup steps done", file=sys.stderr, flush=True)

    # Per-kernel pass, before the timed region: the same steps with every
    # launch bracketed by the library's events, and the phase events.  It
    # gives the per-kernel view and picks the dominant kernel.
    pass_tags = ("sc_pass_mz", "sc_pass_mtq")

    def dominant(per):
        cand = {name: ms for name, (n, ms) in per.items() if name not in pass_tags}
        cand["sc_pass"] = sum(per.get(t, (0, 0.0))[1] for t in pass_tags)
        return max(cand, key=cand.get)

    pk.acsc_stats_only(None)
    pk.acsc_stats_enable(True)
    torch.cuda.synchronize()
    marks = []
    for _ in range(args.steps):
        marks.append(step(True))
    torch.cuda.synchronize()
    stats = pk.acsc_stats_read()
    pk.acsc_stats_enable(False)
    for mk in marks:
        for ph, (x0, x1) in mk.items():
            phase_ms[ph] += x0.elapsed_time(x1) / args.steps
    dom = dominant(stats)
    # Timed region: the same steps with only the dominant kernel's launches
    # bracketed by events (two event records per launch of every kernel cost
    # the step about 1%); a dominant pair of pass kernels times every launch
    pk.acsc_stats_only(None if dom == "sc_pass" else dom)
    pk.acsc_stats_enable(True)
    torch.cuda.synchronize()
    start, stop = ev(), ev()
    start.record(stream)
    for _ in range(args.steps):
        step(False)
    stop.record(stream)
    torch.cuda.synchronize()
    timed_stats = pk.acsc_stats_read()
    pk.acsc_stats_enable(False)
    pk.acsc_stats_only(None)
    total_ms = start.elapsed_time(stop)
    ms_per_step = total_ms / args.steps
    print(f"[bench] {args.steps} timed steps: {ms_per_step:.3f} ms/step", file=sys.stderr, flush=True)

    # ---------------- algorithmic work of one step ----------------
    f_line = touched_line_fraction(H, K, esz)
    pack_bytes = f_line * rows * H * esz + rows * K * (esz + 2)
    unpack_bytes = rows * H * esz + rows * K * (esz + 2)
    passes = 2 * q + 2
    # with a large enough batch the first pass rides on the EMA's sweep over
    # M (one fused kernel, tagged sc_ema): the shadow is then streamed by
    # 2q + 1 passes, and the EMA kernel also does the first product
    pass_launches = sum(stats.get(t, (0, 0.0))[0] for t in ("sc_pass_mz", "sc_pass_mtq")) / args.steps
    fused_first = int(round(pass_launches)) == passes - 1
    shadow_passes = passes - 1 if fused_first else passes
    kk = min(r + p, min(gs.shapes[0]))
    # every form moves the same bytes per row: the key-driven pack writes the
    # index lists the index-driven one reads, and likewise for the unpack
    work = {"ac_pack": dict(bytes=L * pack_bytes, calls=1), "ac_pack_idx": dict(bytes=L * pack_bytes, calls=1),
            "ac_unpack": dict(bytes=L * unpack_bytes, calls=1),
            "ac_unpack_idx": dict(bytes=L * unpack_bytes, calls=1),
            "sc_ema": dict(bytes=0.0, calls=0), "sc_pass": dict(flops=0.0, bytes=0.0, calls=0),
            "sc_correct": dict(bytes=0.0, flops=0.0, calls=0),
            "sc_blend": dict(bytes=0.0, flops=0.0, calls=0), "sc_gv": dict(bytes=0.0, flops=0.0, calls=0)}
    for mt in mats:
        m, n = mt["m"], mt["n"]
        k = min(r + p, m, n, pk.SC_KMAX)
        work["sc_ema"]["bytes"] += m * n * (4 + 4 + gsz + (2 if gsz == 2 else 0))   # + bf16 shadow
        work["sc_ema"]["calls"] += 1
        work["sc_ema"]["flops"] = work["sc_ema"].get("flops", 0.0) + (2.0 * m * n * k if fused_first else 0.0)
        work["sc_pass"]["flops"] += shadow_passes * 2.0 * m * n * k
        work["sc_pass"]["bytes"] += shadow_passes * float(gsz) * m * n     # the shadow (bf16) or M (fp32)
        work["sc_pass"]["calls"] += shadow_passes
        work["sc_correct"]["bytes"] += 3.0 * m * n * gsz
        work["sc_correct"]["flops"] += 4.0 * m * n * r + 3.0 * m * n
        work["sc_correct"]["calls"] += 1
        work["sc_blend"]["bytes"] += 2.0 * m * n * gsz
        work["sc_blend"]["flops"] += 2.0 * m * n * r + 3.0 * m * n
        work["sc_blend"]["calls"] += 1
        work["sc_gv"]["bytes"] += 1.0 * m * n * gsz
        work["sc_gv"]["flops"] += 2.0 * m * n * r
        work["sc_gv"]["calls"] += 1
    ac_tags = ("ac_pack", "ac_pack_idx", "ac_unpack", "ac_unpack_idx")
    ac_bytes = sum(work[t]["bytes"] for t in ac_tags)
    step_bytes = ac_bytes + work["sc_ema"]["bytes"] + work["sc_pass"]["bytes"] + work["sc_correct"]["bytes"]
    step_flops = work["sc_pass"]["flops"] + work["sc_ema"].get("flops", 0.0) + work["sc_correct"]["flops"]
    value = step_bytes / (ms_per_step * 1e-3) / 1e9

    # ---------------- per-kernel view (library event timing) ----------------
    per_step = {name: (n / args.steps, ms / args.steps) for name, (n, ms) in stats.items()}
    groups = {"sc_pass": ("sc_pass_mz", "sc_pass_mtq")}
    kern = {}
    for name, (n, ms) in per_step.items():
        kern[name] = dict(launches_per_step=n, ms_per_step=ms, avg_us=1e3 * ms / max(n, 1e-9))
    # roofline models for the kernels whose work has a clean algorithmic count
    def model(name):
        if name in ac_tags or name == "sc_ema":
            return "hbm", work[name]["bytes"], work[name]["calls"]
        if name == "sc_blend":
            return "hbm", work["sc_blend"]["bytes"], work["sc_blend"]["calls"]
        if name == "sc_gv":
            return "hbm", work["sc_gv"]["bytes"], work["sc_gv"]["calls"]
        if name in groups["sc_pass"]:
            return "mfma", work["sc_pass"]["flops"], work["sc_pass"]["calls"]
        return None
    pass_ms = sum(per_step.get(t, (0, 0.0))[1] for t in groups["sc_pass"])
    pass_n = sum(per_step.get(t, (0, 0.0))[0] for t in groups["sc_pass"])
    # the dominant kernel's launches as timed inside the timed region
    timed = {name: (n / args.steps, ms / args.steps) for name, (n, ms) in timed_stats.items()}
    if dom == "sc_pass":
        # a pass is bound by whichever roof is lower at its arithmetic
        # intensity (k FLOP per byte of the streamed shadow): below the ridge
        # point (peak FLOP/s over peak B/s) that is HBM
        peak_mm = PEAK_BF16 if gs.dtype == torch.bfloat16 else PEAK_F32
        ai = work["sc_pass"]["flops"] / work["sc_pass"]["bytes"]
        ridge = peak_mm * 1e12 / (PEAK_HBM * 1e9)
        if ai < ridge:
            bound, amount, calls = "hbm", work["sc_pass"]["bytes"], work["sc_pass"]["calls"]
        else:
            bound, amount, calls = "mfma", work["sc_pass"]["flops"], work["sc_pass"]["calls"]
        dom_ms = sum(timed.get(t, (0, 0.0))[1] for t in groups["sc_pass"])
        dom_n = sum(timed.get(t, (0, 0.0))[0] for t in groups["sc_pass"])
    else:
        mm = model(dom)
        dom_n, dom_ms = timed[dom]
        bound, amount, calls = mm if mm else ("latency", 0.0, dom_n)
    # achieved = algorithmic work of every launch of the kernel in the timed
    # region / the summed event-measured duration of those launches
    avg_s = dom_ms * 1e-3 / max(dom_n, 1e-9)
    total_s = dom_ms * 1e-3
    per_launch = amount / max(dom_n, 1e-9)
    if bound == "hbm":
        achieved = amount / total_s / 1e9
        roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM, "unit": "GB/s",
                "frac": round(achieved / PEAK_HBM, 4)}
    elif bound == "mfma":
        achieved = amount / total_s / 1e12
        peak = PEAK_BF16 if gs.dtype == torch.bfloat16 else PEAK_F32
        roof = {"bound": "mfma", "achieved": round(achieved, 2), "peak": peak, "unit": "TFLOP/s",
                "frac": round(achieved / peak, 4)}
    else:
        roof = {"bound": "latency", "achieved": None, "peak": None, "unit": None, "frac": None}
    roof.update({"kernel": dom, "avg_launch_us": round(avg_s * 1e6, 2),
                 "launches_per_step": dom_n, "work_per_launch": per_launch,
                 "work_unit": "bytes" if bound == "hbm" else "flops",
                 "traffic": measured_traffic(dom, cfg.cid)})

    comp = {}
    for name in ac_tags + ("sc_ema", "sc_gv", "sc_blend"):
        if name in per_step:
            n, ms = per_step[name]
            gbs = work[name]["bytes"] / (ms * 1e-3) / 1e9
            comp[name] = {"GB/s": round(gbs, 1), "frac_hbm": round(gbs / PEAK_HBM, 4),
                          "ms_per_step": round(ms, 4), "launches_per_step": n}
    if pass_ms > 0:
        tf = work["sc_pass"]["flops"] / (pass_ms * 1e-3) / 1e12
        pk_ = PEAK_BF16 if gs.dtype == torch.bfloat16 else PEAK_F32
        comp["sc_pass"] = {"TFLOP/s": round(tf, 2), "frac_mfma": round(tf / pk_, 4),
                           "GB/s": round(work["sc_pass"]["bytes"] / (pass_ms * 1e-3) / 1e9, 1),
                           "frac_hbm": round(work["sc_pass"]["bytes"] / (pass_ms * 1e-3) / 1e9 / PEAK_HBM, 4),
                           "ms_per_step": round(pass_ms, 4), "launches_per_step": pass_n}
    comp["phase_ms"] = {k: round(v, 4) for k, v in phase_ms.items()}
    comp["sc_correct_step"] = {"GB/s": round(work["sc_correct"]["bytes"] / (phase_ms["correct"] * 1e-3) / 1e9, 1),
                               "TFLOP/s": round(work["sc_correct"]["flops"] / (phase_ms["correct"] * 1e-3) / 1e12, 2)}
    comp["ac_step"] = {"GB/s": round(ac_bytes / (phase_ms["ac"] * 1e-3) / 1e9, 1)}
    comp["kernels"] = {k: {kk_: round(v, 4) if isinstance(v, float) else v for kk_, v in d.items()}
                       for k, d in sorted(kern.items())}

    # the method's cadence (Table 2: an anchor arrives every K = 20 fast
    # steps): every step masks and corrects, one step in 20 also builds the
    # prior; device time from the summed kernel times of each part
    corr_tags = ("sc_vconvert", "sc_gv", "sc_utt", "sc_inner_reduce", "sc_filter", "sc_ux", "sc_blend")
    part_ms = {"masking": 0.0, "correction": 0.0, "build": 0.0}
    for name, (n, ms) in per_step.items():
        part = "masking" if name.startswith("ac_") else "correction" if name in corr_tags else "build"
        part_ms[part] += ms
    staleness = 20
    cyc_ms = part_ms["masking"] + part_ms["correction"] + part_ms["build"] / staleness
    cyc_bytes = ac_bytes + work["sc_correct"]["bytes"] + (work["sc_ema"]["bytes"] + work["sc_pass"]["bytes"]) / staleness
    comp["per_cycle"] = {"builds_per_step": f"1/{staleness}", "kernel_ms": {k: round(v, 4) for k, v in part_ms.items()},
                         "ms_per_step": round(cyc_ms, 4), "GB/s": round(cyc_bytes / (cyc_ms * 1e-3) / 1e9, 1),
                         "frac_hbm": round(cyc_bytes / (cyc_ms * 1e-3) / 1e9 / PEAK_HBM, 4),
                         "basis": "summed kernel times of the timed steps (library events), one build per "
                                  f"{staleness} masked and corrected steps"}

    if not args.no_adamw:
        comp["sc_correct_adamw"] = adamw_component(pk, mats, r, gs, max(1, min(args.steps, 5)), stream)
    if not args.no_bernoulli:
        comp["ac_bernoulli"] = bernoulli_component(pk, xs, gxs, keys, act, keep, esz, max(1, min(args.steps, 5)),
                                                   stream)

    if not args.no_powersgd:
        comp["psgd"] = psgd_component(pk, mats, gs, max(1, min(args.steps, 5)), stream)

    def other_arrangement(name, kernel_stats=False):
        mode[0] = name
        for _ in range(args.warmup):
            step(False)
        torch.cuda.synchronize()
        if kernel_stats:
            pk.acsc_stats_enable(True)
            torch.cuda.synchronize()
        a0, a1 = ev(), ev()
        a0.record(stream)
        for _ in range(args.steps):
            step(False)
        stream.wait_stream(astream)                    # the last build is part of the timed work
        a1.record(stream)
        torch.cuda.synchronize()
        mode[0] = "overlap"
        ams = a0.elapsed_time(a1) / args.steps
        out = {"ms_per_step": round(ams, 4), "value": round(step_bytes / (ams * 1e-3) / 1e9, 1),
               "unit": "GB/s", "speedup": round(ms_per_step / ams, 4), "steps": args.steps}
        if kernel_stats:
            st = pk.acsc_stats_read()
            pk.acsc_stats_enable(False)
            # the masking kernels on their own (in the timed step they share
            # the GPU with the Rayleigh-Ritz step)
            for tag in ac_tags:
                if tag in st:
                    kms = st[tag][1] / args.steps
                    gbs = work[tag]["bytes"] / (kms * 1e-3) / 1e9
                    out[tag] = {"GB/s": round(gbs, 1), "frac_hbm": round(gbs / PEAK_HBM, 4),
                                "ms_per_step": round(kms, 4), "avg_us": round(1e3 * kms / work[tag]["calls"], 2)}
        return out

    # the same steps in one stream, one part after another
    comp["serial_step"] = other_arrangement("serial", kernel_stats=True)
    if not args.no_async:
        # the same steps with the build on its own stream (the correction uses the
        # previous build's prior); the first such step corrects with the last
        # serial step's prior
        comp["async_step"] = other_arrangement("async")

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(cfg, args.cpu_seconds)

    shapes = "+".join(f"{m}x{n}" for m, n in gs.shapes)
    line = {
        "metric": METRIC, "value": round(value, 1), "unit": "GB/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"{cfg.name}: activation [{act.B},{act.S},{H}] keep {keep} (K={K}) "
                               f"fwd+bwd x{L} layers; gradients {shapes} x{L} layers, rank-{gs.rank} "
                               f"signal + noise; r={r}, k={kk}, power_iters={q}",
                   "step": "anchor-prior subspace iteration alone; then its Rayleigh-Ritz step and the correction with that prior, the masking beside them on a second stream",
                   "step_bytes": step_bytes, "step_flops": step_flops,
                   "step_TFLOP/s": round(step_flops / (ms_per_step * 1e-3) / 1e12, 2)},
        "roofline": roof,
        "cpu_baseline": cpu,
        "components": comp,
    }
    print(json.dumps(line), flush=True)
    return 0


def adamw_component(pk, mats, r, gs, calls, stream):
    """The next row after the correction: the corrected AdamW step (the
    correction with the optimiser update fused into its blend), on the same
    matrices, timed on its own after the step loop.  Algorithmic bytes per
    element: G read twice (X = U^T G V needs all of G before any element of
    G_proj exists) and the fp32 weights and both moments read and written."""
    import torch
    import workloads
    dev = mats[0]["G_mask"].device
    items = []
    for j, mt in enumerate(mats):
        g = torch.Generator(device=dev).manual_seed(500 + j)
        W = torch.randn(mt["m"], mt["n"], device=dev, generator=g)
        items.append(dict(G=mt["G_mask"], prior=(mt["out"][0], mt["out"][3], mt["out"][2]), ws=mt["ws"],
                          state=(W, torch.zeros_like(W), torch.zeros_like(W))))
    hp = dict(lr=2e-5, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.01, max_norm=0.2)
    pk.sc_correct_adamw_batched(items, r, workloads.ALPHA, step=1, dtype=gs.dtype, **hp)
    torch.cuda.synchronize()
    pk.acsc_stats_enable(True)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for t in range(calls):
        pk.sc_correct_adamw_batched(items, r, workloads.ALPHA, step=t + 2, dtype=gs.dtype, **hp)
    e1.record(stream)
    torch.cuda.synchronize()
    st = pk.acsc_stats_read()
    pk.acsc_stats_enable(False)
    ms = e0.elapsed_time(e1) / calls
    elems = float(sum(mt["m"] * mt["n"] for mt in mats))
    gsz = 2 if gs.dtype == torch.bfloat16 else 4
    algo = elems * (2 * gsz + 24)
    out = {"ms_per_call": round(ms, 4), "GB/s": round(algo / (ms * 1e-3) / 1e9, 1),
           "frac_hbm": round(algo / (ms * 1e-3) / 1e9 / PEAK_HBM, 4), "bytes_per_call": algo,
           "hparams": hp}
    if "sc_blend_adamw" in st:
        n, kms = st["sc_blend_adamw"]
        bb = elems * (gsz + 24)
        rate = bb * calls / (kms * 1e-3) / 1e9     # every call's launches cover all elements once
        out["sc_blend_adamw"] = {"ms_per_call": round(kms / calls, 4), "GB/s": round(rate, 1),
                                 "frac_hbm": round(rate / PEAK_HBM, 4)}
    out["kernels"] = {k: {"launches_per_call": n / calls, "ms_per_call": round(v / calls, 4)}
                      for k, (n, v) in sorted(st.items())}
    del items
    torch.cuda.empty_cache()
    return out


def bernoulli_component(pk, xs, gxs, keys, act, keep, esz, calls, stream):
    """The Bernoulli mask variant on the same boundaries: per layer the mask
    (row offsets and bitmaps, from the key) once, then pack and unpack of the
    activation and of its gradient; timed on its own after the step loop.
    Algorithmic bytes: pack, the 128-byte lines of x holding a kept entry
    (1 - (1 - q)^E of them, E entries per line) plus the payload and its
    indices; unpack, the dense write plus the payload read; mask, the
    bitmaps and offsets written."""
    import torch
    H, rows = act.H, act.B * act.S
    L = len(xs)
    ys = torch.empty(rows, H, dtype=act.dtype, device=xs[0].device)
    masks = [pk.ac_bern_mask(rows, H, keep, keys[l]) for l in range(L)]
    torch.cuda.synchronize()
    nnz = [int(rp[-1].item()) for rp, _ in masks]
    bufs = [torch.empty(n, dtype=act.dtype, device=xs[0].device) for n in nnz]
    idxs = [torch.empty(n, dtype=torch.int16, device=xs[0].device) for n in nnz]

    def run():
        for l in range(L):
            rp, bits = pk.ac_bern_mask(rows, H, keep, keys[l])
            for src in (xs[l], gxs[l]):
                pk.lib.ac_bern_pack(pk._ptr(src), pk._dt(src), rows, H, H, pk._ptr(rp), pk._ptr(bits),
                                    pk._ptr(bufs[l]), pk._ptr(idxs[l]), nnz[l], pk._stream())
                pk.ac_bern_unpack(bufs[l], H, rp, bits, 1.0 / keep, y=ys)
    run()
    torch.cuda.synchronize()
    pk.acsc_stats_enable(True)
    for _ in range(calls):
        run()
    torch.cuda.synchronize()
    st = pk.acsc_stats_read()
    pk.acsc_stats_enable(False)
    q = round(keep * 65536) / 65536
    E = 128 // esz
    line = 1.0 - (1.0 - q) ** E
    nz = sum(nnz) / L
    work = {"ac_bern_pack": line * rows * H * esz + nz * (esz + 2),
            "ac_bern_unpack": rows * H * esz + nz * esz + rows * H / 8,
            "ac_bern_mask": rows * H / 8 + 8 * (rows + 1)}
    out = {"keep": keep, "kept_per_row": round(nz / rows, 2)}
    for k, b in work.items():
        if k in st:
            n, ms = st[k]
            per = ms / n
            out[k] = {"launches_per_step": n / calls, "avg_us": round(1e3 * per, 2),
                      "GB/s": round(b / (per * 1e-3) / 1e9, 1), "frac_hbm": round(b / (per * 1e-3) / 1e9 / PEAK_HBM, 4)}
    if "ac_bern_scan" in st:
        n, ms = st["ac_bern_scan"]
        out["ac_bern_scan"] = {"avg_us": round(1e3 * ms / n, 2)}
    del bufs, idxs, ys
    return out


def psgd_component(pk, mats, gs, calls, stream):
    """The data-parallel compressor the method is paired with: one PowerSGD
    step with error feedback on every gradient of the step (x64 ranks; equal
    ranks share a call), timed on its own after the step loop.  Algorithmic
    bytes per element: the first sweep reads G and the fp32 memory and writes
    the memory and its bf16 copy (12 with bf16 G), the second projection
    reads the copy (2), the decompression reads and writes the memory and
    writes the output (10)."""
    import torch
    from paper_2609_14339_amd.powersgd import PowerSGDState
    dev = mats[0]["G_mask"].device
    grads = [mt["G_mask"] for mt in mats]
    state = PowerSGDState([(mt["m"], mt["n"]) for mt in mats], 64.0, gs.dtype, dev, seed=3)
    outs = [torch.empty_like(g) for g in grads]
    state.step(grads, outs, stream)
    torch.cuda.synchronize()
    pk.acsc_stats_enable(True)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(calls):
        state.step(grads, outs, stream)
    e1.record(stream)
    torch.cuda.synchronize()
    st = pk.acsc_stats_read()
    pk.acsc_stats_enable(False)
    ms = e0.elapsed_time(e1) / calls
    elems = float(sum(mt["m"] * mt["n"] for mt in mats))
    gsz = 2 if gs.dtype == torch.bfloat16 else 4
    algo = elems * ((gsz + 8 + 2) + 2 + 10)
    full = elems * gsz
    out = {"ms_per_call": round(ms, 4), "GB/s": round(algo / (ms * 1e-3) / 1e9, 1),
           "frac_hbm": round(algo / (ms * 1e-3) / 1e9 / PEAK_HBM, 4), "bytes_per_call": algo,
           "ranks": sorted(set(state.ranks)), "compression": round(full / gsz / state.sent_elements(), 2)}
    # per sweep, each covering every element once per call: the first sweep
    # (fused with P = M Q where the group's row blocks fill the GPU, else the
    # sweep and a pass over the copy), the second projection, the decompression
    sweeps = (("first_sweep", ("psgd_feedback_mq", "psgd_feedback", "psgd_pass_mq"), gsz + 10),
              ("psgd_pass_mtp", ("psgd_pass_mtp",), 2), ("psgd_decompress", ("psgd_decompress",), 10))
    for name, tags, per_elem in sweeps:
        kms = sum(st[t][1] for t in tags if t in st)
        if kms > 0:
            rate = elems * per_elem * calls / (kms * 1e-3) / 1e9
            out[name] = {"ms_per_call": round(kms / calls, 4), "GB/s": round(rate, 1),
                         "frac_hbm": round(rate / PEAK_HBM, 4), "bytes_per_elem": per_elem}
    out["kernels"] = {k: {"launches_per_call": n / calls, "ms_per_call": round(v / calls, 4)}
                      for k, (n, v) in sorted(st.items())}
    del state, outs
    torch.cuda.empty_cache()
    return out


TRAFFIC_FILE = os.path.join(ROOT, "profiles", "hotpath_70b_4layer_hbm_traffic.txt")


def kernel_sources_digest() -> str:
    """SHA-256 over the library's kernel sources (csrc/*.hip, csrc/*.h), in name order."""
    import hashlib
    d = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2609_14339_amd", "csrc")
    for name in sorted(os.listdir(csrc)):
        if name.endswith((".hip", ".h")):
            with open(os.path.join(csrc, name), "rb") as f:
                d.update(name.encode() + b"\0" + f.read())
    return d.hexdigest()


def measured_traffic(tag: str, cid: int):
    """HBM bytes per launch of kernel `tag` from the stored counter summary
    (FETCH_SIZE + WRITE_SIZE, each scaled by a plain copy kernel's reading),
    or None when there is none for this workload or the kernel sources have
    changed since the counters were taken."""
    if cid != 5 or not os.path.exists(TRAFFIC_FILE):
        return None
    digest, table = None, {}
    with open(TRAFFIC_FILE) as f:
        for line in f:
            if line.startswith("# sources_sha256:"):
                digest = line.split(":", 1)[1].strip()
            elif line.startswith("traffic "):
                _, name, per_launch = line.split()[:3]
                table[name] = float(per_launch)
    if digest != kernel_sources_digest() or tag not in table:
        return None
    return table[tag]


def _lscpu() -> dict:
    """Model, sockets, cores and hardware threads of the host (lscpu), and the
    CPUs this process may run on."""
    info = {"model": platform.processor() or "unknown"}
    try:
        out = subprocess.run(["lscpu"], capture_output=True, text=True).stdout
        kv = {l.split(":", 1)[0].strip(): l.split(":", 1)[1].strip() for l in out.splitlines() if ":" in l}
        sockets = int(kv.get("Socket(s)", "1"))
        cores = int(kv.get("Core(s) per socket", "0")) * sockets
        info = {"model": kv.get("Model name", info["model"]), "sockets": sockets, "cores": cores,
                "threads": int(kv.get("CPU(s)", "0")), "threads_per_core": int(kv.get("Thread(s) per core", "1"))}
    except Exception:
        pass
    info["affinity"] = len(os.sched_getaffinity(0))
    return info


def _timed(fn, repeat_below_s: float = 10.0):
    """Wall time of fn(): the median of three runs when one run takes less
    than repeat_below_s, else that one run.  Returns (seconds, runs)."""
    t = time.time()
    fn()
    first = time.time() - t
    if first >= repeat_below_s:
        return first, 1
    times = [first]
    for _ in range(2):
        t = time.time()
        fn()
        times.append(time.time() - t)
    return sorted(times)[1], 3


def cpu_baseline(cfg, budget_s: float):
    """The oracle as it stands, on host cores, on a bounded sample of the same
    workload, and single-thread figures of the two small configurations:
      mask leg      the C oracle's pack + unpack of 2048 rows of layer 0 (one
                    thread: the C oracle is single-threaded);
      spectral leg  the float64 oracle's EMA + LAPACK SVD + correction of a
                    leading block of the first gradient (LAPACK/BLAS threads
                    as reported by threadpoolctl);
      C1 / C2       the same legs at the tiny and 1B-class configurations with
                    BLAS held to one thread (C1 whole; C2 the whole activation
                    and the first 2048 x 2048 gradient).
    `value` is the algorithmic bytes of the two sample legs over their summed
    time; legs under 10 s are the median of three runs."""
    import numpy as np
    import torch
    import workloads
    from oracle import mask as om
    from oracle import spectral as osp
    try:
        from threadpoolctl import threadpool_info, threadpool_limits
        blas_threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        threadpool_limits = None
        blas_threads = 1

    def mask_leg(c, rows):
        act = c.act
        H = act.H
        K = om.keep_count(H, act.keep[0])
        esz = 2 if act.dtype == torch.bfloat16 else 4
        x = workloads.activation(act, c.cid, 0, 0, "cpu", rows=rows)
        xh = x.view(torch.int16).numpy().view(np.uint16) if x.dtype == torch.bfloat16 else x.numpy()
        key = om.mask_key(**{k: v for k, v in workloads.mask_key_fields(c.cid).items()}, B=act.B, S=act.S, H=H)

        def run():
            vals, idx = om.pack(xh, K, key)
            om.unpack(vals, H, key, H / K, idx=idx)
        secs, runs = _timed(run)
        nbytes = (touched_line_fraction(H, K, esz) * rows * H * esz + rows * K * (esz + 2)
                  + rows * H * esz + rows * K * (esz + 2))
        return secs, runs, nbytes

    def spectral_leg(c, m, n):
        gs = c.grad
        gsz = 2 if gs.dtype == torch.bfloat16 else 4
        spec = workloads.GradSpec(((m, n),), min(gs.rank, m, n), gs.s_range, (min(gs.r[0], m, n),),
                                  gs.dtype, gs.anc_noise, gs.mask_noise)
        gp = workloads.grad_pair(spec, c.cid, 0, 0, "cpu")
        Ga, Gm = gp.G_anc.double().numpy(), gp.G_mask.double().numpy()

        def run():
            osp.corrected_step(np.zeros((m, n)), Ga, Gm, workloads.BETA, spec.r[0], workloads.TAU,
                               workloads.ALPHA)
        secs, runs = _timed(run)
        # EMA (M and G read, M written), one read of M for the SVD, the correction's 3 mn
        return secs, runs, m * n * (4 + 4 + gsz) + 4 * m * n + 3 * m * n * gsz

    act, gs = cfg.act, cfg.grad
    rows = 2048
    t_ac, r_ac, ac_bytes = mask_leg(cfg, rows)
    # spectral sample: leading block of the first gradient matrix, sized to the budget
    m0, n0 = gs.shapes[0]
    side = 1024
    while side * 2 <= min(m0, n0) and (side * 2) ** 3 * 4 / 2e10 < budget_s:
        side *= 2
    m, n = min(side, m0), min(side, n0)
    t_sc, r_sc, sc_bytes = spectral_leg(cfg, m, n)
    single = {}
    if threadpool_limits is not None:
        with threadpool_limits(limits=1):
            for cid in (1, 2):
                c = workloads.CONFIGS[cid]
                ta, ra, ba = mask_leg(c, c.act.B * c.act.S)
                mm, nn = c.grad.shapes[0]
                ts, rs, bs = spectral_leg(c, mm, nn)
                single[f"C{cid}"] = {"threads": 1, "mask_s": round(ta, 4), "mask_runs": ra,
                                     "mask_rows": c.act.B * c.act.S, "spectral_s": round(ts, 4),
                                     "spectral_runs": rs, "spectral_block": f"{mm}x{nn}",
                                     "GB/s": round((ba + bs) / (ta + ts) / 1e9, 4)}
    total = t_ac + t_sc
    return {"value": round((ac_bytes + sc_bytes) / total / 1e9, 3), "unit": "GB/s",
            "cores": int(blas_threads), "kind": "oracle",
            "sample": f"C oracle pack+unpack of {rows} rows x H={act.H} (1 thread, {t_ac:.3f} s, "
                      f"{'median of 3' if r_ac == 3 else 'one run'}); float64 oracle EMA + LAPACK SVD + "
                      f"correction of a {m}x{n} block of the {m0}x{n0} gradient ({blas_threads} BLAS threads, "
                      f"{t_sc:.2f} s, {'median of 3' if r_sc == 3 else 'one run'})",
            "legs": {"mask": {"threads": 1, "seconds": round(t_ac, 4), "runs": r_ac},
                     "spectral": {"threads": int(blas_threads), "seconds": round(t_sc, 3), "runs": r_sc}},
            "single_thread": single, "host": _lscpu(), "seconds": round(total, 2)}


if __name__ == "__main__":
    sys.exit(main())
