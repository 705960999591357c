"""Throughput of the one-GPU 3DGS training-view hot path.

A step is one training view through every phase: projection, visible-set
extraction, tile binning + sort, forward raster fused with the L1 loss (and
the realized active set: the primitives some pixel blended, as ascending ids),
backward, sparse Adam over the visible rows with its steps staged as a
publication message, and the commit of that message to a replica (the
pending-update publication).  The workload is the 1M-Gaussian
SH-degree-3 room scene with 32 forward-facing 1920x1080 cameras; steps cycle
through the cameras.  The primitive pool is stored in spatial (Morton) order
of the means, a load-time layout step outside the timed region
(--id-order given keeps the generator's order; the extras time the other
order too).  Inputs (scene, Adam state, all 32 targets) are resident in HBM
before the timed region.

Each view's commit to the replica runs on a second stream, started after the
next view's forward + loss so that it runs beside that view's backward raster
(which reads projection outputs, not the replica); --no-overlap runs
everything on one stream.  Every timed view's apply completes inside the timed region.

Prints one JSON line (the driver's contract) with a roofline entry for the
dominant kernel (timed with HIP events on the stream it runs on) and the CPU
oracle timed on a bounded sample of the same workload.  Extras beside it
(--no-extras skips them): the scope hazards and admission gate between
consecutive views, two-view task units, the host planner (graph,
partition, schedule) on synthetic captures of 1,000 to 50,000 images, the
same training step on the other four workloads (short runs: views/s and
per-phase fractions of peak), the publication kernels alone (pack, apply,
versioned commit) on the 3M and 10M workloads, and the oracle's per-stage
times on every workload's view sample.
"""
from __future__ import annotations

import argparse
import gc
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, GB/s
FP32_PEAK_TFLOPS = 157.3       # MI355X vector FP32 (packed), TFLOP/s

# Algorithmic work per unit (see the design notes for the derivation).
FWD_FLOP_EVAL = 13.0           # per evaluated (pixel, pair): offsets, quadratic form, exp, alpha
FWD_FLOP_INC = 9.0             # per included pair: transmittance update + colour accumulation
BWD_FLOP_EVAL = 13.0           # per replayed (pixel, pair): alpha recomputation
BWD_FLOP_INC = 54.0            # per included pair: transmittance recovery, dL/dalpha, 9 partials + their sum


# HBM traffic of the dominant kernel (k_raster_bwd) on this workload, from two
# rocprofv3 --pmc passes (FETCH_SIZE, then WRITE_SIZE; KiB per dispatch, mean
# of the 10 dispatches of an 8-step run without extras: 2 warm-up and 8 timed),
# each scaled by what the same counter reads for a plain device copy of known
# size (a 1 GiB read registers as 0.5 GiB of FETCH_SIZE, a 1 GiB write as
# 1 GiB of WRITE_SIZE).  Valid only for the workload and the code it was
# measured on (comments aside): the kernel's source and the bin sort, whose
# tile dispatch order decides what the kernel finds in L2, and the pool's
# storage order; reported as null for other workloads, another storage order
# and once either source changes.
TRAFFIC = {
    "kernel": "k_raster_bwd",
    "phase": "raster_bwd_pixels",
    "workload": "room-1M-L3-1080p",
    "id_order": "spatial",
    "sources": ["paper_2607_19893_amd/csrc/raster.hip", "paper_2607_19893_amd/csrc/binsort.hip"],
    "code_sha256": "60c6eb1a4bc46d587fb4164bc2cc0fa91dee0deab096d3be3fda849634a6a28d",
    "fetch_kib": 109111.74, "fetch_scale": 1048576.0 / 524294.5,
    "write_kib": 91881.94, "write_scale": 1048576.0 / 1048576.0,
    "profile": "profiles/k_raster_bwd-room-1M-1080p_hbm_traffic.md",
}


def no_collector():
    """Run a full collector pass now and switch the collector off (until
    gc.enable()): a pass over the process's Python objects inside a timed
    loop can hold the issuing thread for tens of milliseconds and idle the
    GPU at a random phase."""
    gc.collect()
    gc.disable()


def code_digest(text):
    """sha256 of a C/C++ source with comments, blank lines and trailing blanks removed."""
    import hashlib
    import re
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    text = re.sub(r"//[^\n]*", "", text)
    text = "\n".join(line.rstrip() for line in text.splitlines() if line.strip())
    return hashlib.sha256(text.encode()).hexdigest()


def traffic_digest():
    return code_digest("\n".join(open(os.path.join(ROOT, f)).read() for f in TRAFFIC["sources"]))


def traffic_bytes(workload, phase, id_order):
    """HBM bytes per launch of the dominant kernel on `workload`, or None if the counters were taken on
    another workload, kernel or storage order, or the code changed since."""
    if workload != TRAFFIC["workload"] or phase != TRAFFIC["phase"] or id_order != TRAFFIC["id_order"]:
        return None
    try:
        digest = traffic_digest()
    except OSError:
        return None
    if digest != TRAFFIC["code_sha256"]:
        return None
    return 1024.0 * (TRAFFIC["fetch_kib"] * TRAFFIC["fetch_scale"] + TRAFFIC["write_kib"] * TRAFFIC["write_scale"])


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=64)
    ap.add_argument("--warmup", type=int, default=8)
    ap.add_argument("--workload", default="room")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-views", type=int, default=8, help="views of the CPU oracle sample")
    ap.add_argument("--no-overlap", action="store_true",
                    help="run every phase on one stream (by default each view's apply to the replica runs on a "
                         "second stream, beside the next view's backward raster)")
    ap.add_argument("--apply-after", type=int, default=None,
                    help="phase index after which the previous view's commit starts on the second stream "
                         "(default: the pipeline's choice)")
    ap.add_argument("--no-extras", action="store_true",
                    help="skip the separate timings of the scope hazards / admission gate and of two-view task units")
    ap.add_argument("--dense-params", action="store_true",
                    help="hold the parameter groups as five dense tensors instead of dense means and SH beside one "
                         "[n, 8] head table of quat, log_scale and opacity (same arithmetic, different addresses)")
    ap.add_argument("--row-major-tiles", action="store_true",
                    help="let the raster workgroups take the tiles in row-major order instead of the bin sort's "
                         "longest-first dispatch order (same results)")
    ap.add_argument("--id-order", choices=("spatial", "given"), default="spatial",
                    help="storage order of the primitive pool: spatial (Morton order of the means, a load-time "
                         "layout step) or given (the generator's order); the scene's content is the same")
    ap.add_argument("--delta-only", action="store_true",
                    help="only time the publication kernels alone (cold) on --workload and print them; for "
                         "profiling those kernels")
    ap.add_argument("--copy-probe-mib", type=int, default=0,
                    help="only run a plain device copy (read + write of this many MiB, 4 times) and exit; "
                         "its HBM counters calibrate the traffic counters of the path's kernels")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU: this build has no multi-GPU path (collectives and sharding are "
              "out of scope); run with --gpus 1", file=sys.stderr)
        sys.exit(2)

    import torch
    if args.copy_probe_mib > 0:
        copy_probe(args.copy_probe_mib)
        return
    from paper_2607_19893_amd.pipeline import ViewTrainer

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    if args.apply_after is not None:
        ViewTrainer.APPLY_AFTER = args.apply_after
    if args.delta_only:
        r = run_workload(args.workload, 2, 1, overlap=not args.no_overlap, id_order=args.id_order)
        print(json.dumps({"delta": {r["w"].name: bench_delta(r["tr"], r["cams"])}}), flush=True)
        return
    run = run_workload(args.workload, args.steps, args.warmup, overlap=not args.no_overlap,
                       packed=not args.dense_params, row_major=args.row_major_tiles, id_order=args.id_order)
    tr, cams, targets, w = run.pop("tr"), run.pop("cams"), run.pop("targets"), run.pop("w")

    extras = {}
    if not args.no_extras:
        extras["scope_gate"] = bench_scope_gate(tr, cams, targets, args.steps)
        extras["unit2"] = bench_unit(tr, cams, targets, args.steps, run["step"])
        extras["planner"] = bench_planner()
        log("extras: " + json.dumps(extras))
    del tr, targets
    torch.cuda.empty_cache()
    if not args.no_extras:
        # the same workload with the pool in the other storage order (same step, same views)
        other = "given" if args.id_order == "spatial" else "spatial"
        r = run_workload(args.workload, args.steps, args.warmup, overlap=not args.no_overlap, id_order=other)
        extras["other_id_order"] = {k: r[k] for k in ("id_order", "views_per_s", "ms_per_step", "phases_ms")}
        del r
        torch.cuda.empty_cache()
        # every other workload through the same timed step (short runs), and the
        # publication kernels alone on the two workloads whose step carries them
        extras["workloads"] = {}
        extras["delta"] = {}
        for name in OTHER_WORKLOADS:
            r = run_workload(name, OTHER_STEPS, OTHER_WARMUP, overlap=not args.no_overlap, id_order=args.id_order)
            if name in DELTA_WORKLOADS:
                extras["delta"][r["w"].name] = bench_delta(r["tr"], r["cams"])
            extras["workloads"][r["w"].name] = {k: r[k] for k in ("id_order", "views_per_s", "ms_per_step", "steps", "views",
                                                                  "mean_visible", "mean_pairs", "phases_ms",
                                                                  "phases_frac")}
            del r
            torch.cuda.empty_cache()
        log("workloads: " + json.dumps(extras["workloads"]))
        log("delta: " + json.dumps(extras["delta"]))

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(w, args.cpu_views)
        if not args.no_extras:
            extras["planner"]["oracle"] = planner_oracle_time(PLAN_ORACLE_VIEWS)
            extras["oracle_stages"] = oracle_stage_times()

    out = {
        "metric": "train views/sec (fwd+bwd+sparse Adam), 1M Gaussians 1080p",
        "value": run["views_per_s"],
        "unit": "views/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": run["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": w.name, "gaussians": w.scene.n, "sh_degree": w.scene.sh_degree,
                   "width": cams[0].width, "height": cams[0].height, "views": len(cams),
                   "mean_visible": run["mean_visible"], "mean_pairs": run["mean_pairs"],
                   "step": "project+visible+bin_sort+fwd_l1+active_set+bwd+sparse_adam_publish+commit",
                   "apply_overlapped": not args.no_overlap,
                   "param_layout": "dense" if args.dense_params else "head8",
                   "id_order": args.id_order,
                   "tile_dispatch": "row_major" if args.row_major_tiles else "longest_first"},
        "roofline": run["roofline"],
        "phases_ms": run["phases_ms"],
        "phases_frac": run["phases_frac"],
        "cpu_baseline": cpu,
        "extras": extras,
    }
    print(json.dumps(out), flush=True)


# the other workloads of the default run: short timed runs of the same step
OTHER_WORKLOADS = ("tiny", "ring", "spiral", "aerial")
OTHER_STEPS, OTHER_WARMUP = 24, 6
DELTA_WORKLOADS = ("spiral", "aerial")


_RENDERERS = {}


def gpu_render(scene, cam):
    """Target image of a workload whose targets are renders of its perturbed
    copy: the copy rendered by the library's own projection, binning and
    forward raster (made once per workload before any timing)."""
    import torch
    from paper_2607_19893_amd.pipeline import ViewTrainer
    key = id(scene)
    tr = _RENDERERS.get(key)
    if tr is None:
        _RENDERERS.clear()
        tr = _RENDERERS[key] = ViewTrainer(scene, capacity=1, max_width=cam.width, max_height=cam.height)
    if cam.width > tr.width or cam.height > tr.height:
        tr._set_image(cam.width, cam.height)
    tr.ensure_capacity([cam])
    tr.project(cam)
    tr.visible()
    tr.bin_sort()
    tr.raster_fwd(active=False)
    torch.cuda.synchronize()
    n = cam.width * cam.height
    return tr.img.view(-1)[:3 * n].cpu().numpy().reshape(3, cam.height, cam.width).copy()


def oracle_render(scene, cam):
    """The same target image made by the CPU oracle (its timing legs only)."""
    import oracle
    pr = oracle.project(scene, cam, 0)
    return oracle.render(oracle.visible(pr.tiles), pr, cam).img.astype(np.float32)


def run_workload(name, steps, warmup, overlap=True, packed=True, row_major=False, id_order="spatial"):
    """Build the workload, store its primitives in `id_order` ("spatial": the
    pool's Morton order; "given": the generator's order), make its inputs
    resident, and time `steps` training views (after `warmup` untimed ones that
    take the timed path exactly).  Returns the throughput, per-phase times and
    rooflines, and the trainer."""
    import torch
    from paper_2607_19893_amd import scenes
    from paper_2607_19893_amd.pipeline import ViewTrainer, to_u32
    t0 = time.time()
    w = scenes.workload(name)
    cams = w.cameras
    log("workload %s: n=%d, %d views, %dx%d (generated in %.1fs)" % (w.name, w.scene.n, len(cams), cams[0].width,
                                                                     cams[0].height, time.time() - t0))
    if id_order == "spatial":
        t0 = time.time()
        w = scenes.spatially_ordered(w)
        log("primitives stored in spatial (Morton) order (%.1fs)" % (time.time() - t0))
    tr = ViewTrainer(w.scene, capacity=1, max_width=max(c.width for c in cams),
                     max_height=max(c.height for c in cams), lr=w.lr, beta1=w.beta1, beta2=w.beta2, eps=w.eps,
                     packed=packed)
    tr.longest_first = not row_major
    need = tr.ensure_capacity(cams)
    log("pair capacity %d (max pairs over the views %d)" % (tr.capacity, need))
    t0 = time.time()
    targets = [torch.from_numpy(w.target(i, render=gpu_render).reshape(-1)).to(tr.dev) for i in range(len(cams))]
    _RENDERERS.clear()
    log("targets resident (%.1fs)" % (time.time() - t0))

    # pair statistics per view (untimed): evaluated / included (pixel, pair) counts
    ev_pairs, inc_pairs, vis_counts, pair_counts, w_iters, w_hits = [], [], [], [], [], []
    front = [in_front(w.scene.mean, c) for c in cams]
    for c in cams:
        tr.project(c); tr.visible(); tr.bin_sort()
        tr.pair_stats.zero_()
        tr.raster_fwd(active=False, stats=True)
        torch.cuda.synchronize()
        st = tr.pair_stats.cpu().numpy()
        ev_pairs.append(int(st[0])); inc_pairs.append(int(st[1]))
        w_iters.append(int(st[2])); w_hits.append(int(st[3]))
        vis_counts.append(int(to_u32(tr.counts[0:1])[0])); pair_counts.append(int(to_u32(tr.counts[1:2])[0]))

    step = 0
    nviews = len(cams)
    nph = len(ViewTrainer.PHASES)
    nev = nph + (2 if overlap else 1)
    # the warm-up takes the timed path exactly, timing events included: the
    # runtime's first use of timing events on the two streams costs a one-time
    # stall of tens of milliseconds in a launch, which must not land in the
    # timed region
    wevs = [[torch.cuda.Event(enable_timing=True) for _ in range(nev)] for _ in range(warmup)]
    for k in range(warmup):
        step += 1
        tr.step(cams[k % nviews], step, version=step, target=targets[k % nviews], events=wevs[k], overlap=overlap)
    tr.flush_apply()
    torch.cuda.synchronize()
    assert to_u32(tr.status)[0] == 0, "device status flags set during warm-up"

    # per-phase times (untimed pass): every phase bracketed by events.  Each
    # recorded event is a marker the device processes between two kernels
    # (about 5 us each on this path, nine a view), so the timed region below
    # brackets only the phase whose rate the roofline reports
    pevs = [[torch.cuda.Event(enable_timing=True) for _ in range(nev)] for _ in range(steps)]
    pviews = []
    torch.cuda.synchronize()
    no_collector()
    for k in range(steps):
        step += 1
        v = (warmup + k) % nviews
        pviews.append(v)
        tr.step(cams[v], step, version=step, target=targets[v], events=pevs[k], overlap=overlap)
    tr.flush_apply()
    torch.cuda.synchronize()
    gc.enable()
    assert to_u32(tr.status)[0] == 0, "device status flags set during the per-phase pass"
    phase_ms = np.zeros(nph)
    for k in range(steps):
        for p in range(nph):
            if p == nph - 1 and overlap:
                phase_ms[p] += pevs[k][-2].elapsed_time(pevs[k][-1])    # the apply, on its own stream
            else:
                phase_ms[p] += pevs[k][p].elapsed_time(pevs[k][p + 1])
    phase_ms /= steps
    log("%s per-phase ms: " % w.name + ", ".join("%s %.3f" % (n, t) for n, t in zip(ViewTrainer.PHASES, phase_ms)))
    names = list(ViewTrainer.PHASES)
    # the dominant kernel of the step: the longest phase on the step's stream (an
    # overlapped apply runs on the second stream, beside the next view's phases)
    on_path = [n for n in names if n != "apply" or not overlap]
    dom = max(on_path, key=lambda n: phase_ms[names.index(n)])
    pd = names.index(dom)

    # the timed region: `steps` views, only the dominant phase bracketed by events
    evs = []
    for _ in range(steps):
        e = [None] * nev
        e[pd] = torch.cuda.Event(enable_timing=True)
        e[pd + 1] = torch.cuda.Event(enable_timing=True)
        evs.append(e)
    views = []
    torch.cuda.synchronize()
    no_collector()
    t_start = time.perf_counter()
    for k in range(steps):
        step += 1
        v = (warmup + steps + k) % nviews
        views.append(v)
        tr.step(cams[v], step, version=step, target=targets[v], events=evs[k], overlap=overlap)
    tr.flush_apply()
    t_issued = time.perf_counter()
    torch.cuda.synchronize()
    t_end = time.perf_counter()
    gc.enable()
    wall = t_end - t_start
    log("%s: host issue time %.3f ms per step (device %.3f ms per step)"
        % (w.name, 1e3 * (t_issued - t_start) / steps, 1e3 * wall / steps))
    assert to_u32(tr.status)[0] == 0, "device status flags set during the timed steps"
    dom_ms = float(np.mean([evs[k][pd].elapsed_time(evs[k][pd + 1]) for k in range(steps)]))
    log("%s: dominant phase %s %.4f ms in the timed region" % (w.name, dom, dom_ms))

    def mean_work(vs):
        return phase_work(tr, w.scene.n, float(np.mean([front[v] for v in vs])),
                          float(np.mean([vis_counts[v] for v in vs])), float(np.mean([pair_counts[v] for v in vs])),
                          float(np.mean([ev_pairs[v] for v in vs])), float(np.mean([inc_pairs[v] for v in vs])),
                          cams[0].num_tiles)

    ev_mean = float(np.mean([ev_pairs[v] for v in views]))
    inc_mean = float(np.mean([inc_pairs[v] for v in views]))
    V_mean = float(np.mean([vis_counts[v] for v in views]))
    M_mean = float(np.mean([pair_counts[v] for v in views]))
    proofs = mean_work(pviews)
    per_phase = {}
    for name, t in zip(names, phase_ms):
        bound, work, peak, unit = proofs[name]
        ach = work / (t * 1e-3)
        per_phase[name] = {"ms": round(float(t), 4), "bound": bound, "achieved": round(ach, 2), "peak": peak,
                           "unit": unit, "frac": round(ach / peak, 4)}
    # the roofline of the dominant kernel: its work over the timed views and its
    # event time inside the timed region
    bound, work, peak, unit = mean_work(views)[dom]
    ach = work / (dom_ms * 1e-3)
    tb = traffic_bytes(w.name, dom, id_order)
    roofline = {"kernel": dom, "bound": bound, "achieved": round(ach, 3), "peak": peak, "unit": unit,
                "frac": round(ach / peak, 5), "traffic": round(tb) if tb is not None else None,
                "ms": round(dom_ms, 4)}
    log("%s phase rooflines: " % w.name + json.dumps(per_phase))
    wi_mean = float(np.mean([w_iters[v] for v in views]))
    wh_mean = float(np.mean([w_hits[v] for v in views]))
    log("%s mean per view: V=%.0f M=%.0f evaluated=%.3g included=%.3g; forward (pixel row, pair) steps %.3g, "
        "with an included pixel %.3g (%.1f%%), included lanes per such step %.1f of 16"
        % (w.name, V_mean, M_mean, ev_mean, inc_mean, wi_mean, wh_mean, 100 * wh_mean / max(wi_mean, 1),
           inc_mean / max(wh_mean, 1)))
    return {"w": w, "tr": tr, "cams": cams, "targets": targets, "step": step, "id_order": id_order,
            "views_per_s": round(steps / wall, 3), "ms_per_step": round(1e3 * wall / steps, 4), "steps": steps,
            "views": nviews, "mean_visible": round(V_mean), "mean_pairs": round(M_mean), "roofline": roofline,
            "phases_ms": {k: v["ms"] for k, v in per_phase.items()},
            "phases_frac": {k: v["frac"] for k, v in per_phase.items()}}


def phase_work(tr, N, F_mean, V_mean, M_mean, ev_mean, inc_mean, T_tiles):
    """Algorithmic work of each phase per view: (bound, work in GB or TFLOP, peak, unit)."""
    row_bytes = 4 * tr.row_len
    fwd_flops = FWD_FLOP_EVAL * ev_mean + FWD_FLOP_INC * inc_mean
    bwd_flops = BWD_FLOP_EVAL * ev_mean + BWD_FLOP_INC * inc_mean
    # projection: means of every primitive; log-scale, quaternion of those in
    # front of the near plane; opacity + colour coefficients of the visible
    # ones; radius + tile count of every primitive; the 2D record of the visible
    proj_bytes = 12 * N + 28 * F_mean + 4 * (tr.row_len - 10) * V_mean + 8 * N + 40 * V_mean
    # visible set: the per-primitive predicate read, the ids written
    vis_bytes = 4 * N + 4 * V_mean
    # binning as a 64-bit (tile, depth) key sort: duplication (16 B per visible
    # primitive, 12 B per pair), LSD radix passes of 24 B per pair each (key +
    # value, read + write), one per 11 bits of the 31 depth + ceil(log2 T) tile
    # bits, and the range extraction (8 B per pair)
    key_bits = 31 + int(np.ceil(np.log2(max(T_tiles, 2))))
    sort_bytes = 16 * V_mean + 12 * M_mean + 24 * M_mean * int(np.ceil(key_bits / 11)) + 8 * M_mean
    # per-primitive backward: the 48-byte pair slots, then per visible row the
    # parameters read (4P), the 2D record and id (68 B) and the gradient row written (4P)
    pbwd_bytes = 48 * M_mean + V_mean * (2 * row_bytes + 68)
    # Adam + staging per visible row: p, g, m, v read and p, m, v written (7 row
    # reads/writes), the message row and id written, the id read
    adam_bytes = V_mean * (8 * row_bytes + 8)
    # commit per row: message row + id read, replica row read and written, published version read and written
    apply_bytes = V_mean * (3 * row_bytes + 12)
    hbm = lambda b: ("hbm", b / 1e9, HBM_PEAK_GBS, "GB/s")
    return {
        "project": hbm(proj_bytes),
        "visible": hbm(vis_bytes),
        "bin_sort": hbm(sort_bytes),
        "raster_fwd_l1": ("alu", fwd_flops / 1e12, FP32_PEAK_TFLOPS, "TFLOP/s"),
        "raster_bwd_pixels": ("alu", bwd_flops / 1e12, FP32_PEAK_TFLOPS, "TFLOP/s"),
        "raster_bwd_project": hbm(pbwd_bytes),
        "adam_publish": hbm(adam_bytes),
        "apply": hbm(apply_bytes),
    }


def bench_delta(tr, cams, reps=20):
    """The publication kernels alone, each launched on all compute units on the
    current stream: gs_delta_pack of the visible rows' parameters into a
    message, gs_delta_apply (ADD) of that message into the replica, and the
    versioned ring commit (gs_publish_commit, foreground) of an Adam message.
    Rows are those of view 0's visible set.  Each launch is timed cold, with
    HIP events around it alone: a 1 GiB fill before it evicts the L2 and the
    256 MB Infinity Cache, so no launch reads what the previous one left
    there; the mean over `reps` launches is reported."""
    import torch
    from paper_2607_19893_amd import gsmi
    from paper_2607_19893_amd.pipeline import to_u32
    tr.project(cams[0]); tr.visible()
    torch.cuda.synchronize()
    K = int(to_u32(tr.counts[0:1])[0])
    P4 = 4 * tr.row_len
    version = int(to_u32(tr.ring_state)[0])
    e = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    evict = torch.empty(1 << 28, dtype=torch.float32, device=tr.dev)

    def timed(fn, before=None):
        fn()                                   # warm-up launch
        torch.cuda.synchronize()
        total = 0.0
        for _ in range(reps):
            if before is not None:
                before()
            evict.fill_(1.0)
            e[0].record()
            fn()
            e[1].record()
            torch.cuda.synchronize()
            total += e[0].elapsed_time(e[1])
        return total / reps

    out = {"rows": K, "row_bytes": P4}
    # pack: ids read, rows gathered, message (ids + rows) written
    ms = timed(lambda: tr.pack_params(version))
    b = 2.0 * K * (4 + P4)
    out["pack"] = {"ms": round(ms, 4), "gbs": round(b / ms / 1e6, 1), "frac": round(b / ms / 1e6 / HBM_PEAK_GBS, 4)}
    # apply (ADD, version stamp): message read, replica rows read and written, versions written
    ms = timed(lambda: tr.apply(gsmi.GS_APPLY_ADD))
    b = K * (4 + P4) + 2.0 * K * P4 + 4 * K
    out["apply"] = {"ms": round(ms, 4), "gbs": round(b / ms / 1e6, 1), "frac": round(b / ms / 1e6 / HBM_PEAK_GBS, 4)}
    # the versioned commit: stage one Adam message per version, commit it
    # (foreground, all CUs); the staging is outside the timed launches
    ver = [version]

    def stage():
        ver[0] += 1
        tr.adam_publish(ver[0], ver[0], tr.msgs[ver[0] & 1])

    def commit():
        tr.commit(ver[0], background=False)

    stage()
    ms = timed(commit, before=stage)
    b = K * (4 + P4) + 2.0 * K * P4 + 8 * K
    out["commit"] = {"ms": round(ms, 4), "gbs": round(b / ms / 1e6, 1), "frac": round(b / ms / 1e6 / HBM_PEAK_GBS, 4)}
    assert to_u32(tr.status)[0] == 0, "device status flags set by the publication kernels"
    # for comparison: a library row gather of the same rows (torch.index_select of K rows of a
    # row_len-float table by the same ascending ids), the access pattern with no arithmetic
    table = torch.zeros(tr.n, tr.row_len, device=tr.dev)
    ids = tr.vis_idx[:K].to(torch.int64)
    dst = torch.empty(K, tr.row_len, device=tr.dev)
    ms = timed(lambda: torch.index_select(table, 0, ids, out=dst))
    b = 2.0 * K * P4 + 8 * K
    out["row_gather_probe"] = {"ms": round(ms, 4), "gbs": round(b / ms / 1e6, 1),
                               "frac": round(b / ms / 1e6 / HBM_PEAK_GBS, 4)}
    del table, ids, dst
    return out


# the oracle's view sample per workload: every view of the two small
# workloads, the first two and the last of the others
ORACLE_STAGE_VIEWS = {"tiny": "all", "ring": "all", "room": (0, 1, -1), "spiral": (0, 1, -1), "aerial": (0, 1, -1)}


def oracle_stage_times():
    """Per-stage wall time of the CPU oracle (as it stands) on each workload's view sample."""
    import oracle
    from paper_2607_19893_amd import scenes
    out = {}
    for name, sel in ORACLE_STAGE_VIEWS.items():
        w = scenes.workload(name)
        views = list(range(len(w.cameras))) if sel == "all" else [v % len(w.cameras) for v in sel]
        m = [np.zeros_like(a) for _, a in w.scene.groups()]
        v = [np.zeros_like(a) for _, a in w.scene.groups()]
        tot = {}
        targets = {i: w.target(i, render=oracle_render) for i in views}    # inputs, outside the timing
        t0 = time.perf_counter()
        for k, i in enumerate(views):
            r = oracle.train_view(w.scene, w.cameras[i], targets[i], m, v, k + 1, lr=w.lr)
            for st, t in r.times.items():
                tot[st] = tot.get(st, 0.0) + t
        dt = time.perf_counter() - t0
        out[w.name] = {"views": views, "s_per_view": {k: round(t / len(views), 4) for k, t in tot.items()},
                       "views_per_s": round(len(views) / dt, 4), "threads": oracle.num_threads()}
        log("oracle %s: %s" % (w.name, out[w.name]))
    return out


def bench_scope_gate(tr, cams, targets, steps):
    """Hazard sets and throughput-first admission between consecutive views
    A -> B of the workload: read scope = projection-visible set, update scope =
    realized active set, evidence = the backward's |dL/d(u,v)| of A (tau 0.2).
    Scopes and evidence are prepared untimed; the timed part is one
    gs_scope_conflicts (bitmaps and id lists out) and one gs_admission_gate per
    transition, on the current stream."""
    import torch
    from paper_2607_19893_amd import gsmi
    n = tr.n
    words = gsmi.scope_words(n)
    nv = len(cams)
    R = torch.zeros(nv, max(1, words), dtype=torch.int32, device=tr.dev)
    Wr = torch.zeros_like(R)
    G = torch.zeros(nv, max(1, n), device=tr.dev)
    for i, c in enumerate(cams):
        tr.project(c); tr.visible(); tr.bin_sort(); tr.raster_fwd(active=True); tr.loss_l1(targets[i])
        tr.raster_bwd(grad2d=False)
        gsmi.gs_scope_from_pred(gsmi.GS_PRED_U32_NONZERO, tr.tiles, n, 0, R[i])
        gsmi.gs_scope_from_pred(gsmi.GS_PRED_U8_NONZERO, tr.active, n, 0, Wr[i])
        G[i].copy_(tr.grad_norm)
    out_bm = [torch.zeros(max(1, words), dtype=torch.int32, device=tr.dev) for _ in range(3)]
    out_id = [torch.zeros(max(1, n), dtype=torch.int32, device=tr.dev) for _ in range(3)]
    counts = torch.zeros(4, dtype=torch.int32, device=tr.dev)
    res = torch.zeros(16, dtype=torch.int32, device=tr.dev)
    ws = torch.zeros(gsmi.gs_workspace_bytes(gsmi.GS_WS_SCOPE, n), dtype=torch.uint8, device=tr.dev)
    args_ = [gsmi.make_gate_args(Wr[i], G[i], 0.2, evidence=R[i]) for i in range(nv)]
    torch.cuda.synchronize()
    e0, e1, e2 = (torch.cuda.Event(enable_timing=True) for _ in range(3))
    t_conf = t_gate = 0.0
    hz = np.zeros(4)
    reasons = {}
    moved = 0.0
    no_collector()
    for k in range(steps):
        a, b = k % nv, (k + 1) % nv
        e0.record()
        gsmi.gs_scope_conflicts(R[a], Wr[a], R[b], Wr[b], n, out_bm[0], out_bm[1], out_bm[2], out_id[0], out_id[1],
                                out_id[2], counts, ws)
        e1.record()
        gsmi.gs_admission_gate(R[b], out_bm[1], args_[a], n, res, ws)
        e2.record()
        torch.cuda.synchronize()
        t_conf += e0.elapsed_time(e1)
        t_gate += e1.elapsed_time(e2)
        c = counts.cpu().numpy().view(np.uint32).astype(np.float64)
        hz += c
        r = gsmi.gate_result_from(res)
        reasons[r.reason] = reasons.get(r.reason, 0) + 1
        # bytes: conflicts read 4 scopes and write 3 bitmaps and the id lists;
        # the gate reads 4 scopes and ||g_A|| at C_A and D+
        moved += 7 * words * 4 + 4 * float(c[:3].sum()) + 4 * words * 4 + 4 * (r.n_active + r.n_delayed)
    gc.enable()
    t_conf /= steps
    t_gate /= steps
    hz /= steps
    ms = t_conf + t_gate
    gbs = moved / steps / (ms * 1e-3) / 1e9
    return {"transitions": steps, "ms_conflicts": round(t_conf, 4), "ms_gate": round(t_gate, 4),
            "mean_waw": round(hz[0]), "mean_raw": round(hz[1]), "mean_war": round(hz[2]), "mean_read": round(hz[3]),
            "gate_reasons": {str(k): v for k, v in sorted(reasons.items())}, "hbm_gbs": round(gbs, 1),
            "hbm_frac": round(gbs / HBM_PEAK_GBS, 4)}


def bench_unit(tr, cams, targets, steps, step0):
    """Task units of two consecutive views (gradients summed over the union of
    their visible sets, one sparse Adam + staging + commit per unit), timed
    over `steps` views on one stream."""
    import torch
    nv = len(cams)
    units = max(1, steps // 2)
    version = int(tr.ring_state.cpu().numpy().view(np.uint32)[0])
    step = step0
    for u in range(2):                                   # warm-up
        step += 1; version += 1
        v = (2 * u) % nv
        tr.step_unit([cams[v], cams[(v + 1) % nv]], step, version, [targets[v], targets[(v + 1) % nv]])
    torch.cuda.synchronize()
    no_collector()
    t0 = time.perf_counter()
    for u in range(units):
        step += 1; version += 1
        v = (2 * u) % nv
        tr.step_unit([cams[v], cams[(v + 1) % nv]], step, version, [targets[v], targets[(v + 1) % nv]])
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    gc.enable()
    from paper_2607_19893_amd.pipeline import to_u32
    assert to_u32(tr.status)[0] == 0, "device status flags set during the task units"
    return {"units": units, "views_per_unit": 2, "views_per_s": round(2 * units / dt, 2),
            "ms_per_unit": round(1e3 * dt / units, 4)}


# the planner's settings: outlier cap, neighbours kept per view, logical
# regions, task-unit size (K = 4 and two views per unit are the paper's
# defaults; the cap and top-k are this build's choice)
PLAN = {"track_cap": 64, "top_k": 16, "K": 4, "unit_size": 2, "max_iters": 20}
PLAN_SIZES = (1000, 2000, 5000, 10000, 20000, 50000)   # image counts the paper times its planner at
PLAN_ORACLE_VIEWS = 1000


def bench_planner():
    """Wall time of the native planner (graph, partition, schedule) on
    synthetic aerial captures of each size, host arrays resident."""
    from paper_2607_19893_amd import gsmi, scenes
    out = {"settings": PLAN, "threads": os.cpu_count(), "sizes": {}}
    for n in PLAN_SIZES:
        c = scenes.capture_tracks(n, seed=5)
        t0 = time.perf_counter()
        G = gsmi.gs_rlg_build(c.item_ptr, c.item_tracks, c.n_tracks, PLAN["track_cap"], PLAN["top_k"])
        t1 = time.perf_counter()
        group, C, rounds = gsmi.gs_lp_partition(c.position, G, PLAN["K"], PLAN["max_iters"])
        t2 = time.perf_counter()
        cycle, order, ug, tr = gsmi.gs_sds_order(group, C, G, PLAN["unit_size"])
        t3 = time.perf_counter()
        out["sizes"][str(n)] = {"observations": int(c.item_ptr[-1]), "edges": int(G.edge_dst.size),
                                "rounds": rounds, "s_graph": round(t1 - t0, 4), "s_partition": round(t2 - t1, 4),
                                "s_schedule": round(t3 - t2, 4), "s_total": round(t3 - t0, 4),
                                "zero_transitions": round(float(np.mean(tr[1:] == 0.0)), 4)}
        log("planner %d views: %s" % (n, out["sizes"][str(n)]))
    return out


def planner_oracle_time(n):
    """The oracle planner on the same kind of capture (one size), for comparison."""
    import oracle
    from paper_2607_19893_amd import scenes
    c = scenes.capture_tracks(n, seed=5)
    t0 = time.perf_counter()
    R = oracle.rlg_build([c.tracks_of(i) for i in range(c.n)], c.n_tracks, PLAN["track_cap"], PLAN["top_k"])
    P = oracle.lp_partition(c.position, R, PLAN["K"], PLAN["max_iters"])
    oracle.sds_order(P.group, P.coupling, PLAN["K"], R, PLAN["unit_size"])
    return {"views": n, "s_total": round(time.perf_counter() - t0, 3)}


def in_front(mean, cam):
    """Primitives whose camera-space depth lies beyond the near plane (the ones projection reads further)."""
    R = np.asarray(cam.R, np.float64).reshape(3, 3)
    z = mean.astype(np.float64) @ R[2] + float(cam.t[2])
    return int(np.count_nonzero(z > cam.near_z))


def copy_probe(mib):
    """A plain elementwise copy of known size: reads and writes `mib` MiB per launch."""
    import torch
    n = mib * (1 << 20) // 4
    a = torch.ones(n, dtype=torch.float32, device="cuda")
    b = torch.empty_like(a)
    for _ in range(4):
        torch.neg(a, out=b)
    torch.cuda.synchronize()
    print(json.dumps({"copy_probe_bytes_read": 4 * n, "copy_probe_bytes_written": 4 * n, "launches": 4}), flush=True)


def cpu_baseline(w, nviews):
    """The CPU oracle, as it stands, on `nviews` full views of the same workload."""
    import oracle
    targets = [w.target(i, render=oracle_render) for i in range(nviews)]    # inputs, outside the timing
    t0 = time.perf_counter()
    done = 0
    m = [np.zeros_like(a) for _, a in w.scene.groups()]
    v = [np.zeros_like(a) for _, a in w.scene.groups()]
    for i in range(nviews):
        cam = w.cameras[i % len(w.cameras)]
        oracle.train_view(w.scene, cam, targets[i], m, v, i + 1, lr=w.lr, with_pairs=False)
        done += 1
    dt = time.perf_counter() - t0
    return {"value": round(done / dt, 4), "unit": "views/s", "cores": oracle.num_threads(), "kind": "oracle",
            "sample": "%d full views (%s, %dx%d) through the oracle's projection, per-pixel render, L1, exact "
                      "backward, Adam and pack; %.1f s" % (done, w.name, w.cameras[0].width,
                                                            w.cameras[0].height, dt)}


if __name__ == "__main__":
    main()
