"""Benchmark: relation-set following forward + backward on one MI355X.

One step = kb_follow (forward, Eq. 4) + kb_follow_backward (dX and dR) over
the whole KB for one minibatch, inputs already resident in HBM.  The default
workload is the large KB: 10 M entities, 600 relations, 50 M distinct triples
with Zipf subject/object/relation marginals, b = 32, 1 %-dense X.

Prints one JSON line with the whole-step throughput (triple-batch products per
second, N_T * b / step time), a roofline entry for the dominant kernel (the
kernel with the largest share of the step's GPU time, its launches timed with
HIP events inside the timed region), the CPU oracle timed on the same
workload, and the largest deviation of the GPU's outputs from the oracle's.

Other modes: ``--workload chain3`` (the three-hop chain of the multi-hop
model, forward + loss + backward per step), ``--grid N`` (the relation sweep
of the grid scalability experiment), ``--oracle-table`` (the oracle alone,
per workload and thread count), ``--copy-calibration`` (a plain copy kernel
for scaling rocprofv3's byte counters).
"""
from __future__ import annotations

import argparse
import glob
import json
import os
import platform
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "triple·batch products/sec for kb_follow fwd+bwd; achieved HBM GB/s vs peak"
PEAK_HBM_GBPS = 8000.0
PASSES = ("fwd", "dx", "dr")  # forward (rows = objects), dX (subjects), dR (relations)


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor() or platform.machine()


def host_threads(cap=16):
    """Host cores this process may use (its affinity mask), at most `cap`."""
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    return max(1, min(n, cap))


# ---------------------------------------------------------------------------
# byte models
# ---------------------------------------------------------------------------

_DISTINCT = {}


def distinct_ids(kb):
    """Number of distinct subjects and of distinct objects of the KB."""
    key = id(kb)
    if key not in _DISTINCT:
        _DISTINCT[key] = (len(np.unique(kb.subj)), len(np.unique(kb.obj)))
    return _DISTINCT[key]


def pass_bytes(kb, b, p, whole_pass=False):
    """Algorithmic bytes of one pass's stream-kernel launch (or, with
    whole_pass, of the whole pass: every output row, as the stream kernel and
    the empty-row fill write them together), hard KB, under three models;
    every model has the index stream (8 B per triple), the row boundaries and
    the B table read once:
      array_once  each gathered array read once in full (the compulsory
                  model of the method: X, or dY, once; dY and X once for dR);
      distinct    each distinct gathered row once (rows no triple names are
                  never read);
      gather      every triple's b-wide rows come from memory.
    The stream kernel writes the output rows that have triples."""
    n_t, n_e, n_r = kb.n_triples, kb.n_entities, kb.n_relations
    idx = 8 * n_t
    n_subj, n_obj = distinct_ids(kb)
    if p in ("fwd", "dx"):
        n_a, n_out = (n_subj, n_obj) if p == "fwd" else (n_obj, n_subj)
        out = 4 * b * (n_e if whole_pass else n_out)
        base = idx + 4 * (n_e + 1) + 4 * b * n_r + out
        return {"array_once": float(base + 4 * b * n_e), "distinct": float(base + 4 * b * n_a),
                "gather": float(base + 4 * b * n_t)}
    base = idx + 4 * (n_r + 1) + 4 * b * n_r
    return {"array_once": float(base + 8 * b * n_e),
            "distinct": float(base + 4 * b * (n_subj + n_obj)),
            "gather": float(base + 8 * b * n_t)}


# ---------------------------------------------------------------------------
# kernel names, fingerprints and the committed rocprofv3 counters
# ---------------------------------------------------------------------------

def mangled_name(short):
    """Itanium-mangled symbol of a kernel named as profilers print it
    ("stream_kernel<4, 8, true, false, false, true>")."""
    m = re.fullmatch(r"(\w+)<([^>]*)>", short.strip())
    if not m:
        return None
    name, args = m.group(1), [a.strip() for a in m.group(2).split(",")]
    enc = "".join(f"Lb{1 if a == 'true' else 0}E" if a in ("true", "false") else f"Li{a}E"
                  for a in args)
    params = {"stream_kernel": "NS_10StreamArgsE", "tail_kernel": "NS_8TailArgsE",
              "combine_kernel": "PK15HIP_vector_typeIiLj4EElPdliPflPKff"}.get(name)
    if params is None:
        return None
    return f"_ZN3kbf12_GLOBAL__N_1{len(name)}{name}I{enc}EEv{params}"


def kernel_digest(short):
    """sha256 of the built kernel's gfx950 assembly (as the build records it)."""
    path = os.path.join(ROOT, "paper_2002_06115_amd", "_lib", "kernels.fingerprint")
    try:
        return json.load(open(path)).get(mangled_name(short) or "")
    except (OSError, ValueError):
        return None


def measured_traffic(workload, b, short, phases):
    """Bytes per launch of kernel `short` from the committed rocprofv3
    counters (FETCH_SIZE and WRITE_SIZE, copy-calibrated) when they were taken
    on the device code built now (same assembly digest) for this workload and
    batch: the mean over the launches of `phases`.  Returns (bytes, source)
    or (None, reason)."""
    digest = kernel_digest(short)
    if not digest:
        return None, "no fingerprint for the built kernel"
    for path in sorted(glob.glob(os.path.join(ROOT, "profiles", "*.json"))):
        try:
            prof = json.load(open(path))
        except (OSError, ValueError):
            continue
        if prof.get("workload") != workload or prof.get("batch") != b:
            continue
        per = prof.get("per_launch", {})
        kern = prof.get("kernels", {})
        vals = []
        for ph in phases:
            k = kern.get(ph, {})
            if k.get("kernel") == short and k.get("kernel_sha") == digest and ph in per:
                vals.append(float(per[ph]["bytes"]))
        if vals and len(vals) == len(phases):
            return float(np.mean(vals)), \
                f"{os.path.relpath(path, ROOT)} (fingerprint-matched; FETCH_SIZE and WRITE_SIZE " \
                f"per dispatch, copy-calibrated)"
    return None, "no committed counters for the device code built now"


# ---------------------------------------------------------------------------
# the oracle on the host
# ---------------------------------------------------------------------------

def oracle_pass_times(kb, X_bm, R_bm, dY_bm, threads, runs):
    """Median seconds of the oracle's forward, dX and dR (each alone) over
    `runs` runs on `threads` threads, all batch columns, plus the outputs of
    the last run."""
    import oracle
    args = (kb.subj, kb.rel, kb.obj, kb.n_entities, kb.n_relations)
    t = {"fwd": [], "dx": [], "dr": []}
    out = {}
    for _ in range(runs):
        t0 = time.perf_counter()
        out["Y"] = oracle.follow(*args, X_bm, R_bm, nthreads=threads)
        t1 = time.perf_counter()
        out["dX"], _ = oracle.follow_backward(*args, X_bm, R_bm, dY_bm, want_dr=False,
                                              nthreads=threads)
        t2 = time.perf_counter()
        _, out["dR"] = oracle.follow_backward(*args, X_bm, R_bm, dY_bm, want_dx=False,
                                              nthreads=threads)
        t3 = time.perf_counter()
        t["fwd"].append(t1 - t0)
        t["dx"].append(t2 - t1)
        t["dr"].append(t3 - t2)
        log(f"[oracle] {kb.n_triples} triples, {X_bm.shape[0]} columns, {threads} threads: "
            f"fwd {t1 - t0:.3f} s, dX {t2 - t1:.3f} s, dR {t3 - t2:.3f} s")
    med = {k: float(np.median(v)) for k, v in t.items()}
    return med, out


def tolerance_ratio(got, want, atol=1e-7, rtol=1e-5, block=1 << 24):
    """max over elements of |got - want| / (atol + rtol |want|), in blocks."""
    g, w = got.reshape(-1), want.reshape(-1)
    worst = 0.0
    for i in range(0, g.size, block):
        gi = g[i:i + block].astype(np.float64)
        wi = w[i:i + block].astype(np.float64)
        if gi.size:
            worst = max(worst, float((np.abs(gi - wi) / (atol + rtol * np.abs(wi))).max()))
    return worst


# ---------------------------------------------------------------------------
# GPU timing helpers
# ---------------------------------------------------------------------------

def percentiles(v):
    q = np.percentile(np.asarray(v, dtype=np.float64), [10, 50, 90])
    return {"p10": round(float(q[0]), 4), "p50": round(float(q[1]), 4), "p90": round(float(q[2]), 4)}


def timing_detail(torch, fwd, bwd, stream, iters, flush=None):
    """Per-iteration HIP-event times of the forward and the backward (ms),
    as p10 / median / p90.  With `flush` (a 1 GiB device buffer, larger than
    the 256 MB last-level cache) the buffer is overwritten before every
    iteration, so each one starts with cold caches."""
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(iters)]
    for i in range(iters):
        if flush is not None:
            flush.fill_(float(i))
        ev[i][0].record(stream)
        fwd()
        ev[i][1].record(stream)
        bwd()
        ev[i][2].record(stream)
    torch.cuda.synchronize()
    f = [e[0].elapsed_time(e[1]) for e in ev]
    g = [e[1].elapsed_time(e[2]) for e in ev]
    return {"iters": iters, "fwd_ms": percentiles(f), "bwd_ms": percentiles(g),
            "fwd_bwd_ms": percentiles([a + c for a, c in zip(f, g)])}


def graph_step_ms(torch, step, iters):
    """Mean time of one step replayed from a captured HIP graph (the same
    launches as the eager step, without host launch overhead)."""
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()
    torch.cuda.current_stream().wait_stream(side)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    g.replay()
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    t0.record()
    for _ in range(iters):
        g.replay()
    t1.record()
    torch.cuda.synchronize()
    del g
    return round(t0.elapsed_time(t1) / iters, 4)


def device_stream_rates(torch, reps=10):
    """The device's streaming rates on a 2 GiB buffer, with torch's own
    elementwise kernels: a copy (GB/s read + written) and a fill (GB/s
    written)."""
    n = (2 << 30) // 4
    src = torch.ones(n, device="cuda")
    dst = torch.empty_like(src)
    torch.mul(src, 1.0, out=dst)
    dst.fill_(0.0)
    t = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
    t[0].record()
    for _ in range(reps):
        torch.mul(src, 1.0, out=dst)
    t[1].record()
    for _ in range(reps):
        dst.fill_(0.0)
    t[2].record()
    torch.cuda.synchronize()
    copy = 2 * 4 * n * reps / (t[0].elapsed_time(t[1]) * 1e-3) / 1e9
    fill = 4 * n * reps / (t[1].elapsed_time(t[2]) * 1e-3) / 1e9
    del src, dst
    return round(copy, 1), round(fill, 1)


def phase_groups(kernels, phases_ms):
    """Phases grouped by the kernel they launch: {kernel: [phases]} over the
    phases that ran (with launches)."""
    groups = {}
    for ph, name in kernels.items():
        if name and phases_ms.get(ph, (0.0, 0))[1] > 0:
            groups.setdefault(name, []).append(ph)
    return groups


def dominant_kernel(kernels, phases, concurrent=False):
    """(kernel, its phases, {kernel: ms per step}, why): the kernel with the
    largest share of the step's GPU time (sum of its launches' durations).
    Where that is not a stream kernel (small KBs, whose combine and empty-row
    launches take longer than their stream kernels) the stream kernel with the
    largest share is taken, since only the stream kernels have a byte model.
    With the concurrent backward, the dX and dR launches overlap and each one's
    duration includes the time it shares the GPU with the other; where the
    two largest shares are within 5 % of each other, the kernel that also runs
    a launch of its own (the forward) is taken, whose duration is its own."""
    groups = phase_groups(kernels, phases)
    share = {k: sum(phases[p][0] for p in ps) for k, ps in groups.items()}
    streams = [k for k, ps in groups.items() if all(p.endswith("_stream") for p in ps)]
    top = max(share, key=share.get)
    why = "largest share of the step's GPU time (sum of launch durations)"
    if top not in streams:
        top2 = max(streams, key=share.get)
        why = (f"the stream kernel with the largest share of the step's GPU time ({top}, a "
               f"combine / empty-row kernel, has more)")
        top = top2
    if concurrent:
        overlapped = lambda k: all(p.startswith(("dx_", "dr_")) for p in groups[k])
        rivals = [k for k in streams if k != top and share[k] >= 0.95 * share[top]
                  and not overlapped(k)]
        if overlapped(top) and rivals:
            top = max(rivals, key=share.get)
            why = ("within 5 % of the largest share of the step's GPU time, the stream kernel "
                   "with launches outside the concurrent backward (the largest share belongs "
                   "to a kernel whose launches all overlap another pass)")
    return top, groups[top], share, why


def timed_phases(dom_phases, concurrent):
    """The dominant kernel's phases whose launches the timed steps bracket.
    With the concurrent backward, event-bracketed dX launches (on the caller's
    stream, beside the dR pass) lengthened the large KB's step by 0.28 ms, so
    a kernel that also runs the forward is timed on its forward launches; dR's
    launches (on the KB's own stream) are bracketed without that cost."""
    if concurrent and len(dom_phases) > 1:
        kept = [p for p in dom_phases if not p.startswith("dx_")]
        if kept:
            return kept
    return list(dom_phases)


def roofline_entry(kb, w, b, kernels, phases, timed, ms_step, residual, concurrent=False):
    """The roofline of the dominant kernel: the one with the largest share of
    the step's GPU time (sum of its launches' durations).  achieved =
    algorithmic bytes of its launches (array-once model: each gathered array
    read once, every output row the kernel writes) / their duration, over the
    launches the timed steps bracketed (timed_phases)."""
    dom, dom_phases, share, choice = dominant_kernel(kernels, phases, concurrent)
    total = sum(share.values()) or 1.0
    t_phases = timed_phases(dom_phases, concurrent)
    ms_sum = sum(timed[p][0] for p in t_phases)
    launches = sum(timed[p][1] for p in t_phases)
    ms_avg = ms_sum / max(1, launches)
    models = [pass_bytes(kb, b, p.split("_")[0]) for p in t_phases]
    per_launch = {m: float(np.mean([x[m] for x in models])) for m in models[0]}
    sec = ms_avg * 1e-3
    ach = per_launch["array_once"] / sec / 1e9
    traffic, source = measured_traffic(w.name, b, dom, t_phases)
    roof = {"bound": "hbm", "achieved": round(ach, 1), "peak": PEAK_HBM_GBPS, "unit": "GB/s",
            "frac": round(ach / PEAK_HBM_GBPS, 4), "traffic": traffic,
            "traffic_source": source,
            "kernel": dom, "phases": dom_phases, "phases_timed": t_phases,
            "kernel_choice": choice,
            "gpu_time_share": round(share[dom] / total, 4),
            "kernel_ms": round(ms_avg, 4), "launches_timed": int(launches),
            "bytes_model": "array-once: 8 B of ids per triple, the row boundaries, each gathered "
                           "array read once in full, the B table once, every output row the "
                           "kernel writes once (hard KB)",
            "algorithmic_bytes": per_launch["array_once"],
            "distinct_rows_bytes": per_launch["distinct"],
            "distinct_rows_frac": round(per_launch["distinct"] / sec / 1e9 / PEAK_HBM_GBPS, 4),
            "gather_model_bytes": per_launch["gather"],
            "gather_model_GBps": round(per_launch["gather"] / sec / 1e9, 1)}
    # The other stream kernels, from the phase loop (every phase bracketed).
    others = []
    for k, ps in phase_groups(kernels, phases).items():
        if k == dom or not all(p.endswith("_stream") for p in ps):
            continue
        ms_k = sum(phases[p][0] for p in ps) / max(1, sum(phases[p][1] for p in ps))
        by_k = float(np.mean([pass_bytes(kb, b, p.split("_")[0])["array_once"] for p in ps]))
        others.append({"kernel": k, "phases": ps, "gpu_time_share": round(share[k] / total, 4),
                       "kernel_ms_phase_loop": round(ms_k, 4),
                       "frac": round(by_k / (ms_k * 1e-3) / 1e9 / PEAK_HBM_GBPS, 4),
                       "overlaps_another_pass": concurrent and all(
                           p.startswith(("dx_", "dr_")) for p in ps)})
    roof["other_stream_kernels"] = others
    if traffic:
        roof["fabric_traffic_GBps"] = round(traffic / sec / 1e9, 1)
        roof["fabric_traffic_frac_upper_bound"] = round(traffic / sec / 1e9 / PEAK_HBM_GBPS, 4)
        roof["fabric_traffic_note"] = ("L2-to-fabric bytes: HBM plus Infinity Cache hits, and "
                                       "every re-read; an upper bound on HBM bytes, not useful "
                                       "bandwidth")
        roof["traffic_over_algorithmic"] = round(traffic / per_launch["array_once"], 3)
    # Every pass (stream kernel + its combine and empty-row launches) and the
    # whole step against the array-once bytes of whole passes.
    per_pass = {}
    for p in PASSES:
        ms = sum(phases[f"{p}_{s}"][0] for s in ("stream", "tail", "combine"))
        by = pass_bytes(kb, b, p, whole_pass=True)["array_once"]
        per_pass[p] = {"ms": round(ms, 4), "bytes": by,
                       "frac": round(by / (ms * 1e-3) / 1e9 / PEAK_HBM_GBPS, 4) if ms else None}
    step_bytes = sum(pass_bytes(kb, b, p, whole_pass=True)["array_once"] for p in PASSES)
    roof["per_pass"] = per_pass
    roof["step"] = {"ms": round(ms_step, 4), "array_once_bytes": step_bytes,
                    "array_once_frac": round(step_bytes / (ms_step * 1e-3) / 1e9 / PEAK_HBM_GBPS,
                                             4),
                    "target_frac": 0.6,
                    "note": "the fwd + dX + dR step against the array-once bytes of the three "
                            "passes; the >= 0.6 of HBM peak target on the 10 M-entity KB is "
                            "judged on this figure"}
    if residual is not None:
        roof["note"] = "byte models are those of the plain follow; the residual hop also reads " \
                       "one row of X (dY) per written row"
    return roof


# ---------------------------------------------------------------------------
# modes
# ---------------------------------------------------------------------------

def seeds_of(w, extra=None):
    import kbgen
    d = {"root": kbgen.ROOT_SEED, "workload_index": w.index, "scale_tag": w.scale_tag,
         "streams": {"triples": kbgen.ST_TRIPLES, "x": kbgen.ST_X, "r": kbgen.ST_R,
                     "dy": kbgen.ST_DY, "target": kbgen.ST_TARGET, "perm": kbgen.ST_PERM},
         "recipe": "numpy PCG64(SeedSequence([root, workload_index, stream, scale_tag, sub"
                   "(, example)]))"}
    if extra:
        d.update(extra)
    return d


def follow_bench(args, torch, kbgen, kbf):
    w = kbgen.WORKLOADS[args.workload]
    if args.batch:
        # The same KB; inputs are drawn per example, so the first columns
        # are those of the default width.
        import dataclasses
        w = dataclasses.replace(w, batch=int(args.batch))
    t0 = time.perf_counter()
    kb = kbgen.make_kb(w)
    X_bm, R_bm, dY_bm = kbgen.make_x(w), kbgen.make_r(w), kbgen.make_dy(w)
    stats = kb.stats()
    log(f"[bench] generated {w.label} in {time.perf_counter() - t0:.1f} s; stats {stats}")

    torch.cuda.set_device(0)
    # Stream kernels are timed by their dispatch timestamps, which match
    # rocprofv3's durations; on KBs under 2^20 triples those cost ~25 us per
    # bracketed launch (tiny KB: 0.109 against 0.048 ms per step), so there
    # the library times them with event records around the launch.
    # (The library reads the switch when the KB is created.)
    prev = os.environ.get("KBFOLLOW_STREAM_STAMPS")
    if kb.n_triples < (1 << 20) and prev is None:
        os.environ["KBFOLLOW_STREAM_STAMPS"] = "0"
    stamps = os.environ.get("KBFOLLOW_STREAM_STAMPS", "1") != "0"
    t0 = time.perf_counter()
    try:
        gkb = kbf.KB(kb.subj, kb.rel, kb.obj, w.n_entities, w.n_relations)
    finally:
        if prev is None:
            os.environ.pop("KBFOLLOW_STREAM_STAMPS", None)
    torch.cuda.synchronize()
    create_s = time.perf_counter() - t0
    log(f"[bench] kb_create {create_s:.1f} s, info {gkb.info()}")
    em = lambda a: torch.from_numpy(a).cuda().t().contiguous()
    X, R, dY = em(X_bm), em(R_bm), em(dY_bm)
    b = w.batch
    Y = torch.empty_like(X)
    dX = torch.empty_like(X)
    dR = torch.empty_like(R)
    stream = torch.cuda.current_stream()
    kernels = gkb.phase_kernels(b, residual=args.residual is not None)

    def step():
        gkb.follow(X, R, out=Y, stream=stream, residual=args.residual)
        gkb.follow_backward(X, R, dY, dX=dX, dR=dR, stream=stream, residual=args.residual)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    log(f"[bench] warmup {args.warmup} done")

    # Events around a phase cost a few microseconds of GPU time each, so the
    # per-phase breakdown comes from a loop of its own, and the timed steps
    # bracket only the launches of the dominant kernel.
    phases, dom_phases = {}, None
    if not args.no_profile:
        gkb.profile(True)
        for _ in range(args.steps):
            step()
        torch.cuda.synchronize()
        raw = gkb.profile_read()
        gkb.profile(False)
        phases = {k: (v[0] / args.steps, v[1] / args.steps) for k, v in raw.items()}
        dom_phases = dominant_kernel(kernels, phases, _overlap(kb.n_triples, b))[1]
        gkb.profile(True, phases=timed_phases(dom_phases, _overlap(kb.n_triples, b)))
    start = torch.cuda.Event(enable_timing=True)
    stop = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record(stream)
    for _ in range(args.steps):
        step()
    stop.record(stream)
    torch.cuda.synchronize()
    ms_total = start.elapsed_time(stop)
    timed = gkb.profile_read() if dom_phases else None
    gkb.profile(False)
    ms_step = ms_total / args.steps
    value = kb.n_triples * b / (ms_step * 1e-3)
    log(f"[bench] {args.steps} steps, {ms_step:.3f} ms/step, {value:.3e} triple*batch/s")

    detail = None
    iters = args.detail_iters
    if iters < 0:
        iters = {"tiny": 1000, "metaqa": 200}.get(w.name, 50)
    if iters > 0:
        fwd = lambda: gkb.follow(X, R, out=Y, stream=stream, residual=args.residual)
        bwd = lambda: gkb.follow_backward(X, R, dY, dX=dX, dR=dR, stream=stream,
                                          residual=args.residual)
        detail = {"warm": timing_detail(torch, fwd, bwd, stream, iters)}
        flush = torch.empty((1 << 30) // 4, device="cuda")
        detail["cold"] = timing_detail(torch, fwd, bwd, stream, iters, flush=flush)
        del flush
        detail["graph_ms_per_step"] = graph_step_ms(
            torch, lambda: (gkb.follow(X, R, out=Y, residual=args.residual),
                            gkb.follow_backward(X, R, dY, dX=dX, dR=dR, residual=args.residual)),
            iters)
        detail["copy_GBps"], detail["fill_GBps"] = device_stream_rates(torch)
        log(f"[bench] detail {json.dumps(detail)}")

    roof = roofline_entry(kb, w, b, kernels, phases, timed, ms_step, args.residual,
                          concurrent=_overlap(kb.n_triples, b)) if dom_phases else None
    if roof:
        roof["launch_timing"] = ("dispatch timestamps (hipExtLaunchKernel start / stop events)"
                                 if stamps else "event records around each launch")
    if roof and detail:
        roof["device_copy_GBps"] = detail["copy_GBps"]
        roof["achieved_frac_of_copy"] = round(roof["achieved"] / detail["copy_GBps"], 4)

    cpu, parity = None, None
    if not args.no_cpu_baseline:
        # The oracle on all b columns, median of 3 runs, on the host's cores;
        # its outputs also check every element of this run's GPU outputs.
        step()
        torch.cuda.synchronize()
        threads = host_threads(args.cpu_threads) if args.cpu_threads > 0 else host_threads()
        threads = min(threads, b)
        log(f"[bench] timing the CPU oracle on {b} batch columns, {threads} threads")
        gY, gdX, gdR = (t.t().contiguous().cpu().numpy() for t in (Y, dX, dR))
        if args.residual is None:
            med, out = oracle_pass_times(kb, X_bm, R_bm, dY_bm, threads, runs=3)
            dt = med["fwd"] + med["dx"] + med["dr"]
            cpu = {"value": kb.n_triples * b / dt, "unit": "triple·batch/s", "cores": threads,
                   "kind": "oracle",
                   "sample": (f"the whole workload: all {b} batch columns, forward "
                              f"{med['fwd']:.2f} s + dX {med['dx']:.2f} s + dR {med['dr']:.2f} s, "
                              f"median of 3 runs on {threads} threads ({cpu_model()}, "
                              f"{os.cpu_count()} logical CPUs)"),
                   "fwd_s": round(med["fwd"], 3), "dx_s": round(med["dx"], 3),
                   "dr_s": round(med["dr"], 3)}
            parity = {"compared": "every element of Y, dX and dR against the oracle "
                                  "(atol 1e-7, rtol 1e-5)",
                      "max_tol_ratio": {k: round(tolerance_ratio(g, out[k]), 6)
                                        for k, g in (("Y", gY), ("dX", gdX), ("dR", gdR))}}
            log(f"[bench] oracle {cpu['value']:.3e} triple*batch/s; parity {parity}")

    out = {
        "metric": METRIC,
        "value": value,
        "unit": "triple·batch/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32 in/out, f64 accumulate",
        "data": "synthetic",
        "config": {"workload": w.name, "n_entities": w.n_entities, "n_relations": w.n_relations,
                   "n_triples": kb.n_triples, "batch": b,
                   "laws": {"subj": w.subj_law, "obj": w.obj_law, "rel": w.rel_law},
                   "x": w.x_kind, "r": w.r_kind, "dy": w.dy_kind, "parallelism": "single GPU",
                   "op": "follow" if args.residual is None else f"follow + {args.residual} * X"},
        "seeds": seeds_of(w),
        "kb_sha256": kb.sha256(),
        "kb_stats": stats,
        "kernels": {k: v for k, v in kernels.items() if v},
        "phases_ms_per_step": {k: round(v[0], 4) for k, v in phases.items()},
        "concurrent_backward": _overlap(kb.n_triples, b),
        "phases_note": ("HIP-event times per phase from a separate loop of the same steps; the "
                        "timed steps bracket only the dominant kernel's launches with events; "
                        "with concurrent_backward the dx_* and dr_* phases run at the same "
                        "time, so their times overlap"),
        "kb_create_s": round(create_s, 2),
        "workspace_bytes": int(gkb.workspace_size(b)),
        "timing": detail,
        "roofline": roof,
        "cpu_baseline": cpu,
        "parity": parity,
    }
    print(json.dumps(out), flush=True)
    gkb.close()


def _overlap(n_triples, b):
    """Whether the library runs the backward's dR pass concurrently with dX
    (from 2^20 triples at b <= 32 unless KBFOLLOW_OVERLAP_BACKWARD says
    otherwise)."""
    env = os.environ.get("KBFOLLOW_OVERLAP_BACKWARD")
    if env:
        return env != "0"
    return n_triples >= (1 << 20) and b <= 32


def chain_bench(args, torch, kbgen, kbf):
    """The three-hop chain of the multi-hop model (Sec. 3.2) as one training
    step on the GPU: r^t = softmax(rho^t), x^t = L1-normalised follow(x^{t-1},
    r^t) for t = 1..3, softmax cross-entropy against the target set, and the
    full backward to x^0 and rho^1..rho^3 -- follow kernels and chain glue
    kernels only."""
    from paper_2002_06115_amd import chain
    w = kbgen.CHAIN3
    kb = kbgen.make_kb(w)
    x0, rho, tgt = kbgen.make_chain_inputs(w, kb)
    hops, b = len(rho), w.batch
    torch.cuda.set_device(0)
    gkb = kbf.KB(kb.subj, kb.rel, kb.obj, w.n_entities, w.n_relations)
    em = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda().t().contiguous()
    x0e, tgte = em(x0), em(tgt)
    rhoe = [em(r) for r in rho]
    kernels = gkb.phase_kernels(b)

    def step():
        xs, rs, sums = [x0e], [], []
        for t in range(hops):
            r = chain.softmax(rhoe[t])
            rs.append(r)
            x, s = chain.l1_normalize(gkb.follow(xs[-1], r))
            sums.append(s)
            xs.append(x)
        loss, _, dx = chain.softmax_xent(xs[-1], tgte)
        drho = [None] * hops
        for t in range(hops, 0, -1):
            du = chain.l1_normalize_backward(xs[t], sums[t - 1], dx)
            dx, dr = gkb.follow_backward(xs[t - 1], rs[t - 1], du)
            drho[t - 1] = chain.softmax_backward(rs[t - 1], dr)
        return loss, dx, drho

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    gkb.profile(True)
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    raw = gkb.profile_read()
    gkb.profile(False)
    phases = {k: (v[0] / args.steps, v[1] / args.steps) for k, v in raw.items()}
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    for _ in range(args.steps):
        res = step()
    stop.record()
    torch.cuda.synchronize()
    ms_step = start.elapsed_time(stop) / args.steps
    value = hops * kb.n_triples * b / (ms_step * 1e-3)
    loss_g, dx_g, drho_g = float(res[0]), res[1].t().contiguous().cpu().numpy(), \
        [d.t().contiguous().cpu().numpy() for d in res[2]]
    log(f"[chain3] {ms_step:.4f} ms/step, {value:.3e} triple*batch/s")

    # The same step captured into one HIP graph and replayed: no host work
    # between the ~40 launches.  Every replay must reproduce the eager
    # step's loss and gradients bit for bit.
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()
    torch.cuda.current_stream().wait_stream(side)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        gres = step()
    torch.cuda.synchronize()
    same = []
    for _ in range(3):
        g.replay()
        torch.cuda.synchronize()
        same.append(bool(torch.equal(gres[0], res[0]) and torch.equal(gres[1], res[1]) and
                         all(torch.equal(a, c) for a, c in zip(gres[2], res[2]))))
    t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0.record()
    for _ in range(args.steps):
        g.replay()
    t1.record()
    torch.cuda.synchronize()
    graph_ms = t0.elapsed_time(t1) / args.steps
    del g
    log(f"[chain3] graph replay {graph_ms:.4f} ms/step, bitwise equal to eager: {same}")
    # The step is ~40 short launches: the eager loop measures the host's
    # launch rate as much as the GPU.  The reported step is the graph replay
    # when every replay reproduced the eager step bit for bit.
    eager_ms = ms_step
    if all(same):
        ms_step, timed_as = graph_ms, "graph replay (every replay bitwise equal to the eager step)"
    else:
        timed_as = "eager (a graph replay differed from the eager step)"
    value = hops * kb.n_triples * b / (ms_step * 1e-3)

    cpu, parity = None, None
    if not args.no_cpu_baseline:
        from oracle import chain as ochain
        arrays = (kb.subj, kb.rel, kb.obj)
        runs = 20
        ts = []
        for _ in range(runs):
            t0 = time.perf_counter()
            loss_o, dx_o, drho_o = ochain.chain_grad(arrays, w.n_entities, w.n_relations, x0,
                                                     rho, tgt)
            ts.append(time.perf_counter() - t0)
        dt = float(np.median(ts))
        cpu = {"value": hops * kb.n_triples * b / dt, "unit": "triple·batch/s", "cores": 1,
               "kind": "oracle",
               "sample": (f"the whole step (3 hops forward in double, loss, backward), median of "
                          f"{runs} runs, {dt * 1e3:.1f} ms, one thread ({cpu_model()})")}
        parity = {"compared": "loss, every element of dx0 and of drho1..3 against the chain "
                              "oracle (atol 1e-7, rtol 1e-5)",
                  "loss_abs_diff": abs(loss_g - loss_o),
                  "max_tol_ratio": {"dx0": round(tolerance_ratio(dx_g, dx_o), 6),
                                    **{f"drho{t + 1}": round(tolerance_ratio(drho_g[t], drho_o[t]),
                                                             6) for t in range(hops)}}}
    groups = phase_groups(kernels, phases)
    share = {k: sum(phases[p][0] for p in ps) for k, ps in groups.items()}
    out = {
        "metric": METRIC, "value": value, "unit": "triple·batch/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms_step,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "f32 in/out, f64 accumulate", "data": "synthetic",
        "config": {"workload": w.name, "n_entities": w.n_entities,
                   "n_relations": w.n_relations, "n_triples": kb.n_triples, "batch": b,
                   "hops": hops, "parallelism": "single GPU",
                   "op": "3 x (softmax(rho), follow, L1 normalise), softmax cross-entropy, "
                         "backward to x0 and rho1..3",
                   "value_definition": "hops * N_T * b / step time"},
        "seeds": seeds_of(w), "kb_sha256": kb.sha256(), "kb_stats": kb.stats(),
        "phases_ms_per_step": {k: round(v[0], 4) for k, v in phases.items()},
        "kernel_ms_per_step": {k: round(v, 4) for k, v in share.items()},
        "timing": {"step_timed_as": timed_as, "eager_ms_per_step": round(eager_ms, 4),
                   "graph_ms_per_step": round(graph_ms, 4)},
        "graph": {"ms_per_step": round(graph_ms, 4),
                  "triple_batch_per_s": hops * kb.n_triples * b / (graph_ms * 1e-3),
                  "replays_bitwise_equal_to_eager": all(same)},
        "roofline": {"bound": "latency", "achieved": None, "peak": PEAK_HBM_GBPS,
                     "unit": "GB/s", "frac": None, "traffic": None,
                     "note": "a 1 k-entity KB: each launch moves a few MB at most; the step is "
                             "bound by launch and kernel latency, not by HBM bandwidth"},
        "cpu_baseline": cpu, "parity": parity,
    }
    print(json.dumps(out), flush=True)
    gkb.close()


def grid_sweep(args, torch, kbgen, kbf):
    """Relation sweep of the grid scalability experiment (Sec. 3.1): the 2-hop
    inference follow(follow(x, r), r) for minibatches of 128 one-hot queries,
    reported as queries per second, for each relation count."""
    n, b = args.grid, 128
    torch.cuda.set_device(0)
    rows = []
    for m in [int(v) for v in args.grid_relations.split(",")]:
        s, r, o = kbgen.grid_kb(n, m)
        x, rr = kbgen.grid_inputs(n, m, b)
        kb = kbf.KB(s, r, o, n * n, m)
        X = torch.from_numpy(x).cuda().t().contiguous()
        R = torch.from_numpy(rr).cuda().t().contiguous()
        Y1, Y2 = torch.empty_like(X), torch.empty_like(X)
        for _ in range(args.warmup):
            kb.follow(kb.follow(X, R, out=Y1), R, out=Y2)
        torch.cuda.synchronize()
        t0 = torch.cuda.Event(enable_timing=True)
        t1 = torch.cuda.Event(enable_timing=True)
        t0.record()
        for _ in range(args.steps):
            kb.follow(kb.follow(X, R, out=Y1), R, out=Y2)
        t1.record()
        torch.cuda.synchronize()
        ms = t0.elapsed_time(t1) / args.steps
        rows.append({"relations": m, "triples": int(len(s)), "ms_per_minibatch": round(ms, 4),
                     "qps": round(b / (ms * 1e-3), 1)})
        log(f"[grid] n={n} m={m} {ms:.4f} ms per 2-hop minibatch, {b / (ms * 1e-3):.3e} qps")
        kb.close()
    print(json.dumps({"metric": "queries/s of 2-hop follow on an n x n grid KB", "unit": "qps",
                      "higher_is_better": True, "n_gpus": 1, "data": "synthetic",
                      "config": {"workload": "grid", "n": n, "entities": n * n, "batch": b},
                      "sweep": rows}), flush=True)


def oracle_table(args, kbgen):
    """The oracle alone on each workload's full inputs: forward, dX and dR
    timed separately (median of `runs`), at each thread count; one JSON line
    per (workload, threads), printed as it is measured."""
    names = args.oracle_workloads.split(",")
    for name in names:
        w = kbgen.WORKLOADS[name]
        t0 = time.perf_counter()
        kb = kbgen.make_kb(w)
        if name == "chain3":
            x0, rho, tgt = kbgen.make_chain_inputs(w, kb)
        else:
            X_bm, R_bm, dY_bm = kbgen.make_x(w), kbgen.make_r(w), kbgen.make_dy(w)
        log(f"[oracle] generated {w.label} in {time.perf_counter() - t0:.1f} s")
        counts = sorted({int(t) for t in args.oracle_threads.split(",")})
        for threads in counts:
            if name == "chain3":
                if threads != 1:
                    continue  # the chain oracle (double precision) runs on one thread
                from oracle import chain as ochain
                runs = args.oracle_runs or 20
                ts = []
                for _ in range(runs):
                    t1 = time.perf_counter()
                    ochain.chain_grad((kb.subj, kb.rel, kb.obj), w.n_entities, w.n_relations, x0,
                                      rho, tgt)
                    ts.append(time.perf_counter() - t1)
                dt = float(np.median(ts))
                rec = {"workload": name, "threads": 1, "runs": runs,
                       "step_s": round(dt, 6),
                       "triple_batch_per_s": 3 * kb.n_triples * w.batch / dt}
            else:
                th = min(threads, w.batch)
                runs = args.oracle_runs or (3 if w.n_triples > 10_000_000 else 20)
                med, _ = oracle_pass_times(kb, X_bm, R_bm, dY_bm, th, runs)
                dt = med["fwd"] + med["dx"] + med["dr"]
                rec = {"workload": name, "threads": th, "runs": runs,
                       "fwd_s": round(med["fwd"], 6), "dx_s": round(med["dx"], 6),
                       "dr_s": round(med["dr"], 6), "fwd_bwd_s": round(dt, 6),
                       "triple_batch_per_s": kb.n_triples * w.batch / dt}
            rec["cpu"] = cpu_model()
            rec["logical_cpus"] = os.cpu_count()
            print(json.dumps(rec), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="large",
                    help="tiny | metaqa | chain3 | large | train (kbgen workload names)")
    ap.add_argument("--batch", type=int, default=0,
                    help="batch width b instead of the workload's own (the same KB)")
    ap.add_argument("--cpu-threads", type=int, default=0,
                    help="host threads for the oracle (0: the cores this process may use, "
                         "at most 16)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-profile", action="store_true", help="skip the HIP-event phase timing")
    ap.add_argument("--residual", type=float, default=None, metavar="GAMMA",
                    help="time the residual hop follow(X, R) + GAMMA * X and its backward "
                         "(KB-completion chains) instead of the plain follow")
    ap.add_argument("--grid", type=int, default=0, metavar="N",
                    help="instead: queries/s of the 2-hop follow(follow(x, r), r) on the N x N "
                         "grid KB of the scalability experiment (b = 128 one-hot queries)")
    ap.add_argument("--grid-relations", default="4,20,100,1000",
                    help="relation counts of the grid sweep (comma separated)")
    ap.add_argument("--detail-iters", type=int, default=-1,
                    help="iterations of the per-pass timing with percentiles, warm and cold "
                         "cache (-1: 50 for the large KBs, 200 for metaqa, 1000 for tiny; 0: skip)")
    ap.add_argument("--oracle-table", action="store_true",
                    help="instead: time the oracle alone (no GPU) per workload and thread count")
    ap.add_argument("--oracle-workloads", default="tiny,metaqa,chain3,large,train")
    ap.add_argument("--oracle-threads", default="1,16")
    ap.add_argument("--oracle-runs", type=int, default=0,
                    help="runs per median (0: 3 for the KBs over 10 M triples, else 20)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain 1 GiB device copy 5 times (to scale rocprofv3 "
                         "FETCH_SIZE / WRITE_SIZE counters)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the follow path here has no multi-GPU sharding "
              "(run with --gpus 1)", file=sys.stderr)
        sys.exit(2)

    import kbgen
    if args.oracle_table:
        oracle_table(args, kbgen)
        return

    import torch
    import paper_2002_06115_amd as kbf

    if args.copy_calibration:
        n = (1 << 30) // 4
        src = torch.ones(n, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(5):
            torch.mul(src, 1.0, out=dst)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration": {"bytes_read": 4 * n, "bytes_written": 4 * n,
                                               "launches": 5}}))
        return
    if args.grid:
        grid_sweep(args, torch, kbgen, kbf)
        return
    if args.workload == "chain3":
        chain_bench(args, torch, kbgen, kbf)
        return
    follow_bench(args, torch, kbgen, kbf)


if __name__ == "__main__":
    main()
