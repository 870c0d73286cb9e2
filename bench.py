"""Benchmark: relation-set following forward + backward on one MI355X.

One step = kb_follow (forward, Eq. 4) + kb_follow_backward (dX and dR) over
the whole KB for one minibatch, inputs already resident in HBM.  The default
workload is the large KB: 10 M entities, 600 relations, 50 M distinct triples
with Zipf subject/object/relation marginals, b = 32, 1 %-dense X.

Prints one JSON line with the whole-step throughput (triple-batch products per
second, N_T * b / step time), a roofline entry for the dominant kernel (HIP
event time inside the timed region) and the CPU oracle timed on a bounded
sample of the same workload.
"""
from __future__ import annotations

import argparse
import json
import os
import platform
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "triple·batch products/sec for kb_follow fwd+bwd; achieved HBM GB/s vs peak"
PEAK_HBM_GBPS = 8000.0
DOMINANT_KERNEL_NAMES = {
    "fwd_stream": "stream_kernel (forward: objects, gathers X and R)",
    "dx_stream": "stream_kernel (dX: subjects, gathers dY and R)",
    "dr_stream": "stream_kernel (dR: relations, gathers X and dY)",
}


def log(*a):
    print(*a, file=sys.stderr, flush=True)


_DISTINCT = {}


def distinct_ids(kb):
    """Number of distinct subjects and of distinct objects of the KB."""
    key = id(kb)
    if key not in _DISTINCT:
        _DISTINCT[key] = (len(np.unique(kb.subj)), len(np.unique(kb.obj)))
    return _DISTINCT[key]


def pass_bytes(kb, b, phase, whole_pass=False):
    """Algorithmic bytes of one stream-kernel launch under three models, all
    with the index stream (8 B per triple), the row offsets and R:
      gather      every triple's b-wide operand rows come from memory;
      compulsory  each distinct gathered row once (rows no triple names are
                  never read);
      array_once  each operand array read once in full.
    The stream kernel writes the output rows that have triples; with
    whole_pass the rows without triples (written by the zero fill) count
    too, as for the whole pass."""
    n_t, n_e, n_r = kb.n_triples, kb.n_entities, kb.n_relations
    idx = 8 * n_t
    n_subj, n_obj = distinct_ids(kb)
    if phase in ("fwd_stream", "dx_stream"):
        n_a, n_out = (n_subj, n_obj) if phase == "fwd_stream" else (n_obj, n_subj)
        out = 4 * b * (n_e if whole_pass else n_out)
        gather = idx + 4 * (n_e + 1) + 4 * b * n_t + 4 * b * n_r + out    # A gathered per triple
        comp = idx + 4 * (n_e + 1) + 4 * b * n_a + 4 * b * n_r + out
        once = idx + 4 * (n_e + 1) + 4 * b * n_e + 4 * b * n_r + out
    else:
        gather = idx + 4 * (n_r + 1) + 8 * b * n_t + 4 * b * n_r
        comp = idx + 4 * (n_r + 1) + 4 * b * (n_subj + n_obj) + 4 * b * n_r
        once = idx + 4 * (n_r + 1) + 8 * b * n_e + 4 * b * n_r
    return float(gather), float(comp), float(once)


def column_tiling(b):
    """(VEC, LPT): 4 floats per lane when b % 4 == 0 (else 1), lanes per group
    b / VEC rounded up to a power of two, at most 32."""
    vec = 4 if b % 4 == 0 else 1
    lanes, lpt = -(-b // vec), 1
    while lpt < lanes and lpt < 32:
        lpt *= 2
    return vec, lpt


MAX_LDS_B = 80 * 1024     # B slice staged in LDS with two workgroups per CU
MAX_LDS_BIG = 160 * 1024  # with one workgroup per CU (hard KB only)


def stream_launch(b, b_rows, hard=True):
    """(LPT, lds) of the stream kernel a pass launches for batch b when its B
    table has b_rows rows (R for forward and dX, X for dR): B in LDS when its
    column slice fits (hard KB: rows cut into 32-column slices where that
    makes it fit).  The library also needs the LDS variant to keep at least as
    many waves on a CU as the register variant, which holds for the hard-KB,
    non-residual variants at b >= 32."""
    vec, lpt = column_tiling(b)
    if b_rows * vec * lpt * 4 <= MAX_LDS_B:
        return lpt, True
    if not hard:
        return lpt, False
    narrow = 8 if vec == 4 and lpt > 8 else lpt
    if b_rows * vec * narrow * 4 <= MAX_LDS_BIG:
        return narrow, True
    return lpt, False


def stream_kernel_symbol(b, weighted=False, residual=False, plain_loads=False, lds=False,
                         lpt=None):
    """Mangled name of the stream-kernel instance a pass launches for batch b:
    lane layout from column_tiling (or lpt lanes per group), raw-buffer loads
    unless a table reaches 4 GB, B staged in LDS (lds) or held in registers."""
    vec, lpt0 = column_tiling(b)
    lpt = lpt or lpt0
    flag = lambda v: 1 if v else 0
    return (f"_ZN3kbf12_GLOBAL__N_113stream_kernelILi{vec}ELi{lpt}ELb{flag(not plain_loads)}"
            f"ELb{flag(weighted)}ELb{flag(residual)}ELb{flag(lds and not plain_loads)}"
            f"EEEvNS_10StreamArgsE")


def overlap_backward(n_triples, b):
    """Whether the library runs the backward's dR pass concurrently with dX
    (from 2^20 triples at b <= 32 unless KBFOLLOW_OVERLAP_BACKWARD says
    otherwise)."""
    env = os.environ.get("KBFOLLOW_OVERLAP_BACKWARD")
    if env:
        return env != "0"
    return n_triples >= (1 << 20) and b <= 32


def measured_traffic(workload, b, phase, symbol):
    """DRAM bytes of one launch from the committed rocprofv3 counters, if they
    were taken on the device code of the kernel that is built now (same
    per-kernel assembly digest; a profile lists the kernel of each pass under
    "kernels", else one kernel for all)."""
    import glob
    fp_path = os.path.join(ROOT, "paper_2002_06115_amd", "_lib", "kernels.fingerprint")
    try:
        digest = json.load(open(fp_path)).get(symbol)
    except (OSError, ValueError):
        return None
    if not digest:
        return None
    for path in glob.glob(os.path.join(ROOT, "profiles", "*.json")):
        try:
            prof = json.load(open(path))
        except (OSError, ValueError):
            continue
        k = prof.get("kernels", {}).get(phase, prof)
        if prof.get("workload") == workload and prof.get("batch") == b \
                and k.get("symbol") == symbol and k.get("kernel_sha") == digest \
                and phase in prof.get("per_launch", {}):
            return float(prof["per_launch"][phase]["bytes"])
    return None


def cpu_baseline(kb, X_bm, R_bm, dY_bm, cols, threads, runs=3):
    """The oracle on the host cores: forward and backward (dX + dR) timed
    separately, median of `runs` runs on `threads` threads over `cols` batch
    columns, plus one thread on one column."""
    import oracle
    s, r, o = kb.subj, kb.rel, kb.obj
    n_e, n_r = kb.n_entities, kb.n_relations
    Xs, Rs, dYs = X_bm[:cols], R_bm[:cols], dY_bm[:cols]
    oracle.follow(s[:1000], r[:1000], o[:1000], n_e, n_r, Xs[:1], Rs[:1])  # load + warm

    def timed(c, nthreads):
        t0 = time.perf_counter()
        oracle.follow(s, r, o, n_e, n_r, Xs[:c], Rs[:c], nthreads=nthreads)
        t1 = time.perf_counter()
        oracle.follow_backward(s, r, o, n_e, n_r, Xs[:c], Rs[:c], dYs[:c], nthreads=nthreads)
        return t1 - t0, time.perf_counter() - t1

    multi = sorted((timed(cols, threads) for _ in range(runs)), key=sum)[runs // 2]
    fwd_s, bwd_s = multi
    dt = fwd_s + bwd_s
    one = timed(1, 1)
    return {
        "value": kb.n_triples * cols / dt,
        "unit": "triple·batch/s",
        "cores": int(min(threads, cols)),
        "kind": "oracle",
        "sample": (f"same KB, {cols} of {X_bm.shape[0]} batch columns, forward {fwd_s:.2f} s + "
                   f"backward (dX + dR) {bwd_s:.2f} s, median of {runs} runs on "
                   f"{min(threads, cols)} threads of {os.cpu_count()} ({cpu_model()})"),
        "fwd_s": round(fwd_s, 3),
        "bwd_s": round(bwd_s, 3),
        "single_thread_value": kb.n_triples / sum(one),
        "single_thread_sample": (f"1 batch column on 1 thread, forward {one[0]:.2f} s + "
                                 f"backward {one[1]:.2f} s"),
    }


def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor() or platform.machine()


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


def probe_lib():
    """The measurement library (libkbprobe.so), or None when it is not built."""
    import ctypes
    from paper_2002_06115_amd import build as kbuild
    if not os.path.exists(kbuild.PROBE_LIB):
        return None
    lib = ctypes.CDLL(kbuild.PROBE_LIB)
    P, I64, I32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32
    F = ctypes.POINTER(ctypes.c_float)
    lib.kbp_gather_time.argtypes = [P, I64, I32, P, I32, P, I32, P, F]
    lib.kbp_stream_read_time.argtypes = [P, I64, I32, P, I32, P, F]
    lib.kbp_stream_copy_time.argtypes = [P, P, I64, I32, I32, P, F]
    lib.kbp_stream_write_time.argtypes = [P, I64, I32, I32, P, F]
    return lib


def stream_rates(torch, lib, reps=10):
    """Device streaming rates on a 2 GiB buffer (best over a few grid sizes):
    sequential read GB/s, copy GB/s (bytes read + written) and non-temporal
    zero-fill GB/s."""
    import ctypes
    n = (2 << 30) // 4
    src = torch.ones(n, device="cuda")
    dst = torch.empty_like(src)
    read, copy, write = [], [], []
    for blocks in (1024, 4096, 16384):
        scratch = torch.empty(blocks * 256, device="cuda")
        ms = ctypes.c_float()
        if lib.kbp_stream_read_time(src.data_ptr(), n // 4, blocks, scratch.data_ptr(), reps,
                                    None, ctypes.byref(ms)) != 0:
            raise SystemExit("kbp_stream_read_time failed")
        read.append(4 * n / (ms.value * 1e-3) / 1e9)
        if lib.kbp_stream_copy_time(src.data_ptr(), dst.data_ptr(), n // 4, blocks, reps, None,
                                    ctypes.byref(ms)) != 0:
            raise SystemExit("kbp_stream_copy_time failed")
        copy.append(2 * 4 * n / (ms.value * 1e-3) / 1e9)
        if lib.kbp_stream_write_time(dst.data_ptr(), n // 4, blocks, reps, None,
                                     ctypes.byref(ms)) != 0:
            raise SystemExit("kbp_stream_write_time failed")
        write.append(4 * n / (ms.value * 1e-3) / 1e9)
    del src, dst, scratch
    return round(max(read), 1), round(max(copy), 1), round(max(write), 1)


def gather_probe(args, torch, kbgen, kbf):
    """The memory system's own rate for each pass's row reads: a pure gather
    (libkbprobe.so, no products, no second operand, no output rows) of the
    index stream a pass reads per triple, beside the pass's stream-kernel
    time, plus uniformly random indices for reference."""
    import ctypes
    lib = probe_lib()
    if lib is None:
        raise SystemExit("libkbprobe.so is not built (run __graft_entry__.build())")
    w = kbgen.WORKLOADS[args.workload]
    kb = kbgen.make_kb(w)
    torch.cuda.set_device(0)
    em = lambda a: torch.from_numpy(a).cuda().t().contiguous()
    X, R, dY = em(kbgen.make_x(w)), em(kbgen.make_r(w)), em(kbgen.make_dy(w))
    b, chunk = w.batch, 256
    gkb = kbf.KB(kb.subj, kb.rel, kb.obj, w.n_entities, w.n_relations)
    Y, dX, dR = torch.empty_like(X), torch.empty_like(X), torch.empty_like(R)
    gkb.follow(X, R, out=Y)
    gkb.follow_backward(X, R, dY, dX=dX, dR=dR)
    torch.cuda.synchronize()
    gkb.profile(True)
    for _ in range(args.steps):
        gkb.follow(X, R, out=Y)
        gkb.follow_backward(X, R, dY, dX=dX, dR=dR)
    ph = gkb.profile_read()
    gkb.profile(False)
    passes = {k: round(ph[k][0] / max(1, ph[k][1]), 4) for k in ("fwd_stream", "dx_stream",
                                                                  "dr_stream")}
    stream_read, stream_copy, stream_write = stream_rates(torch, lib)
    log(f"[probe] 2 GiB sequential read {stream_read} GB/s, copy {stream_copy} GB/s, "
        f"zero fill {stream_write} GB/s")
    lay = {which: kbf.layout_host(kb.subj, kb.rel, kb.obj, w.n_entities, w.n_relations, which)
           for which in (0, 1, 2)}
    rng = np.random.default_rng(np.random.SeedSequence([20020615, 99]))
    streams = [
        ("forward: subjects in object order, rows of X", lay[0][1], X),
        ("dX: objects in subject order, rows of dY", lay[1][1], dY),
        ("dR: objects in relation order, rows of dY", lay[2][1], dY),
        ("dR: subjects in relation order, rows of X", lay[2][2], X),
        ("uniform random entity ids, rows of X",
         rng.integers(0, w.n_entities, kb.n_triples).astype(np.int32), X),
    ]
    rows = []
    for name, ids, table in streams:
        idx = torch.from_numpy(np.ascontiguousarray(ids, dtype=np.int32)).cuda()
        n = idx.numel()
        out = torch.empty(((n + chunk - 1) // chunk) * b, device="cuda")
        ms = ctypes.c_float()
        rc = lib.kbp_gather_time(idx.data_ptr(), n, chunk, table.data_ptr(), b, out.data_ptr(),
                                 max(1, args.steps), ctypes.c_void_p(None), ctypes.byref(ms))
        if rc != 0:
            raise SystemExit(f"kbp_gather_time failed ({rc})")
        rows.append({"stream": name, "rows": n, "ms": round(ms.value, 4),
                     "gathered_GBps": round(n * 4 * b / (ms.value * 1e-3) / 1e9, 1)})
        log(f"[probe] {name}: {ms.value:.4f} ms")
        del idx, out
    print(json.dumps({"metric": "pure-gather time of each pass's per-triple row reads",
                      "config": {"workload": w.name, "batch": b, "chunk": chunk},
                      "stream_kernel_ms": passes, "sequential_read_GBps": stream_read,
                      "copy_GBps": stream_copy, "probe": rows}), flush=True)
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


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="large",
                    help="tiny | metaqa | large | train (kbgen workload names)")
    ap.add_argument("--cpu-cols", type=int, default=0,
                    help="batch columns the oracle times (0 = all b)")
    ap.add_argument("--cpu-threads", type=int, default=16)
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
    ap.add_argument("--gather-probe", action="store_true",
                    help="instead: time a pure gather of each pass's per-triple row reads "
                         "(the memory system's rate for that access pattern) beside the passes")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain 1 GiB device copy 5 times (to scale rocprofv3 "
                         "FETCH_SIZE / WRITE_SIZE counters)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the follow path here has no multi-GPU sharding "
              "(run with --gpus 1)", file=sys.stderr)
        sys.exit(2)

    import torch
    import kbgen
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
    if args.gather_probe:
        gather_probe(args, torch, kbgen, kbf)
        return

    w = kbgen.WORKLOADS[args.workload]
    if w.name == "chain3":
        raise SystemExit("chain3 is a parity case, not a bench workload")
    t0 = time.perf_counter()
    kb = kbgen.make_kb(w)
    X_bm, R_bm, dY_bm = kbgen.make_x(w), kbgen.make_r(w), kbgen.make_dy(w)
    log(f"[bench] generated {w.label} in {time.perf_counter() - t0:.1f} s; stats {kb.stats()}")

    torch.cuda.set_device(0)
    t0 = time.perf_counter()
    gkb = kbf.KB(kb.subj, kb.rel, kb.obj, w.n_entities, w.n_relations)
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

    def step():
        gkb.follow(X, R, out=Y, stream=stream, residual=args.residual)
        gkb.follow_backward(X, R, dY, dX=dX, dR=dR, stream=stream, residual=args.residual)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    log(f"[bench] warmup {args.warmup} done")

    # Events around a phase cost a few microseconds of GPU time each, so the
    # per-phase breakdown comes from a loop of its own, and the timed steps
    # bracket only the dominant stream kernel (the roofline's kernel).
    phases, dom = {}, None
    if not args.no_profile:
        gkb.profile(True)
        for _ in range(args.steps):
            step()
        torch.cuda.synchronize()
        phases = gkb.profile_read()
        gkb.profile(False)
        # With the backward's dX and dR passes running concurrently their
        # launch durations overlap and are no per-kernel cost, so the
        # roofline is then taken on the forward stream kernel, which runs
        # alone; otherwise on the slowest of the three.
        candidates = ("fwd_stream",) if overlap_backward(kb.n_triples, b) else \
            ("fwd_stream", "dx_stream", "dr_stream")
        dom = max(candidates, key=lambda p: phases[p][0])
        gkb.profile(True, phases=[dom])
    start = torch.cuda.Event(enable_timing=True)
    stop = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record(stream)
    for _ in range(args.steps):
        step()
    stop.record(stream)
    torch.cuda.synchronize()
    ms_total = start.elapsed_time(stop)
    dom_timed = gkb.profile_read()[dom] if dom else None
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
        lib = probe_lib()
        if lib is not None:
            (detail["stream_read_GBps"], detail["copy_GBps"],
             detail["write_GBps"]) = stream_rates(torch, lib)
        log(f"[bench] detail {json.dumps(detail)}")

    roof = None
    if dom:
        # The dominant kernel's mean launch time within the timed steps.
        ms_avg = dom_timed[0] / max(1, dom_timed[1])
        gather_b, comp_b, once_b = pass_bytes(kb, b, dom)
        sec = ms_avg * 1e-3
        b_rows = w.n_entities if dom == "dr_stream" else w.n_relations
        lpt, lds = stream_launch(b, b_rows, hard=args.residual is None)
        if os.environ.get("KBFOLLOW_B_IN_LDS") == "0":
            lpt, lds = None, False
        symbol = stream_kernel_symbol(b, residual=args.residual is not None,
                                      plain_loads=os.environ.get("KBFOLLOW_PLAIN_LOADS") == "1",
                                      lds=lds, lpt=lpt)
        traffic = measured_traffic(w.name, b, dom, symbol)
        roof = {"bound": "hbm", "achieved": round(comp_b / sec / 1e9, 1), "peak": PEAK_HBM_GBPS,
                "kernel_choice": ("forward stream kernel: dX and dR run concurrently, so their "
                                  "launch durations overlap" if dom == "fwd_stream"
                                  and overlap_backward(kb.n_triples, b) else
                                  "the slowest of the three stream kernels"),
                "unit": "GB/s", "frac": round(comp_b / sec / 1e9 / PEAK_HBM_GBPS, 4),
                "traffic": traffic,
                "kernel": DOMINANT_KERNEL_NAMES[dom], "kernel_ms": round(ms_avg, 4),
                "bytes_model": "compulsory: 8 B of ids per triple, row offsets, every distinct "
                               "gathered row once, R, every output row once",
                "algorithmic_bytes": comp_b,
                "gather_model_bytes": gather_b,
                "gather_model_GBps": round(gather_b / sec / 1e9, 1),
                "array_once_bytes": once_b,
                "array_once_GBps": round(once_b / sec / 1e9, 1),
                "array_once_frac": round(once_b / sec / 1e9 / PEAK_HBM_GBPS, 4)}
        # The whole step (fwd + dX + dR and their combine and zero-fill
        # launches) against the three passes' bytes.
        step_sec = ms_step * 1e-3
        step = [pass_bytes(kb, b, p, whole_pass=True) for p in ("fwd_stream", "dx_stream", "dr_stream")]
        step_comp, step_once = sum(x[1] for x in step), sum(x[2] for x in step)
        roof["step"] = {"ms": round(ms_step, 4),
                        "compulsory_bytes": step_comp,
                        "compulsory_frac": round(step_comp / step_sec / 1e9 / PEAK_HBM_GBPS, 4),
                        "array_once_bytes": step_once,
                        "array_once_frac": round(step_once / step_sec / 1e9 / PEAK_HBM_GBPS, 4)}
        if traffic:
            roof["hbm_measured_GBps"] = round(traffic / sec / 1e9, 1)
            roof["hbm_measured_frac"] = round(traffic / sec / 1e9 / PEAK_HBM_GBPS, 4)
        if detail and "stream_read_GBps" in detail:
            # The device's own streaming rates (libkbprobe.so, 2 GiB buffer):
            # a sequential read, and a copy (bytes read + written).
            rd, cp = detail["stream_read_GBps"], detail["copy_GBps"]
            roof["stream_read_GBps"] = rd
            roof["copy_GBps"] = cp
            roof["achieved_frac_of_copy"] = round(comp_b / sec / 1e9 / cp, 4)
            if traffic:
                roof["hbm_measured_frac_of_stream_read"] = round(traffic / sec / 1e9 / rd, 4)
                roof["hbm_measured_frac_of_copy"] = round(traffic / sec / 1e9 / cp, 4)

    cpu = None
    if not args.no_cpu_baseline:
        cols = b if args.cpu_cols <= 0 else max(1, min(args.cpu_cols, b))
        threads = max(1, min(cols, args.cpu_threads, os.cpu_count() or 1))
        log(f"[bench] timing the CPU oracle on {cols} batch columns, {threads} threads")
        cpu = cpu_baseline(kb, X_bm, R_bm, dY_bm, cols, threads)
        log(f"[bench] oracle {cpu['value']:.3e} triple*batch/s")

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
        "phases_ms_per_step": {k: round(v[0] / args.steps, 4) for k, v in phases.items()},
        "concurrent_backward": overlap_backward(kb.n_triples, b),
        "phases_note": ("HIP-event times per phase from a separate loop of the same steps; the "
                        "timed steps bracket only the roofline's kernel with events; with "
                        "concurrent_backward the dx_* and dr_* phases run at the same time, so "
                        "their times overlap"),
        "kb_create_s": round(create_s, 2),
        "timing": detail,
        "roofline": roof,
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
