#!/usr/bin/env python
"""Throughput of the trace-attribution join on one MI355X.

One step = one opattr_attribute call (invocation-order matching, layer-dedup
broadcast, enclosure, aggregation) over the large synthetic trace: 10M kernel
launches on 16 streams, 500k nested ranges (depth <= 8), 1000 kernel names
Zipf(1.1), layer dedup 48 layers / 3 classes, 1M profiled rows of 20 fp32
counters. Inputs are resident in HBM before the timed region. Prints one JSON
line: records/s (wall clock over the timed steps, no probe events inside
them), per-step spread and graph-replayed step time, the dominant kernel
against the HBM roofline (HIP probe events recorded by the library around its
launch, on its stream), a per-kernel table, a device copy's rate in the same
run, rows for the other workloads and launch orders, and the oracle's rate on
one host core as a reported CPU baseline.
"""
import argparse
import json
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "kernel records attributed/sec (match+enclose+aggregate); % of HBM peak"
HBM_PEAK_GBPS = 8000.0  # MI355X HBM3E


def algorithmic_bytes(tr):
    """Compulsory bytes of one step: every input read once, every output
    written once, at the ABI widths (duplicate counter rows reused by dedup
    count once)."""
    T, P, R = tr["seq"].size, tr["pf_name"].size, tr["r_start"].size
    part = 4 if tr.get("part_id") is not None else 0
    G = tr["n_ops"] + 1
    NP = tr.get("n_parts", 0) or 0
    timeline = T * (4 + 8 + 4 + 2 + 4 + part)      # seq, start, dur, stream, name, part
    profiled = P * (4 + 20 * 4)                     # name + 20 counters
    ranges = R * (8 + 8 + 2 + 4)                    # start, end, stream, op
    outputs = T * (4 + 4)                           # match, range_id
    table = G * 192 + 4 * NP                        # op rows + class map
    return timeline + profiled + ranges + outputs + table


def eligible_launches(tr):
    """Launches that rank themselves (not a layer duplicate, valid name)."""
    import numpy as np

    ok = tr["name_id"] < tr["n_names"]
    part = tr.get("part_id")
    if part is None or tr.get("part_rep") is None:
        return int(ok.sum())
    rep = tr["part_rep"]
    p = part.astype(np.int64)
    own = (p < 0) | (rep[np.clip(p, 0, rep.size - 1)] == p)
    return int((ok & own).sum())


def fused_kernels(tr):
    """The kernels of one opattr_attribute step on the fused path (kernels
    stream-major with dense seq, sparse ranges), each with the probe that
    brackets it, the stream it runs on and its algorithmic bytes per launch
    of the kernel: what it must read and write for its own function."""
    T, P, R = tr["seq"].size, tr["pf_name"].size, tr["r_start"].size
    part = 4 if tr.get("part_id") is not None else 0
    E = eligible_launches(tr)
    return [
        # seq tiles: seq, name and partition of every launch
        dict(kernel="k_f_pass1", probe="tl_hist", stream="caller", bytes=T * (4 + 4 + part)),
        # ranks of the eligible launches: their bucket records in, row and
        # name by seq rank out
        dict(kernel="k_f_pass2", probe="tl_match", stream="caller", bytes=E * (4 + 4 + 4)),
        # every launch's match with the dedup broadcast (seq, name,
        # partition in, match out) and the run reduction (range id and
        # duration of every launch, the op of each range and each profiled
        # counter row once)
        dict(kernel="k_f_agg", probe="agg_runs", stream="caller",
             bytes=T * (4 + 4 + part + 4 + 4 + 4) + R * 4 + P * 80),
        # enclosure: stream and query point of every launch in, range id
        # out; range starts, ends and parents
        dict(kernel="k_enclose", probe="main_pass", stream="side 1",
             bytes=T * (2 + 8 + 4) + R * (8 + 8 + 4)),
        # profiled rows: names in (histograms), names in and slots out
        dict(kernel="k_pf_hist_w", probe="pf_hist", stream="side 2", bytes=P * 4),
        dict(kernel="k_pf_slot_w", probe="pf_slot", stream="side 2", bytes=P * (4 + 4)),
    ]


def source_hash():
    """Hash of the HIP sources: stored traffic counters are valid only for the
    kernels they were taken on."""
    import glob
    import hashlib

    h = hashlib.sha256()
    for f in sorted(glob.glob(os.path.join(ROOT, "paper_2609_11938_amd", "csrc", "*"))) + \
            [os.path.join(ROOT, "include", "opattr.h")]:
        with open(f, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def stored_traffic(kernel, config, emission):
    """HBM bytes per launch of `kernel` from profiles/traffic_<kernel>_<config>_<emission>.txt
    (two rocprofv3 --pmc passes, FETCH_SIZE then WRITE_SIZE, scaled by a plain
    copy of known size), or None when absent or taken on other sources."""
    path = os.path.join(ROOT, "profiles", f"traffic_{kernel}_{config}_{emission}.txt")
    if not os.path.exists(path):
        return None
    kv = {}
    with open(path) as fh:
        for line in fh:
            if ":" in line and not line.startswith("#"):
                k, v = line.split(":", 1)
                kv[k.strip()] = v.strip()
    if kv.get("source_hash") != source_hash():
        return None
    try:
        return float(kv["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def copy_calibration(mb, reps):
    """A plain device-to-device copy of `mb` MiB, `reps` times: the reference
    the FETCH_SIZE / WRITE_SIZE counters are scaled by."""
    import torch

    n = mb * (1 << 20) // 4
    a = torch.arange(n, dtype=torch.int32, device="cuda:0")
    b = torch.empty_like(a)
    for _ in range(reps):
        b.copy_(a)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes": n * 4, "reps": reps}), flush=True)


def stored_kernel_ms(kernel, config, emission):
    """Average duration (ms) of `kernel` in the committed rocprofv3 kernel
    statistics of this workload (profiles/attribute_<config>_<emission>_kernel_stats.txt),
    or None when absent or taken on other sources."""
    path = os.path.join(ROOT, "profiles", f"attribute_{config}_{emission}_kernel_stats.txt")
    if not os.path.exists(path):
        return None
    ok, ms = False, None
    with open(path) as fh:
        for line in fh:
            if line.startswith("# source_hash:"):
                ok = line.split(":", 1)[1].strip() == source_hash()
            f = line.split()
            if len(f) >= 3 and not line.startswith("#") and \
                    (f[0] == kernel or f[0].startswith(kernel + "<")):
                try:
                    ms = float(f[2]) / 1e3
                except ValueError:
                    pass
    return ms if ok else None


def copy_bandwidth(mib=1024, reps=10):
    """Device-to-device copy rate (read + write bytes per second) in the same
    run: the practical HBM ceiling next to the 8 TB/s peak."""
    import torch

    n = mib * (1 << 20) // 4
    a = torch.ones(n, dtype=torch.int32, device="cuda:0")
    b = torch.empty_like(a)
    for _ in range(2):
        b.copy_(a)
    ev = [_events(2) for _ in range(reps)]
    for e0, e1 in ev:
        e0.record()
        b.copy_(a)
        e1.record()
    torch.cuda.synchronize()
    ms = statistics.median(e0.elapsed_time(e1) for e0, e1 in ev)
    del a, b
    return {"bytes": 2 * n * 4, "median_ms": ms, "GBps": 2 * n * 4 / (ms * 1e-3) / 1e9}


def clocks():
    """Current SCLK / MCLK levels as the driver lists them in sysfs (the line
    marked '*' of pp_dpm_sclk / pp_dpm_mclk), or None when unavailable. Read
    from files: no child process is started from this GPU process."""
    import glob

    out = {}
    for dev in sorted(glob.glob("/sys/class/drm/card*/device")):
        for clk in ("sclk", "mclk"):
            try:
                with open(os.path.join(dev, f"pp_dpm_{clk}")) as fh:
                    cur = [ln.strip() for ln in fh if ln.strip().endswith("*")]
            except OSError:
                continue
            if cur:
                out[clk] = cur[0].rstrip("*").strip()
        if out:
            return out
    return None


def cpu_info():
    model = None
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return model, os.cpu_count()


def cpu_baseline(tr, reps=3):
    """The oracle on one host core (the process pinned to core 0, as taskset -c 0
    would): one warm-up run, then `reps` timed runs of the full workload."""
    from oracle import oracle as O

    O.build(force=False)
    prev = os.sched_getaffinity(0)
    os.sched_setaffinity(0, {0})
    try:
        O.attribute(tr)
        times = []
        for _ in range(reps):
            t0 = time.perf_counter()
            O.attribute(tr)
            times.append(time.perf_counter() - t0)
    finally:
        os.sched_setaffinity(0, prev)
    med = statistics.median(times)
    model, ncpu = cpu_info()
    return {"value": tr["seq"].size / med, "unit": "records/s", "cores": 1, "kind": "oracle",
            "sample": f"the full workload ({tr['seq'].size} launches): 1 warm-up + {reps} "
                      f"runs pinned to core 0, median {med:.2f} s (min {min(times):.2f}, "
                      f"max {max(times):.2f}), single-threaded C oracle",
            "cpu_model": model, "nproc": ncpu}


def _events(n):
    import torch

    row = [torch.cuda.Event(enable_timing=True) for _ in range(n)]
    for e in row:
        e.record()  # materialise the HIP event before handing it over
    return row


def measure_next_rows(dt, tr, flags, steps, warmup, out, ws):
    """The rows beyond the core hot path that this library also runs, timed on
    the same trace after the headline measurement: the attribution with the
    kind-aware walk of Alg. 2 (outermost ranges as boundaries, a fifth of the
    others skipped), tiered attribution (correlation map, enclosure, fusion
    map) and layer class discovery (Sec. 3.7)."""
    import torch

    from paper_2609_11938_amd import opattr, tracegen

    T, R = tr["seq"].size, tr["r_start"].size
    NP = tr.get("n_parts", 0) or 0
    rows = {}

    kinds = tracegen.with_range_kinds(tr)["r_kind"]
    dtk = dict(dt, r_kind=torch.from_numpy(kinds).to(dt["seq"].device))

    def walk_step():
        opattr.opattr_attribute(dtk, flags=flags, outputs=out, ws=ws, raise_strict=False)

    for _ in range(warmup):
        walk_step()
    torch.cuda.synchronize()
    diag = opattr.read_diag(out["diag"])
    if diag["status"] != 0:
        raise SystemExit(f"attribution with range kinds reported {diag}")
    pm = opattr.PROBES.index("main_pass")
    ev = [_events(2) for _ in range(steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(steps):
        only = [None] * (2 * len(opattr.PROBES))
        only[2 * pm], only[2 * pm + 1] = ev[k]
        opattr.set_probe_events(only)
        walk_step()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    opattr.set_probe_events(None)
    ms = (t1 - t0) * 1e3 / steps
    enc_ms = statistics.mean(a.elapsed_time(b) for a, b in ev)
    # k_enclose with kinds: stream, query point in, range id out; range
    # starts, ends, parents and kinds
    enc_bytes = T * (2 + 8 + 4) + R * (8 + 8 + 4 + 1)
    enc_gbps = enc_bytes / (enc_ms * 1e-3) / 1e9
    rows["enclose_walk"] = {
        "call": "opattr_attribute, ranges with kinds", "ms_per_step": ms,
        "records_per_s": T / (ms * 1e-3), "boundaries": int((kinds == 1).sum()),
        "skipped": int((kinds == 2).sum()), "kernel": "k_enclose", "kernel_ms": enc_ms,
        "kernel_algorithmic_bytes": enc_bytes, "kernel_GBps": enc_gbps,
        "kernel_frac": enc_gbps / HBM_PEAK_GBPS}

    # all enclosing ranges of every launch as CSR lists (one call into a
    # buffer sized by a first call)
    first = opattr.opattr_enclose_all(dtk, flags=flags, ws=ws)
    total = int(first["ids"].numel())
    ids = torch.empty(max(total, 1), dtype=torch.int32, device=dt["seq"].device)
    for _ in range(warmup):
        opattr.opattr_enclose_all(dtk, flags=flags, ids=ids, ws=ws)
    ev = [_events(2) for _ in range(steps)]
    torch.cuda.synchronize()
    for k in range(steps):
        ev[k][0].record()
        opattr.opattr_enclose_all(dtk, flags=flags, ids=ids, ws=ws)
        ev[k][1].record()
    torch.cuda.synchronize()
    all_ms = statistics.mean(a.elapsed_time(b) for a, b in ev)
    # stream and query point per launch, the lists and offsets out, range
    # starts, ends, parents once
    all_bytes = T * (2 + 8 + 8) + total * 4 + R * (8 + 8 + 4)
    agbps = all_bytes / (all_ms * 1e-3) / 1e9
    rows["enclose_all"] = {
        "call": "opattr_enclose_all (CSR lists, innermost first)", "entries": total,
        "ms_per_call": all_ms, "records_per_s": T / (all_ms * 1e-3),
        "algorithmic_bytes": all_bytes, "achieved_GBps": agbps, "frac": agbps / HBM_PEAK_GBPS}

    # tiered attribution: the pipeline of library calls (matching with the
    # dedup broadcast, the walk, the tiers, the table by tier operator) with
    # a correlation map for 40% of the names and a fusion map for 30%
    maps = tracegen.with_attribution_maps(dict(tr, r_kind=kinds))
    dtm = dict(dtk)
    for f in ("corr_name", "corr_op", "fmap_off", "fmap_op"):
        dtm[f] = torch.from_numpy(maps[f]).to(dt["seq"].device)
    res = None
    for _ in range(warmup):
        res = opattr.attribute_tiered(dtm, flags=flags, ws=ws)
    torch.cuda.synchronize()
    diag = opattr.read_diag(res["tiers"]["diag"])
    if diag["status"] not in (0, -4):
        raise SystemExit(f"tiered attribution reported {diag}")
    cov = res["tiers"].coverage_host()
    ev = [_events(4) for _ in range(steps)]
    torch.cuda.synchronize()
    for k in range(steps):
        ev[k][0].record()
        r = opattr.attribute_tiered(dtm, flags=flags, ws=ws)
        ev[k][1].record()
        opattr.opattr_tiers(dtm, r["walk"]["range_id"], r["walk"]["fused"], flags=flags, ws=ws)
        ev[k][2].record()
        opattr.opattr_aggregate_dispatch(dtm, r["match"]["match"], r["walk"]["range_id"],
                                         r["tiers"]["op"], flags=flags, ws=ws)
        ev[k][3].record()
    torch.cuda.synchronize()
    pipe_ms = statistics.mean(e[0].elapsed_time(e[1]) for e in ev)
    tiers_ms = statistics.mean(e[1].elapsed_time(e[2]) for e in ev)
    disp_ms = statistics.mean(e[2].elapsed_time(e[3]) for e in ev)
    # the same in one library call (the ranges and the walk on a side stream)
    one = None
    for _ in range(warmup):
        one = opattr.opattr_attribute_tiered(dtm, flags=flags, ws=ws)
    torch.cuda.synchronize()
    ev1 = [_events(2) for _ in range(steps)]
    torch.cuda.synchronize()
    for k in range(steps):
        ev1[k][0].record()
        opattr.opattr_attribute_tiered(dtm, flags=flags, ws=ws)
        ev1[k][1].record()
    torch.cuda.synchronize()
    one_ms = statistics.mean(a.elapsed_time(b) for a, b in ev1)
    if not torch.equal(one["tier"], res["tiers"]["tier"]):
        raise SystemExit("one-call and composed tiers differ")
    C_ = maps["corr_name"].size
    # opattr_tiers alone: the correlation join (seq, name per launch; name
    # per entry) and the tier pass (name, dur, range id, walk fused in;
    # tier, op, fused out; entry op gathered once per launch at most)
    tier_bytes = T * (4 + 4) + C_ * (4 + 4) + T * (4 + 4 + 4 + 1 + 1 + 4 + 1)
    gbps = tier_bytes / (tiers_ms * 1e-3) / 1e9
    rows["tiered"] = {
        "call": "opattr_attribute_tiered (matching + dedup broadcast, walk, tiers, table)",
        "ms_per_step": one_ms, "records_per_s": T / (one_ms * 1e-3),
        "composed_calls_ms": pipe_ms,
        "correlation_entries": int(C_),
        "coverage_frac": {"high": float(cov["frac"][1]), "nvtx": float(cov["frac"][2]),
                          "fusion": float(cov["frac"][3]),
                          "unattributed": float(cov["frac"][0])},
        "tiers_call_ms": tiers_ms, "tiers_algorithmic_bytes": tier_bytes,
        "tiers_GBps": gbps, "tiers_frac": gbps / HBM_PEAK_GBPS}
    # the per-dispatch table: range id, tier op, match, duration per launch,
    # the op of each range, each counter row once; one row per dispatch out
    G_disp = R + tr["n_ops"] + 1
    disp_bytes = T * (4 + 4 + 4 + 4 + 4) + R * 4 + tr["pf_name"].size * 80 + G_disp * 192
    dgbps = disp_bytes / (disp_ms * 1e-3) / 1e9
    rows["dispatch_table"] = {
        "call": "opattr_aggregate_dispatch", "rows": int(G_disp), "ms_per_call": disp_ms,
        "records_per_s": T / (disp_ms * 1e-3), "algorithmic_bytes": disp_bytes,
        "achieved_GBps": dgbps, "frac": dgbps / HBM_PEAK_GBPS}

    if NP:
        cflags = flags & (opattr.SEQ_DENSE | opattr.VALIDATE)
        res = None
        for _ in range(warmup):
            res = opattr.opattr_dedup_classes(dt, flags=cflags, ws=ws)
        torch.cuda.synchronize()
        diag = opattr.read_diag(res["diag"])
        if diag["status"] != 0:
            raise SystemExit(f"class discovery reported {diag}")
        n_classes = int(torch.unique(res["part_rep"]).numel())
        ev = [_events(2) for _ in range(steps)]
        torch.cuda.synchronize()
        for k in range(steps):
            ev[k][0].record()
            opattr.opattr_dedup_classes(dt, flags=cflags, ws=ws)
            ev[k][1].record()
        torch.cuda.synchronize()
        cls_ms = statistics.mean(a.elapsed_time(b) for a, b in ev)
        # every launch's seq, name, stream and partition read once; the class
        # map written once
        cls_bytes = T * (4 + 4 + 2 + 4) + 4 * NP
        gbps = cls_bytes / (cls_ms * 1e-3) / 1e9
        rows["dedup_classes"] = {
            "call": "opattr_dedup_classes", "ms_per_call": cls_ms,
            "records_per_s": T / (cls_ms * 1e-3), "partitions": int(NP),
            "classes": n_classes, "algorithmic_bytes": cls_bytes, "achieved_GBps": gbps,
            "frac": gbps / HBM_PEAK_GBPS}
    return rows


FLAGS = {"stream_major": 1 | 2 | 4, "seq": 2, "shuffled": 0}  # layout hints per emission


def new_outputs(tr, dev):
    import torch

    from paper_2609_11938_amd import opattr

    T = tr["seq"].size
    return opattr.Outputs(
        match=torch.empty(T, dtype=torch.int32, device=dev),
        range_id=torch.empty(T, dtype=torch.int32, device=dev),
        range_depth=None, name_counts=None,
        table=torch.empty((tr["n_ops"] + 1) * 192, dtype=torch.uint8, device=dev),
        summary=torch.empty(40, dtype=torch.uint8, device=dev))


def timed_steps(step, steps, warmup, flush=None):
    """`warmup` untimed steps, then exactly `steps` timed ones bracketed by
    synchronisations: the wall clock over all of them, and each step's span
    from HIP events recorded on the caller's stream between steps (a flush,
    when given, runs before each step, outside its span)."""
    import torch

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    ev = [_events(2) for _ in range(steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for e0, e1 in ev:
        if flush is not None:
            flush()
        e0.record()
        step()
        e1.record()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    per = [e0.elapsed_time(e1) for e0, e1 in ev]
    return (t1 - t0) * 1e3 / steps, per


def graph_step_ms(step, steps):
    """One step captured in a HIP graph (both side-stream branches) and
    replayed `steps` times: ms per replay, median over the replays."""
    import torch

    cap = torch.cuda.Stream()
    cap.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(cap):
        step()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=cap):
        step()
    g.replay()
    torch.cuda.synchronize()
    ev = [_events(2) for _ in range(steps)]
    torch.cuda.synchronize()
    for e0, e1 in ev:
        e0.record()
        g.replay()
        e1.record()
    torch.cuda.synchronize()
    per = [e0.elapsed_time(e1) for e0, e1 in ev]
    del g
    return statistics.median(per), min(per), max(per)


def spread(per):
    return {"median": statistics.median(per), "min": min(per), "max": max(per)}


def config_row(name, emission, validate, steps, warmup, dev, graph, flush_mib):
    """records/s of one opattr_attribute step on another workload (inputs
    resident; optional graph replay; optional flush of the caches by writing
    a `flush_mib` MiB buffer before each timed step)."""
    import torch

    from paper_2609_11938_amd import opattr, tracegen

    tr = tracegen.generate(name, emission=emission)
    dt = opattr.to_device(tr, dev)
    flags = FLAGS[emission] | (opattr.VALIDATE if validate else 0)
    ws = opattr.Workspace(dev)
    out = new_outputs(tr, dev)
    T = tr["seq"].size

    def step():
        opattr.opattr_attribute(dt, flags=flags, outputs=out, ws=ws, raise_strict=False)

    step()
    torch.cuda.synchronize()
    diag = opattr.read_diag(out["diag"])
    if diag["status"] not in (0, -4):
        raise SystemExit(f"{name}/{emission} reported {diag}")
    flush = None
    if flush_mib:
        buf = torch.empty(flush_mib << 18, dtype=torch.int32, device=dev)

        def flush():
            buf.fill_(1)
    ms, per = timed_steps(step, steps, warmup, flush)
    nbytes = algorithmic_bytes(tr)
    med = statistics.median(per)
    row = {"workload": f"{name}: {T} launches, {tr['n_streams']} streams, "
                       f"{tr['r_start'].size} ranges, {tr['n_names']} names, "
                       f"{tr['pf_name'].size} profiled rows, {tr['n_ops']} ops, "
                       f"emission {emission}" + (", validated" if validate else ""),
           "records_per_s": T / (med * 1e-3), "step_ms": spread(per),
           "algorithmic_bytes": nbytes, "frac_of_hbm_peak": nbytes / (med * 1e-3) / 1e9 /
           HBM_PEAK_GBPS}
    if flush_mib:
        row["flush_mib_before_each_step"] = flush_mib
    else:
        row["ms_per_step_back_to_back"] = ms
    if graph:
        gmed, gmin, gmax = graph_step_ms(step, steps)
        row["graph_step_ms"] = {"median": gmed, "min": gmin, "max": gmax}
        row["graph_records_per_s"] = T / (gmed * 1e-3)
    del dt, out, ws
    torch.cuda.empty_cache()
    return row


def main():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", default="large")
    ap.add_argument("--emission", default="stream_major",
                    choices=["stream_major", "seq", "shuffled"])
    ap.add_argument("--validate", action="store_true", help="also check the layout hints")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-next-rows", action="store_true",
                    help="skip timing the walk with range kinds and class discovery")
    ap.add_argument("--no-other-configs", action="store_true",
                    help="skip the rows of the other workloads and orders")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only run a plain copy of MIB MiB (counter calibration)")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus > 1 or world > 1:
        print("bench.py runs on one GPU only: the attribution join of one trace is "
              "measured on a single MI355X; several GPUs would each take a contiguous "
              "share of the launches, aligned to iterations, and exchange per-name counts.",
              file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2609_11938_amd import opattr, tracegen

    if args.copy_calibration:
        copy_calibration(args.copy_calibration, max(1, args.steps))
        return

    if not os.path.exists(opattr.LIB_PATH):
        import __graft_entry__

        __graft_entry__.build()
    dev = "cuda:0"
    torch.cuda.set_device(0)
    t0 = time.perf_counter()
    tr = tracegen.generate(args.config, emission=args.emission)
    gen_s = time.perf_counter() - t0
    print(f"generated {args.config}/{args.emission}: {tracegen.summary(tr)} in {gen_s:.1f}s",
          file=sys.stderr, flush=True)
    dt = opattr.to_device(tr, dev)
    flags = FLAGS[args.emission] | (opattr.VALIDATE if args.validate else 0)
    ws = opattr.Workspace(dev)
    T = tr["seq"].size
    out = new_outputs(tr, dev)

    def step():
        opattr.opattr_attribute(dt, flags=flags, outputs=out, ws=ws, raise_strict=False)

    # 1. the headline: K steps, no probe events inside them
    ms_per_step, per = timed_steps(step, args.steps, args.warmup)
    diag = opattr.read_diag(out["diag"])
    if diag["status"] != 0:
        raise SystemExit(f"attribution reported status {diag['status']}: {diag}")
    value = T / (ms_per_step * 1e-3)
    total_bytes = algorithmic_bytes(tr)
    print(f"timed {args.steps} steps: {ms_per_step:.4f} ms/step", file=sys.stderr, flush=True)

    # 2. every probe recorded once per step (each recorded event is a stream
    # barrier inside the step: per-kernel spans, not the step time)
    nprobe = len(opattr.PROBES)
    ev_all = [_events(2 * nprobe) for _ in range(args.steps)]
    torch.cuda.synchronize()
    for k in range(args.steps):
        opattr.set_probe_events(ev_all[k])
        step()
    torch.cuda.synchronize()
    opattr.set_probe_events(None)
    probe_ms = {}
    for p, name in enumerate(opattr.PROBES):
        d = [ev_all[k][2 * p].elapsed_time(ev_all[k][2 * p + 1]) for k in range(args.steps)]
        probe_ms[name] = statistics.median(d)
    print("probe ms/step: " + ", ".join(f"{n}={v:.4f}" for n, v in probe_ms.items()),
          file=sys.stderr, flush=True)

    fused = args.emission == "stream_major" and T >= 16 * tr["r_start"].size
    table = []
    if fused:
        for kk in fused_kernels(tr):
            ms = probe_ms[kk["probe"]]
            rp = stored_kernel_ms(kk["kernel"], args.config, args.emission)
            per_launch = stored_traffic(kk["kernel"], args.config, args.emission)
            row = dict(kk, probe_ms=ms, GBps=kk["bytes"] / (ms * 1e-3) / 1e9,
                       rocprof_ms=rp,
                       rocprof_frac=(kk["bytes"] / (rp * 1e-3) / 1e9 / HBM_PEAK_GBPS
                                     if rp else None),
                       measured_bytes=per_launch * T if per_launch is not None else None)
            row["frac"] = row["GBps"] / HBM_PEAK_GBPS
            row["traffic_ratio"] = (row["measured_bytes"] / kk["bytes"]
                                    if row["measured_bytes"] else None)
            table.append(row)
        dom = max(table, key=lambda r: r["probe_ms"])
    else:
        dom = None

    # 3. the dominant kernel timed live: K steps with only its probe pair,
    # recorded on the stream it runs on
    roofline = None
    if dom is not None:
        pdom = opattr.PROBES.index(dom["probe"])
        ev_dom = [_events(2) for _ in range(args.steps)]
        torch.cuda.synchronize()
        t_a = time.perf_counter()
        for k in range(args.steps):
            only = [None] * (2 * nprobe)
            only[2 * pdom], only[2 * pdom + 1] = ev_dom[k]
            opattr.set_probe_events(only)
            step()
        torch.cuda.synchronize()
        t_b = time.perf_counter()
        opattr.set_probe_events(None)
        dom_ms = statistics.mean(e0.elapsed_time(e1) for e0, e1 in ev_dom)
        achieved = dom["bytes"] / (dom_ms * 1e-3) / 1e9
        roofline = {"bound": "hbm", "kernel": dom["kernel"], "achieved": achieved,
                    "peak": HBM_PEAK_GBPS, "unit": "GB/s", "frac": achieved / HBM_PEAK_GBPS,
                    "traffic": dom["measured_bytes"], "algorithmic_bytes": dom["bytes"],
                    "avg_ms": dom_ms, "rocprof_avg_ms": dom["rocprof_ms"],
                    "rocprof_frac": dom["rocprof_frac"],
                    "ms_per_step_with_probe": (t_b - t_a) * 1e3 / args.steps}

    copy = copy_bandwidth()
    gmed, gmin, gmax = graph_step_ms(step, args.steps)
    line = {
        "metric": METRIC, "value": value, "unit": "records/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms_per_step,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "int32+f64", "data": "synthetic",
        "config": {"workload": f"{args.config}: {T} kernel launches, "
                               f"{tr['n_streams']} streams, {tr['r_start'].size} ranges, "
                               f"{tr['n_names']} names, {tr['pf_name'].size} profiled rows, "
                               f"{tr['n_ops']} ops, emission {args.emission}",
                   "kernels": int(T), "streams": tr["n_streams"],
                   "ranges": int(tr["r_start"].size), "names": tr["n_names"],
                   "profiled_rows": int(tr["pf_name"].size), "ops": tr["n_ops"],
                   "partitions": tr["n_parts"], "emission": args.emission,
                   "validate": bool(args.validate)},
        "step_ms": spread(per),
        "graph_step_ms": {"median": gmed, "min": gmin, "max": gmax},
        "roofline": roofline,
        "pipeline": {"algorithmic_bytes": total_bytes,
                     "achieved_GBps": total_bytes / (ms_per_step * 1e-3) / 1e9,
                     "frac_of_hbm_peak": total_bytes / (ms_per_step * 1e-3) / 1e9 / HBM_PEAK_GBPS,
                     "graph_frac_of_hbm_peak": total_bytes / (gmed * 1e-3) / 1e9 / HBM_PEAK_GBPS,
                     "copy_GBps": copy["GBps"], "copy_bytes": copy["bytes"]},
        "kernels": table,
        "probe_ms_median": probe_ms,
        "clocks": clocks(),
    }
    if not args.no_next_rows:
        line["next_rows"] = measure_next_rows(dt, tr, flags, args.steps, args.warmup, out, ws)
    if not args.no_other_configs:
        del dt, out, ws
        torch.cuda.empty_cache()
        rows = {}
        for name, emission, validate, graph, flush in (
                ("tiny", "stream_major", False, True, 0),
                ("gpt2", "stream_major", False, True, 0),
                ("sdpa", "stream_major", False, False, 512),
                ("lstm", "stream_major", False, False, 512),
                ("large", "seq", False, False, 0),
                ("large", "shuffled", False, False, 0),
                ("large", "stream_major", True, False, 0)):
            key = f"{name}_{emission}" + ("_validate" if validate else "")
            rows[key] = config_row(name, emission, validate, args.steps, args.warmup, dev,
                                   graph, flush)
            print(f"row {key}: {rows[key]['records_per_s']:.4g} records/s", file=sys.stderr,
                  flush=True)
        line["other_configs"] = rows
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(tr)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
