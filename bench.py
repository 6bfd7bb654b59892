#!/usr/bin/env python
"""Throughput of the trace-attribution join on one MI355X.

One step = one opattr_attribute call (invocation-order matching, layer-dedup
broadcast, enclosure, aggregation) over the large synthetic trace: 10M kernel
launches on 16 streams, 500k nested ranges (depth <= 8), 1000 kernel names
Zipf(1.1), layer dedup 48 layers / 3 classes, 1M profiled rows of 20 fp32
counters. Inputs are resident in HBM before the timed region. Prints one JSON
line: records/s, the dominant kernel against the HBM roofline (HIP probe events
recorded by the library around its launches), and the oracle's rate on the
host cores as a reported CPU baseline.
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
    """Compulsory bytes: every input read once, every output written once, at
    the ABI widths (duplicate counter rows reused by dedup count once).
    Returns the step total and, per single-kernel probe, that kernel's bytes."""
    T, P, R = tr["seq"].size, tr["pf_name"].size, tr["r_start"].size
    part = 4 if tr.get("part_id") is not None else 0
    G = tr["n_ops"] + 1
    NP = tr.get("n_parts", 0) or 0
    timeline = T * (4 + 8 + 4 + 2 + 4 + part)      # seq, start, dur, stream, name, part
    profiled = P * (4 + 20 * 4)                     # name + 20 counters
    ranges = R * (8 + 8 + 2 + 4)                    # start, end, stream, op
    outputs = T * (4 + 4)                           # match, range_id
    table = G * 192 + 4 * NP                        # op rows + class map
    per_kernel = {
        # k_seqview_dense: seq in, launch-order view out
        "seq_view": T * (4 + 4),
        # k_tl_hist_w: view, name, partition in
        "tl_hist": T * (4 + 4 + part),
        # k_pf_hist_w: row names in
        "pf_hist": P * 4,
        # k_pf_slot_w: row names in, slot table out
        "pf_slot": P * (4 + 4),
        # k_tl_look (per-tile rank, join and dedup lookup): seq, name,
        # partition in; match out
        "tl_match": T * (4 + 4 + part + 4),
        # k_dedup: partition, name, seq in; match out
        "dedup": T * (4 + 4 + 4 + 4),
        # k_enclose: stream, query point in, range id out; range starts, ends
        # and parents
        "main_pass": T * (2 + 8 + 4) + R * (8 + 8 + 4),
        # k_agg_rows: range id, match, duration of every launch, each range's
        # op id and each profiled counter row once
        "agg_runs": T * (4 + 4 + 4) + R * 4 + P * 80,
    }
    return timeline + profiled + ranges + outputs + table, per_kernel


# kernel behind each single-kernel probe (for the rocprofv3 cross-check)
PROBE_KERNEL = {"seq_view": "k_seqview_dense", "tl_hist": "k_tl_hist_w",
                "pf_hist": "k_pf_hist_w", "pf_slot": "k_pf_slot_w",
                "tl_match": "k_tl_look", "dedup": "k_dedup",
                "main_pass": "k_enclose", "agg_runs": "k_agg_rows"}


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


def cpu_baseline(tr, reps=2):
    from oracle import oracle as O

    O.build(force=False)
    times = []
    for _ in range(reps):
        t0 = time.perf_counter()
        O.attribute(tr)
        times.append(time.perf_counter() - t0)
    med = statistics.median(times)
    return {"value": tr["seq"].size / med, "unit": "records/s", "cores": 1, "kind": "oracle",
            "sample": f"the full workload ({tr['seq'].size} launches), {reps} runs, median "
                      f"{med:.2f} s, single-threaded C oracle"}


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
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only run a plain copy of MIB MiB (counter calibration)")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus > 1 or world > 1:
        print("bench.py runs on one GPU only: the attribution join of one trace is "
              "measured on a single MI355X (see DESIGN.md for how it would shard).",
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
    flags = {"stream_major": opattr.KERNELS_STREAM_MAJOR | opattr.SEQ_DENSE |
             opattr.RANGES_NESTED, "seq": opattr.SEQ_DENSE, "shuffled": 0}[args.emission]
    if args.validate:
        flags |= opattr.VALIDATE
    ws = opattr.Workspace(dev)
    T = tr["seq"].size
    out = opattr.Outputs(
        match=torch.empty(T, dtype=torch.int32, device=dev),
        range_id=torch.empty(T, dtype=torch.int32, device=dev),
        range_depth=None, name_counts=None,
        table=torch.empty((tr["n_ops"] + 1) * 192, dtype=torch.uint8, device=dev),
        summary=torch.empty(40, dtype=torch.uint8, device=dev))

    def step():
        opattr.opattr_attribute(dt, flags=flags, outputs=out, ws=ws, raise_strict=False)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    diag = opattr.read_diag(out["diag"])
    if diag["status"] != 0:
        raise SystemExit(f"attribution reported status {diag['status']}: {diag}")

    # probe events: one start/stop pair per instrumented launch group per step.
    # Every probe is recorded once in an untimed pass (to find the dominant
    # kernel); the timed pass records only the dominant kernel's pair, since
    # each recorded event adds a stream barrier.
    nprobe = len(opattr.PROBES)
    total_bytes, kbytes = algorithmic_bytes(tr)

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
        probe_ms[name] = statistics.mean(d)
    dominant = max(kbytes, key=lambda n: probe_ms[n])
    pdom = opattr.PROBES.index(dominant)

    ev_dom = [_events(2) for _ in range(args.steps)]
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    for k in range(args.steps):
        only = [None] * (2 * nprobe)
        only[2 * pdom], only[2 * pdom + 1] = ev_dom[k]
        opattr.set_probe_events(only)
        step()
    torch.cuda.synchronize()
    t_end = time.perf_counter()
    opattr.set_probe_events(None)

    ms_per_step = (t_end - t_start) * 1e3 / args.steps
    value = T / (ms_per_step * 1e-3)
    # the dominant single-kernel probe sets the roofline line, timed live
    dom_ms = statistics.mean(e0.elapsed_time(e1) for e0, e1 in ev_dom)
    achieved = kbytes[dominant] / (dom_ms * 1e-3) / 1e9
    pipe_gbps = total_bytes / (ms_per_step * 1e-3) / 1e9
    per_launch = stored_traffic(PROBE_KERNEL[dominant], args.config, args.emission)
    traffic = per_launch * T if per_launch is not None else None
    print("probe ms/step: " + ", ".join(f"{n}={v:.4f}" for n, v in probe_ms.items()),
          file=sys.stderr, flush=True)

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
        "roofline": {"bound": "hbm", "kernel": PROBE_KERNEL[dominant], "achieved": achieved,
                     "peak": HBM_PEAK_GBPS, "unit": "GB/s", "frac": achieved / HBM_PEAK_GBPS,
                     "traffic": traffic, "algorithmic_bytes": kbytes[dominant],
                     "avg_ms": dom_ms},
        "pipeline": {"algorithmic_bytes": total_bytes, "achieved_GBps": pipe_gbps,
                     "frac_of_hbm_peak": pipe_gbps / HBM_PEAK_GBPS,
                     "probe_ms_untimed_pass": probe_ms},
    }
    if not args.no_next_rows:
        line["next_rows"] = measure_next_rows(dt, tr, flags, args.steps, args.warmup, out, ws)
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(tr)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
