"""profile.json: the attribution's output document (App. A.4 schema), built on
the host from the library's outputs.

One entry in ``operators`` per operator dispatch with kernels (a row of the
per-dispatch table, opattr_aggregate_dispatch): ``operator_id`` is the
operator name and its call index, ``kernels`` the dispatch's kernel records
(name, attribution method and confidence from the tier, duration, stream,
the matched profiled row's 20 counters), ``aggregated`` the dispatch's row of
the table (Eq. 1); kernels no tier attributes go to ``unattributed_kernels``.
This module formats; every number in it comes from the library's outputs
and the trace.
"""
from __future__ import annotations

import json
import math

import numpy as np

SCHEMA_VERSION = "1.0"

# the 20 counters (counter appendix table, rows 1..20) by their profile field
# names; row 13 is spelled as in the schema's listing
COUNTER_FIELDS = (
    "gpu_time_duration_ns", "dram_bytes_read", "dram_bytes_written", "memory_throughput_pct",
    "dram_throughput_pct", "mem_busy_pct", "l1_hit_rate", "l2_hit_rate", "sm_throughput_pct",
    "tensor_core_active_pct", "sm_active_cycles", "achieved_occupancy",
    "warp_cycles_per_instruction", "eligible_cycles_pct", "executed_instructions", "ipc_active",
    "avg_threads_per_warp", "registers_per_thread", "local_memory_spills",
    "dynamic_smem_per_block")

# attribution tiers (OPATTR_TIER_*): method and confidence as in the schema
TIER_METHOD = {0: "unattributed", 1: "torch_profiler_correlation", 2: "nvtx",
               3: "inductor_fusion"}
TIER_CONFIDENCE = {0: None, 1: "high", 2: "medium", 3: "medium"}


def _num(v):
    """JSON number, or null for NaN."""
    v = float(v)
    return None if math.isnan(v) else v


def _call_indices(r_start, r_stream, r_op, n_ops):
    """Dispatch ordinal of every range among the ranges of its operator (by
    start, stream, index), and the count of ranges per operator."""
    R = r_op.size
    order = np.lexsort((np.arange(R), r_stream, r_start, r_op))
    ops = r_op[order].astype(np.int64)
    first = np.searchsorted(ops, ops)  # first position of each op's group
    call = np.empty(R, dtype=np.int64)
    call[order] = np.arange(R) - first
    per_op = np.bincount(ops[ops < n_ops], minlength=n_ops) if R else np.zeros(n_ops, np.int64)
    return call, per_op


def build(trace: dict, match, tier, op, fused, row, table, range_any=None, range_parent=None,
          op_names=None, kernel_names=None, metadata=None, absent_mask=0) -> dict:
    """The profile document.

    trace: host arrays (seq, dur_ns, stream_id, name_id, counters, r_start,
    r_stream, r_op, optional r_kind, fmap_off/fmap_op) and n_ops. match,
    tier, op, fused, row: per launch (row = the per-dispatch table row from
    opattr_aggregate_dispatch); table: that table (opattr_op_row records, R +
    n_ops + 1 rows). range_any / range_parent (from opattr_enclose_walk), when
    given, add the other op ranges a fused kernel's walk passes to
    ``fused_with``. op_names[o] / kernel_names[n] default to "aten::op<o>" and
    "kernel_<n>"."""
    seq = np.asarray(trace["seq"])
    dur = np.asarray(trace["dur_ns"])
    stream = np.asarray(trace["stream_id"])
    name = np.asarray(trace["name_id"])
    counters = np.asarray(trace["counters"])
    r_op = np.asarray(trace["r_op"]).astype(np.int64)
    R, NOPS = r_op.size, int(trace["n_ops"])
    match, tier, op, fused, row = (np.asarray(a) for a in (match, tier, op, fused, row))
    opn = (lambda o: op_names[o]) if op_names is not None else (lambda o: f"aten::op{o}")
    kn = (lambda n: kernel_names[n]) if kernel_names is not None else (lambda n: f"kernel_{n}")
    call, per_op = _call_indices(np.asarray(trace["r_start"]), np.asarray(trace["r_stream"]),
                                 r_op, NOPS)
    width = max(5, len(str(int(seq.max())))) if seq.size else 5
    fo, fop = trace.get("fmap_off"), trace.get("fmap_op")
    kinds = trace.get("r_kind")

    def kernel(i):
        m = int(match[i])
        metrics = None
        if m >= 0:
            vals = counters[m]
            metrics = {f: (None if (absent_mask >> c) & 1 else _num(vals[c]))
                       for c, f in enumerate(COUNTER_FIELDS)}
        t = int(tier[i])
        return {"kernel_id": f"k_{int(seq[i]):0{width}d}", "kernel_name": kn(int(name[i])),
                "attribution_method": TIER_METHOD[t], "confidence": TIER_CONFIDENCE[t],
                "duration_ns": int(dur[i]), "stream_id": int(stream[i]), "metrics": metrics}

    def co_fused(ks, own):
        """operators fused with the dispatch's own: the fusion map's lists for
        its kernel names, and the op ranges on a fused kernel's walk"""
        ops = set()
        for i in ks:
            if not fused[i]:
                continue
            n = int(name[i])
            if fo is not None and n + 1 < len(fo) and fo[n + 1] > fo[n]:
                ops.update(int(v) for v in fop[int(fo[n]):int(fo[n + 1])])
            if range_any is not None and range_parent is not None:
                r = int(range_any[i])
                while r >= 0:
                    k = 0 if kinds is None else int(kinds[r])
                    if k == 1:
                        break
                    if k == 0:
                        ops.add(int(r_op[r]))
                    r = int(range_parent[r])
        ops.discard(own)
        return [opn(o) for o in sorted(o for o in ops if 0 <= o < NOPS)]

    def aggregated(g):
        rec = table[g]
        out = {"total_duration_ns": int(rec["total_ns"]), "kernel_count": int(rec["kernel_count"])}
        for c, f in enumerate(COUNTER_FIELDS):
            out[f] = _num(rec["value"][c])
        return out

    order = np.lexsort((seq, row))
    rows_sorted = row[order]
    cut = np.flatnonzero(np.diff(rows_sorted)) + 1
    groups = np.split(order, cut) if order.size else []
    entries = []
    unattributed = []
    for ks in groups:
        g = int(row[ks[0]])
        if g >= R + NOPS:
            unattributed = [kernel(i) for i in ks]
            continue
        own = int(r_op[g]) if g < R else g - R
        ci = int(call[g]) if g < R else int(per_op[own])
        entries.append((int(seq[ks[0]]), {
            "operator_id": f"{opn(own)}_{ci}", "operator_name": opn(own), "call_index": ci,
            "is_fused": bool(fused[ks].any()), "fused_with": co_fused(ks, own),
            "kernels": [kernel(i) for i in ks], "aggregated": aggregated(g)}))
    entries.sort(key=lambda e: e[0])
    md = {"model_name": "synthetic", "device_name": "AMD Instinct MI355X",
          "compile_mode": "n/a", "capture_timestamp_utc": None}
    md.update(metadata or {})
    return {"schema_version": SCHEMA_VERSION, "capture_metadata": md,
            "operators": [e for _, e in entries], "unattributed_kernels": unattributed}


def write(path: str, doc: dict) -> None:
    """Write the document as JSON (NaN never appears: absent values are null)."""
    with open(path, "w") as f:
        json.dump(doc, f, allow_nan=False, indent=1)
