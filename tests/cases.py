"""Small hand-shaped and random traces for the oracle and parity tests.

Random cases use small integer time axes so that ties occur on purpose:
identical ranges, touching ranges, point ranges, query points equal to a range
endpoint, kernels before and after every range, empty streams.
"""
from __future__ import annotations

import numpy as np

NC = 20


def _nested_intervals(rng, lo, hi, n_target, max_depth):
    """Closed integer intervals inside [lo, hi], properly nested (touching
    siblings, identical and point intervals allowed); about n_target of them."""
    out = []

    def rec(s, e, depth, budget):
        if budget <= 0 or depth > max_depth or len(out) >= n_target:
            return
        k_max = budget if depth == 1 else min(4, budget)
        k = int(rng.integers(1 if depth == 1 else 0, k_max + 1))
        if k == 0:
            return
        pts = np.sort(rng.integers(s, e + 1, size=2 * k))
        for a, b in zip(pts[0::2], pts[1::2]):
            if len(out) >= n_target:
                return
            out.append((int(a), int(b)))
            rec(int(a), int(b), depth + 1, max(1, budget // (2 * k)))

    if n_target > 0:
        rec(lo, hi, 1, n_target)
    return out


def random_trace(seed, T=60, S=3, n_names=5, P=None, R=20, n_ops=7, t_max=60,
                 max_depth=4, nested=True, dedup=False, drop=0.0, extra_pf=0.0,
                 seq_gaps=False):
    rng = np.random.default_rng(seed)
    stream = rng.integers(0, S, size=T).astype(np.uint16)
    name = rng.integers(0, n_names, size=T).astype(np.uint32)
    seq = rng.permutation(T).astype(np.uint32)
    if seq_gaps:
        seq = (seq.astype(np.int64) * 3 + rng.integers(0, 3, size=T)).astype(np.uint32)
    start = rng.integers(0, t_max + 1, size=T).astype(np.uint64)
    dur = rng.integers(1, 1000, size=T).astype(np.uint32)
    part = None
    part_rep = None
    n_parts = 0
    order = np.argsort(seq, kind="stable")
    if dedup:
        # partitions are contiguous runs of launch order; classes copy names
        n_parts = int(rng.integers(2, 7))
        L = max(1, T // (n_parts + 2))
        part_seq = np.full(T, -1, dtype=np.int32)
        pos0 = int(rng.integers(0, 3))
        reps = {}
        part_rep = np.zeros(n_parts, dtype=np.int32)
        n_cls = int(rng.integers(1, 3))
        for p in range(n_parts):
            a = pos0 + p * L
            if a + L > T:
                n_parts = p
                part_rep = part_rep[:p]
                break
            part_seq[a:a + L] = p
            cls = p % n_cls
            if cls not in reps:
                reps[cls] = p
            part_rep[p] = reps[cls]
        part = np.empty(T, dtype=np.int32)
        part[order] = part_seq
        # duplicates copy the representative's names position by position
        name_seq = name[order].copy()
        for p in range(n_parts):
            r = part_rep[p]
            if r != p:
                name_seq[pos0 + p * L:pos0 + (p + 1) * L] = name_seq[pos0 + r * L:pos0 + (r + 1) * L]
        name[order] = name_seq
        if n_parts == 0:
            part, part_rep = None, None
    # profiled rows: eligible launches in seq order, with drops / extras
    elig = np.ones(T, dtype=bool)
    if part is not None:
        pp = part
        elig = (pp < 0) | (part_rep[np.maximum(pp, 0)] == pp)
    pf_seq = [i for i in order if elig[i] and rng.random() >= drop]
    pf_name = name[np.array(pf_seq, dtype=np.int64)] if pf_seq else np.zeros(0, np.uint32)
    if extra_pf > 0:
        k = int(extra_pf * max(1, len(pf_name)))
        ins = rng.integers(0, n_names, size=k).astype(np.uint32)
        pos = rng.integers(0, len(pf_name) + 1, size=k)
        pf_name = np.insert(pf_name, pos, ins)
    pf_name = pf_name.astype(np.uint32)
    if P is not None:
        pf_name = pf_name[:P]
    counters = rng.random((pf_name.size, NC), dtype=np.float32)
    # ranges
    rs, re, rstr = [], [], []
    per = np.bincount(rng.integers(0, S, size=R), minlength=S)
    for s in range(S):
        if nested:
            iv = _nested_intervals(rng, 0, t_max, int(per[s]), max_depth)
        else:
            a = rng.integers(0, t_max + 1, size=int(per[s]))
            b = a + rng.integers(0, t_max // 3 + 1, size=int(per[s]))
            iv = list(zip(a.tolist(), b.tolist()))
        for a, b in iv:
            rs.append(a)
            re.append(b)
            rstr.append(s)
    Rn = len(rs)
    rperm = rng.permutation(Rn)
    r_start = np.array(rs, dtype=np.uint64)[rperm] if Rn else np.zeros(0, np.uint64)
    r_end = np.array(re, dtype=np.uint64)[rperm] if Rn else np.zeros(0, np.uint64)
    r_stream = np.array(rstr, dtype=np.uint16)[rperm] if Rn else np.zeros(0, np.uint16)
    r_op = rng.integers(0, n_ops, size=Rn).astype(np.uint32)
    return dict(seq=seq, start_ns=start, dur_ns=dur, stream_id=stream, name_id=name,
                part_id=part, pf_name=pf_name, counters=counters, r_start=r_start,
                r_end=r_end, r_stream=r_stream, r_op=r_op, part_rep=part_rep,
                n_names=n_names, n_streams=S, n_ops=n_ops, n_parts=n_parts)


def stream_major(tr):
    """Re-emit a trace's kernels in (stream, seq) order and its ranges in
    (stream, start asc, end desc, index asc) nesting order; returns the new
    trace and the permutations (new position -> old index)."""
    korder = np.lexsort((tr["seq"], tr["stream_id"]))
    rorder = np.lexsort((np.arange(tr["r_start"].size), -tr["r_end"].astype(np.float64),
                         tr["r_start"], tr["r_stream"])) if tr["r_start"].size else \
        np.zeros(0, dtype=np.int64)
    out = dict(tr)
    for k in ("seq", "start_ns", "dur_ns", "stream_id", "name_id", "part_id", "query_ns"):
        if out.get(k) is not None:
            out[k] = np.ascontiguousarray(out[k][korder])
    for k in ("r_start", "r_end", "r_stream", "r_op", "r_kind"):
        if out.get(k) is not None:
            out[k] = np.ascontiguousarray(out[k][rorder])
    return out, korder, rorder


def with_kinds(tr, seed, p_boundary=0.2, p_skip=0.25, p_bad=0.0, roots_boundary=False):
    """A copy of tr whose ranges carry enclosure-walk kinds (0 op, 1 boundary,
    2 skip; p_bad of them an invalid kind 3). With roots_boundary, ranges
    that no other range contains become boundaries (profiler steps)."""
    rng = np.random.default_rng(seed)
    R = tr["r_start"].size
    u = rng.random(R)
    kind = np.where(u < p_boundary, 1, np.where(u < p_boundary + p_skip, 2, 0)).astype(np.uint8)
    if roots_boundary and R:
        rs, re, st = tr["r_start"], tr["r_end"], tr["r_stream"]
        order = np.lexsort((np.arange(R), -re.astype(np.int64), rs, st))
        top_end = {}
        for x in order:
            s = int(st[x])
            if s not in top_end or int(re[x]) > top_end[s]:
                kind[x] = 1
                top_end[s] = int(re[x])
    if p_bad:
        kind[rng.random(R) < p_bad] = 3
    out = dict(tr)
    out["r_kind"] = kind
    return out


def class_trace(seed, T=90, n_parts=9, noncontig=False, bad=False, S=3, n_names=4,
                seq_gaps=None):
    """Partitions as consecutive launch-order runs; some copy the (name,
    stream) sequence of an earlier one, some differ in one stream or name."""
    rng = np.random.default_rng(seed)
    if seq_gaps is None:
        seq_gaps = seed % 2 == 0
    tr = random_trace(seed, T=T, S=S, n_names=n_names, R=4, seq_gaps=seq_gaps)
    order = np.argsort(tr["seq"], kind="stable")
    L = T // (n_parts + 1)
    part_seq = np.full(T, -1, np.int32)
    name_seq = tr["name_id"][order].copy()
    st_seq = tr["stream_id"][order].copy()
    for p in range(n_parts):
        a = p * L + 2
        part_seq[a:a + L] = p
        src = int(rng.integers(0, p + 1))
        if src < p and rng.random() < 0.7:
            b = src * L + 2
            name_seq[a:a + L] = name_seq[b:b + L]
            st_seq[a:a + L] = st_seq[b:b + L]
            if rng.random() < 0.3:  # a near copy: one stream differs
                st_seq[a + int(rng.integers(0, L))] ^= 1
    if noncontig:
        part_seq[2 * L + 2 + L // 2] = -1  # a hole in partition 2
    if bad:
        name_seq[5 * L + 3] = tr["n_names"] + 1  # a launch with a bad name
    tr["part_id"] = np.empty(T, np.int32)
    tr["part_id"][order] = part_seq
    tr["name_id"] = tr["name_id"].copy()
    tr["name_id"][order] = name_seq
    tr["stream_id"] = tr["stream_id"].copy()
    tr["stream_id"][order] = st_seq
    tr["n_parts"] = n_parts
    tr["part_rep"] = None
    return tr
