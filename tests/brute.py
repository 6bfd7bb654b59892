"""Brute-force restatements of the join's definitions, for tiny inputs only.

Each function recomputes a stage from its definition by exhaustive search,
without sorting tricks, stacks or sweeps, so that it shares no algorithm with
the oracle it checks.
"""
from __future__ import annotations

import math

import numpy as np

NC = 20
SUM, DWMEAN, MAX = 0, 1, 2
DEFAULT_KIND = [SUM, SUM, SUM, DWMEAN, DWMEAN, DWMEAN, DWMEAN, DWMEAN, DWMEAN, DWMEAN,
                SUM, DWMEAN, DWMEAN, DWMEAN, SUM, DWMEAN, DWMEAN, MAX, SUM, MAX]


def eligible(tr, i):
    part = tr.get("part_id")
    if part is None or tr.get("part_rep") is None:
        return True
    p = int(part[i])
    return p < 0 or int(tr["part_rep"][p]) == p


def iom(tr, policy=0):
    """match[i] = the profiled row of the same name whose replay ordinal equals
    the number of earlier (by seq) eligible launches of that name."""
    T = tr["seq"].size
    name, seq, pf = tr["name_id"], tr["seq"], tr["pf_name"]
    match = np.full(T, -1, dtype=np.int64)
    tl = {}
    pfc = {}
    for n in pf.tolist():
        pfc[n] = pfc.get(n, 0) + 1
    for i in range(T):
        if eligible(tr, i):
            tl[int(name[i])] = tl.get(int(name[i]), 0) + 1
    for i in range(T):
        if not eligible(tr, i):
            continue
        n = int(name[i])
        rank = sum(1 for j in range(T)
                   if j != i and eligible(tr, j) and name[j] == n and seq[j] < seq[i])
        rows = [j for j in range(pf.size) if pf[j] == n]
        if rank < len(rows):
            match[i] = rows[rank]
        if policy == 1 and tl.get(n, 0) != pfc.get(n, 0):
            match[i] = -1
    return match


def dedup(tr, match):
    """Duplicates take the match of the representative's kernel at the same
    launch-order position of their partition (name must agree)."""
    part, rep = tr.get("part_id"), tr.get("part_rep")
    out = match.copy()
    errors = 0
    if part is None or rep is None:
        return out, errors
    T = part.size
    seq, name = tr["seq"], tr["name_id"]

    def members(p):
        return sorted([i for i in range(T) if part[i] == p], key=lambda i: int(seq[i]))

    for i in range(T):
        p = int(part[i])
        if p < 0 or int(rep[p]) == p:
            continue
        r = int(rep[p])
        mp, mr = members(p), members(r)
        pos = mp.index(i)
        if int(rep[r]) == r and pos < len(mr) and name[mr[pos]] == name[i]:
            out[i] = match[mr[pos]]
        else:
            out[i] = -1
            errors += 1
    return out, errors


def enclose(tr):
    """range_id[i] = argmax over ranges r on kernel i's stream with
    s_r <= q_i <= e_r of (s_r, -e_r, r); -1 if none."""
    T = tr["seq"].size
    q = tr.get("query_ns")
    q = tr["start_ns"] if q is None else q
    rs, re, rst = tr["r_start"], tr["r_end"], tr["r_stream"]
    out = np.full(T, -1, dtype=np.int64)
    for i in range(T):
        best = None
        for r in range(rs.size):
            if rst[r] == tr["stream_id"][i] and rs[r] <= q[i] <= re[r]:
                key = (int(rs[r]), -int(re[r]), r)
                if best is None or key > best:
                    best = key
        if best is not None:
            out[i] = best[2]
    return out


def dedup_classes(tr):
    """Per partition: the lowest-numbered partition whose launches (valid
    name and partition) form the same (name, stream) sequence in launch
    order; a partition whose launches are not consecutive in launch order
    (among all launches, by seq then index) is its own class."""
    NP = int(tr.get("n_parts", 0) or 0)
    part, seq, name, st = tr["part_id"], tr["seq"], tr["name_id"], tr["stream_id"]
    T = seq.size
    order = sorted(range(T), key=lambda i: (int(seq[i]), i))
    rank = {i: x for x, i in enumerate(order)}
    members = [[] for _ in range(NP)]
    for i in order:
        p = int(part[i])
        if 0 <= p < NP and int(name[i]) < tr["n_names"]:
            members[p].append(i)
    contig = [not m or rank[m[-1]] - rank[m[0]] + 1 == len(m) for m in members]
    seqs = [[(int(name[i]), int(st[i])) for i in m] for m in members]
    rep = list(range(NP))
    for q in range(NP):
        if not contig[q]:
            continue
        for r in range(q):
            if contig[r] and seqs[r] == seqs[q]:
                rep[q] = r
                break
    return np.array(rep, dtype=np.int64), any(not c for c in contig)


def _range_valid(tr, r):
    kind = tr.get("r_kind")
    return (int(tr["r_stream"][r]) < tr["n_streams"] and int(tr["r_op"][r]) < tr["n_ops"]
            and int(tr["r_start"][r]) <= int(tr["r_end"][r]) < 2 ** 63
            and (kind is None or int(kind[r]) <= 2))


def enclosing_lists(tr):
    """Per kernel: every valid range of its stream whose closed interval holds
    its query point, innermost first (reverse nesting order)."""
    T, R = tr["seq"].size, tr["r_start"].size
    q = tr.get("query_ns")
    q = tr["start_ns"] if q is None else q
    rs, re, rst = tr["r_start"], tr["r_end"], tr["r_stream"]
    out = []
    for i in range(T):
        enc = [r for r in range(R) if _range_valid(tr, r) and rst[r] == tr["stream_id"][i]
               and tr["stream_id"][i] < tr["n_streams"] and int(rs[r]) <= int(q[i]) <= int(re[r])]
        enc.sort(key=lambda r: (int(rs[r]), -int(re[r]), r))
        out.append(enc[::-1])
    return out


def enclose_walk(tr):
    """Alg. 2 written out per kernel: the valid ranges of its stream that
    contain its query point, outermost first in nesting order, are walked
    from the innermost outward; kind 0 (op) ranges are collected, kind 2 is
    passed over, kind 1 ends the walk. Returns range_id (first op collected),
    fused (more than one collected), range_any (innermost of any kind) and,
    per range, range_parent (innermost valid range of the same stream that
    contains it and precedes it in nesting order)."""
    T, R = tr["seq"].size, tr["r_start"].size
    q = tr.get("query_ns")
    q = tr["start_ns"] if q is None else q
    kind = tr.get("r_kind")
    rs, re, rst = tr["r_start"], tr["r_end"], tr["r_stream"]
    rid = np.full(T, -1, dtype=np.int64)
    fused = np.zeros(T, dtype=np.int64)
    rany = np.full(T, -1, dtype=np.int64)
    for i in range(T):
        enc = [r for r in range(R) if _range_valid(tr, r) and rst[r] == tr["stream_id"][i]
               and int(rs[r]) <= int(q[i]) <= int(re[r])]
        enc.sort(key=lambda r: (int(rs[r]), -int(re[r]), r))  # outermost first
        if enc:
            rany[i] = enc[-1]
        ops = []
        for r in reversed(enc):
            k = 0 if kind is None else int(kind[r])
            if k == 0:
                ops.append(r)
            elif k == 1:
                break
        if ops:
            rid[i] = ops[0]
            fused[i] = 1 if len(ops) > 1 else 0
    par = np.full(R, -1, dtype=np.int64)
    for x in range(R):
        if not _range_valid(tr, x):
            continue
        best = None
        for y in range(R):
            if (y != x and _range_valid(tr, y) and rst[y] == rst[x]
                    and int(rs[y]) <= int(rs[x]) and int(re[x]) <= int(re[y])
                    and nesting_before(tr, y, x)):
                key = (int(rs[y]), -int(re[y]), y)
                if best is None or key > best:
                    best = key
        if best is not None:
            par[x] = best[2]
    return rid, fused, rany, par


def nesting_before(tr, a, b):
    """True if range a precedes range b in nesting order (start asc, end desc,
    index asc)."""
    ka = (int(tr["r_start"][a]), -int(tr["r_end"][a]), a)
    kb = (int(tr["r_start"][b]), -int(tr["r_end"][b]), b)
    return ka < kb


def depth(tr):
    """1 + depth of the nearest range earlier in nesting order on the same
    stream whose end is not before this range's end (it contains this one)."""
    R = tr["r_start"].size
    order = sorted(range(R), key=lambda r: (int(tr["r_stream"][r]), int(tr["r_start"][r]),
                                            -int(tr["r_end"][r]), r))
    d = {}
    for pos, r in enumerate(order):
        par = None
        for q in reversed(order[:pos]):
            if tr["r_stream"][q] != tr["r_stream"][r]:
                break
            if tr["r_end"][q] >= tr["r_end"][r]:
                par = q
                break
        d[r] = 1 if par is None else d[par] + 1
    return np.array([d[r] for r in range(R)], dtype=np.int64)


def containers(tr):
    """Number of ranges containing each range (itself included), identical
    intervals nesting in index order."""
    R = tr["r_start"].size
    out = np.zeros(R, dtype=np.int64)
    for r in range(R):
        for a in range(R):
            if tr["r_stream"][a] != tr["r_stream"][r]:
                continue
            if tr["r_start"][a] <= tr["r_start"][r] and tr["r_end"][a] >= tr["r_end"][r] \
                    and (a == r or nesting_before(tr, a, r)):
                out[r] += 1
    return out


def crossing_streams(tr):
    """Streams holding two ranges with s_A < s_B < e_A < e_B."""
    R = tr["r_start"].size
    bad = set()
    s, e, st = tr["r_start"], tr["r_end"], tr["r_stream"]
    for a in range(R):
        for b in range(R):
            if st[a] == st[b] and s[a] < s[b] < e[a] < e[b]:
                bad.add(int(st[a]))
    return bad


def aggregate(tr, match, range_id, agg_kind=None, absent_mask=0):
    """Per operator: counts and ns sums, and per counter the correctly rounded
    (math.fsum) SUM, duration-weighted mean (Eq. 1) or MAX over matched
    kernels."""
    T = tr["seq"].size
    group = [int(tr["r_op"][int(range_id[i])]) if int(range_id[i]) >= 0 else tr["n_ops"]
             for i in range(T)]
    return aggregate_groups(tr, match, group, tr["n_ops"] + 1, agg_kind, absent_mask)


def dispatch_keys(tr, range_id, op=None):
    """Per kernel, its row of the per-dispatch table: its range when the
    kernel's operator is the range's operator, else R + its operator, else
    (unattributed) R + n_ops."""
    R, NOPS = tr["r_start"].size, tr["n_ops"]
    keys = []
    for i in range(tr["seq"].size):
        r = int(range_id[i])
        o = int(op[i]) if op is not None else (int(tr["r_op"][r]) if r >= 0 else -1)
        if r >= 0 and 0 <= o < NOPS and o == int(tr["r_op"][r]):
            keys.append(r)
        elif 0 <= o < NOPS:
            keys.append(R + o)
        else:
            keys.append(R + NOPS)
    return keys


def aggregate_groups(tr, match, group, G, agg_kind=None, absent_mask=0):
    """The same reduction over given groups (group[i] in [0, G))."""
    kind = DEFAULT_KIND if agg_kind is None else list(agg_kind)
    T = tr["seq"].size
    groups = [[] for _ in range(G)]
    for i in range(T):
        groups[group[i]].append(i)
    rows = []
    dur = tr["dur_ns"]
    cnt = tr["counters"]
    for g in range(G):
        ks = groups[g]
        mk = [i for i in ks if match[i] >= 0]
        row = dict(kernel_count=len(ks), total_ns=sum(int(dur[i]) for i in ks),
                   matched_count=len(mk), matched_ns=sum(int(dur[i]) for i in mk))
        vals = []
        for c in range(NC):
            if (absent_mask >> c) & 1 or not mk:
                vals.append(math.nan)
                continue
            ms = [float(cnt[match[i], c]) for i in mk]
            if kind[c] == SUM:
                vals.append(math.fsum(ms))
            elif kind[c] == DWMEAN:
                num = math.fsum(m * float(dur[i]) for m, i in zip(ms, mk))
                vals.append(num / float(row["matched_ns"]) if row["matched_ns"] else math.nan)
            else:
                vals.append(max(ms))
        row["value"] = vals
        rows.append(row)
    return rows


def tiers(tr, policy=1):
    """The decision tree per kernel, from the definitions: the invocation
    index of a launch is its rank among all launches of its (valid) name by
    (seq, index); entry k of a name in the correlation map is its index k;
    under policy 1 (SKIP_NAME) a name whose entry count differs from its
    launch count has no entries. Then HIGH (entry with a valid operator), NVTX
    (the walk's range), FUSION (first listed operator valid), UNATTRIBUTED.
    Returns tier, op, fused and per-tier (count, ns)."""
    T, NN, NOPS = tr["seq"].size, tr["n_names"], tr["n_ops"]
    name = [int(v) for v in tr["name_id"]]
    order = sorted(range(T), key=lambda i: (int(tr["seq"][i]), i))
    index, launches = {}, {}
    for i in order:
        n = name[i]
        if n < NN:
            index[i] = launches.get(n, 0)
            launches[n] = index[i] + 1
    entries = {}
    cn = tr.get("corr_name")
    if cn is not None:
        for j in range(cn.size):
            if int(cn[j]) < NN:
                entries.setdefault(int(cn[j]), []).append(int(tr["corr_op"][j]))
    fo, fop = tr.get("fmap_off"), tr.get("fmap_op")
    rid, wfused, _, _ = enclose_walk(tr)
    tier = np.zeros(T, dtype=np.int64)
    op = np.full(T, -1, dtype=np.int64)
    fused = np.zeros(T, dtype=np.int64)
    cnt, ns = [0] * 4, [0] * 4
    for i in range(T):
        n = name[i]
        ent = None
        if cn is not None and n < NN:
            lst = entries.get(n, [])
            if (policy != 1 or len(lst) == launches.get(n, 0)) and index[i] < len(lst):
                ent = lst[index[i]]
        fl = []
        if fo is not None and n < NN and int(fo[n + 1]) > int(fo[n]):
            fl = [int(v) for v in fop[int(fo[n]):int(fo[n + 1])]]
        if ent is not None and 0 <= ent < NOPS:
            tier[i], op[i] = 1, ent
        elif rid[i] >= 0:
            tier[i], op[i] = 2, int(tr["r_op"][rid[i]])
        elif fl and 0 <= fl[0] < NOPS:
            tier[i], op[i] = 3, fl[0]
        fused[i] = 1 if (wfused[i] or len(fl) > 1) else 0
        cnt[tier[i]] += 1
        ns[tier[i]] += int(tr["dur_ns"][i])
    return tier, op, fused, cnt, ns
