"""Seeded synthetic trace generator for the trace-attribution join.

Builds the four inputs the attribution join consumes -- a kernel timeline (what a
Nsight-Systems export yields, Sec. 3.1), a profiled counter list (the
application-mode replay rows, Sec. 3.1), operator ranges (the NVTX push/pop
brackets, Sec. 3.5) and a layer-partition class map (Sec. 3.7) -- shaped like the
paper's three workloads (Sec. 4.1, Table "tab:workloads") at five sizes.

This module holds none of the attribution arithmetic. It only constructs inputs,
plus two labels it knows by construction:

* ``planted_range[i]``: the innermost bracket that was open when kernel ``i`` was
  emitted, as an index into the emitted range arrays (-1 if none);
* ``pf_src[j]``: the emitted kernel index whose replay produced profiled row ``j``.

Construction recipe (all draws from ``numpy.random.Generator(PCG64(seed))``):

* ``seq`` is the global launch order 0..T-1. Each stream is serial: a kernel starts
  after the previous kernel on its stream ends plus an idle gap ~ Exp(mean 2000 ns);
  durations are ``clamp(rint(LogNormal(mu, sigma)), 1, 2**32-1)``.
* Names are uniform or finite Zipf, ``P(k) ~ (k+1)**-s`` over ``k < n_names``,
  drawn by inverse CDF.
* Ranges are a random bracket sequence per stream: between two consecutive kernels
  of a stream some brackets close and some open (and, optionally, empty brackets
  open and close), with a depth cap. Every bracket endpoint lies strictly inside an
  inter-kernel gap of its stream and all endpoints are distinct, so no range touches
  another or a kernel start.
* Duplicate layer partitions are structural copies of their class representative:
  the same names and streams per position, fresh durations.
* Counters are Uniform[0, 1) float32, 20 per profiled row.
"""
from __future__ import annotations

import numpy as np

N_COUNTERS = 20
MEAN_GAP_NS = 2000.0
U32_MAX = 2**32 - 1

EMISSIONS = ("stream_major", "seq", "shuffled")

# name -> parameters. "ranges" is the exact total range count.
CONFIGS = {
    # 1 stream, 10k kernels, 50 uniform names, 2000 ranges depth 1-4, ~95% enclosed,
    # profiled list = every launch in order.
    "tiny": dict(kind="random", T=10_000, streams=1, names=50, zipf=None,
                 ranges=2_000, depth=4, p_uncovered=0.05, root=False, empty_rate=0.15,
                 n_ops=200, dur=(8.0, 1.0), drop=0.0, seed=1001),
    # GPT-2 shaped: 12 layers x 40 kernels x 200 iterations on 2 streams,
    # model > layer > op ranges (depth 3), layer dedup N=12, K=1.
    "gpt2": dict(kind="gpt2", T=96_000, streams=2, names=24, layers=12, per_layer=40,
                 iters=200, s1_positions=4, op_ranges_s0=20, uncovered_s0=2,
                 n_op_ids=5_000, dur=(8.0, 1.0), seed=1002),
    # SDPA shaped: 1M kernels, 4 streams, 30 names Zipf(1.2), depth <= 6, a root
    # range per stream (100% of kernel time enclosed), equal invocation counts.
    "sdpa": dict(kind="random", T=1_000_000, streams=4, names=30, zipf=1.2,
                 ranges=250_000, depth=6, p_uncovered=0.0, root=True, empty_rate=0.15,
                 n_ops=500, dur=(8.0, 1.0), drop=0.0, seed=1003),
    # LSTM / black-box shaped: 2M kernels, 8 streams, only ~15% of kernels inside
    # ranges, 5% of launches missing from the profiled list.
    "lstm": dict(kind="random", T=2_000_000, streams=8, names=64, zipf=1.2,
                 ranges=20_000, depth=4, p_uncovered=0.85, root=False, empty_rate=0.15,
                 n_ops=200, dur=(8.0, 1.0), drop=0.05, seed=1004),
    # Large: 10M kernels = 4000 iterations x (50 pre + 48 layers x 50 + 50 post),
    # 16 streams, 500k ranges depth <= 8, 1000 names Zipf(1.1), dedup N=48, K=3.
    "large": dict(kind="large", T=10_000_000, streams=16, names=1_000, zipf=1.1,
                  iters=4_000, pre=50, post=50, layers=48, per_layer=50, classes=3,
                  ranges=500_000, depth=8, p_uncovered=0.05, empty_rate=0.15,
                  n_ops=4_096, dur=(9.0, 1.5), seed=1005),
}


def _rng(seed: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(seed))


def _zipf(rng, n: int, s: float, size) -> np.ndarray:
    w = np.arange(1, n + 1, dtype=np.float64) ** (-s)
    cdf = np.cumsum(w)
    cdf /= cdf[-1]
    u = rng.random(size)
    return np.minimum(np.searchsorted(cdf, u, side="right"), n - 1).astype(np.uint32)


def _names(rng, n: int, zipf, size) -> np.ndarray:
    if zipf is None:
        return rng.integers(0, n, size=size, dtype=np.int64).astype(np.uint32)
    return _zipf(rng, n, zipf, size)


def _durations(rng, mu: float, sigma: float, size) -> np.ndarray:
    x = np.rint(rng.lognormal(mu, sigma, size))
    return np.clip(x, 1, U32_MAX).astype(np.uint32)


def _seg_arange(counts: np.ndarray) -> np.ndarray:
    """Concatenation of arange(c) for every c in counts."""
    counts = np.asarray(counts, dtype=np.int64)
    total = int(counts.sum())
    if total == 0:
        return np.zeros(0, dtype=np.int64)
    starts = np.cumsum(counts) - counts
    return np.arange(total, dtype=np.int64) - np.repeat(starts, counts)


# --------------------------------------------------------------------------- #
# Bracket structure of one stream                                              #
# --------------------------------------------------------------------------- #

def _random_profile(rng, n: int, p_trans: float, depth: int, p_uncovered: float,
                    root: bool, empty_rate: float):
    """Depth profile of one stream as (kernel depth d[n], per-gap closes c, empty
    pairs e, opens o, common depth m), gaps 0..n (gap g precedes kernel g)."""
    lo = 1 if root else 0
    trans = np.zeros(n + 1, dtype=bool)
    trans[0] = True
    if n > 1:
        trans[1:n] = rng.random(n - 1) < p_trans
    n_ep = int(trans[:n].sum())
    # depth of every epoch (run of kernels between two transitions)
    ep_depth = rng.integers(1, depth + 1, size=n_ep)
    if not root:
        ep_depth = np.where(rng.random(n_ep) < p_uncovered, 0, ep_depth)
    epoch = np.cumsum(trans[:n]) - 1
    d = ep_depth[epoch].astype(np.int64)

    d_prev = np.zeros(n + 1, dtype=np.int64)
    d_prev[1:] = d
    d_next = np.zeros(n + 1, dtype=np.int64)
    d_next[:n] = d
    m = np.zeros(n + 1, dtype=np.int64)
    inner = np.flatnonzero(trans[1:n]) + 1
    if inner.size:
        hi = np.minimum(d_prev[inner], d_next[inner])
        m[inner] = lo + np.floor(rng.random(inner.size) * (hi - lo + 1)).astype(np.int64)
    # non-transition gaps keep the depth: c = o = 0
    keep = ~trans
    keep[n] = False
    m[keep] = d_prev[keep]
    m[0] = 0
    m[n] = 0
    c = d_prev - m
    o = d_next - m
    e = np.zeros(n + 1, dtype=np.int64)
    tg = np.flatnonzero(trans)
    tg = tg[(tg < n) & (m[tg] < depth)]
    if empty_rate > 0 and tg.size:
        e[tg] = rng.poisson(empty_rate, size=tg.size)
    return d, c, e, o, m


def _stream_events(c, e, o, m, d_prev, gaplen, base):
    """Token order and times of all bracket events of one stream.

    Within a gap: closes (deepest first), then empty pairs (open, close) at depth
    m+1, then opens (shallowest first). Returns per-event arrays
    (time, is_open, level, gap, is_empty)."""
    E = c + 2 * e + o
    n_gaps = E.size
    gap = np.repeat(np.arange(n_gaps, dtype=np.int64), E)
    j = _seg_arange(E)
    cg, eg, og, mg, dpg = c[gap], e[gap], o[gap], m[gap], d_prev[gap]
    is_close = j < cg
    is_pair = (j >= cg) & (j < cg + 2 * eg)
    is_open_tok = j >= cg + 2 * eg
    level = np.where(is_close, dpg - j,
                     np.where(is_pair, mg + 1, mg + 1 + (j - cg - 2 * eg)))
    is_open = is_open_tok | (is_pair & (((j - cg) % 2) == 0))
    time = base[gap] + ((j + 1) * gaplen[gap]) // (E[gap] + 1)
    return time.astype(np.uint64), is_open, level, gap, is_pair


def _build_stream_ranges(rng, d, c, e, o, m, gaplen, base, n_keep, protect_level1):
    """Turn one stream's bracket profile into ranges. Returns
    (start, end, level, open_gap, keep_ids_in_start_order, planted_local[n])."""
    n = d.size
    d_prev = np.zeros(n + 1, dtype=np.int64)
    d_prev[1:] = d
    time, is_open, level, gap, is_empty = _stream_events(c, e, o, m, d_prev, gaplen, base)
    # events are generated in token order already (gap-major, within-gap order)
    op_idx = np.flatnonzero(is_open)
    cl_idx = np.flatnonzero(~is_open)
    # i-th open at a level pairs with the i-th close at that level (alternation)
    op_ord = op_idx[np.lexsort((op_idx, level[op_idx]))]
    cl_ord = cl_idx[np.lexsort((cl_idx, level[cl_idx]))]
    assert op_ord.size == cl_ord.size
    assert np.array_equal(level[op_ord], level[cl_ord])
    # order ranges by open time (= token order)
    perm = np.argsort(op_ord, kind="stable")
    o_ev = op_ord[perm]
    c_ev = cl_ord[perm]
    r_start = time[o_ev]
    r_end = time[c_ev]
    r_level = level[o_ev]
    r_gap = gap[o_ev]
    r_empty = is_empty[o_ev]
    R0 = r_start.size

    # choose which ranges to keep (exact count), never dropping protected roots
    keep = np.ones(R0, dtype=bool)
    if n_keep < R0:
        cand = np.flatnonzero(~((r_level == 1) & protect_level1))
        n_drop = R0 - n_keep
        if n_drop > cand.size:
            raise ValueError("cannot reach the requested range count")
        drop = rng.choice(cand, size=n_drop, replace=False)
        keep[drop] = False

    # planted innermost: deepest kept range containing each kernel
    planted = np.full(n, -1, dtype=np.int64)
    kidx = np.arange(n, dtype=np.int64)
    ne = ~r_empty
    for lvl in range(1, int(d.max(initial=0)) + 1):
        ids = np.flatnonzero(ne & (r_level == lvl))
        sel = kidx[d >= lvl]
        if sel.size == 0:
            continue
        pos = np.searchsorted(r_gap[ids], sel, side="right") - 1
        cand = ids[pos]
        ok = keep[cand]
        planted[sel[ok]] = cand[ok]
    # renumber kept ranges
    newid = np.cumsum(keep) - 1
    planted = np.where(planted >= 0, newid[np.maximum(planted, 0)], -1)
    kept = np.flatnonzero(keep)
    return r_start[kept], r_end[kept], r_level[kept], r_gap[kept], planted


def _stream_times(rng, n, E, dur, base_t=0):
    """Per-stream start times: serial kernels with an idle gap before each, the gap
    widened so that the E[g] bracket endpoints fit strictly inside it."""
    g = np.rint(rng.exponential(MEAN_GAP_NS, size=n + 1)).astype(np.int64)
    need = np.where(E > 0, E + 1, 0)
    g = np.maximum(g, need)
    dur64 = dur.astype(np.int64)
    # start_k = base + sum_{j<=k} g_j + sum_{j<k} dur_j
    inc = g[:n].copy()
    inc[1:] += dur64[:-1]
    start = base_t + np.cumsum(inc)
    end = start + dur64
    gap_base = np.empty(n + 1, dtype=np.int64)
    gap_base[0] = base_t
    gap_base[1:] = end
    return start.astype(np.uint64), g, gap_base


def _calibrate_p(rng, n, target, depth, p_uncovered, root, empty_rate):
    """Transition probability giving about `target` ranges on a stream of n kernels."""
    if target <= 0 or n <= 1:
        return 0.0
    sim = np.random.Generator(np.random.PCG64(12345))
    k = 200_000
    lo = 1 if root else 0
    a = sim.integers(1, depth + 1, size=k)
    b = sim.integers(1, depth + 1, size=k)
    if not root:
        a = np.where(sim.random(k) < p_uncovered, 0, a)
        b = np.where(sim.random(k) < p_uncovered, 0, b)
    hi = np.minimum(a, b)
    mm = lo + np.floor(sim.random(k) * (hi - lo + 1))
    opens = (b - mm).mean() + empty_rate * (mm < depth).mean()
    return min(1.0, target / max(1e-9, (n - 1) * opens))


def _ranges_for_streams(rng, stream_of_seq, dur_seq, n_streams, cfg, r_total, op_ids_fn):
    """Generic random ranges on every stream; returns per-kernel start (seq order),
    range arrays in stream-major nesting order and planted innermost per kernel."""
    T = stream_of_seq.size
    start_seq = np.zeros(T, dtype=np.uint64)
    planted_seq = np.full(T, -1, dtype=np.int64)
    counts = np.bincount(stream_of_seq, minlength=n_streams).astype(np.int64)
    # exact per-stream split of the range budget, proportional to kernel counts
    share = counts / max(1, counts.sum()) * r_total
    per = np.floor(share).astype(np.int64)
    rem = int(r_total - per.sum())
    if rem > 0:
        order = np.argsort(-(share - per), kind="stable")
        per[order[:rem]] += 1
    rs, re, rstr, rlvl = [], [], [], []
    off = 0
    for s in range(n_streams):
        idx = np.flatnonzero(stream_of_seq == s)
        n = idx.size
        if n == 0:
            continue
        p = _calibrate_p(rng, n, per[s] * 1.08 + 8, cfg["depth"], cfg["p_uncovered"],
                         cfg["root"], cfg["empty_rate"])
        for _ in range(20):
            d, c, e, o, m = _random_profile(rng, n, p, cfg["depth"], cfg["p_uncovered"],
                                            cfg["root"], cfg["empty_rate"])
            R0 = int(o.sum() + e.sum())
            if R0 >= per[s]:
                break
            p = min(1.0, p * 1.25)
        else:
            raise RuntimeError("range calibration failed")
        E = c + 2 * e + o
        st, gaplen, base = _stream_times(rng, n, E, dur_seq[idx])
        s_, e_, lvl, _gap, planted = _build_stream_ranges(
            rng, d, c, e, o, m, gaplen, base, per[s], cfg["root"])
        start_seq[idx] = st
        planted_seq[idx] = np.where(planted >= 0, planted + off, -1)
        rs.append(s_)
        re.append(e_)
        rstr.append(np.full(s_.size, s, dtype=np.uint16))
        rlvl.append(lvl)
        off += s_.size
    r_start = np.concatenate(rs)
    r_end = np.concatenate(re)
    r_stream = np.concatenate(rstr)
    r_level = np.concatenate(rlvl)
    r_op = op_ids_fn(r_level, r_start.size)
    return start_seq, dict(start=r_start, end=r_end, stream=r_stream, op=r_op), planted_seq


# --------------------------------------------------------------------------- #
# Workload builders (all arrays in seq order)                                  #
# --------------------------------------------------------------------------- #

def _gen_random(cfg, rng):
    T, S = cfg["T"], cfg["streams"]
    stream = rng.integers(0, S, size=T, dtype=np.int64).astype(np.uint16)
    name = _names(rng, cfg["names"], cfg["zipf"], T)
    dur = _durations(rng, *cfg["dur"], T)
    n_ops = cfg["n_ops"]
    start, ranges, planted = _ranges_for_streams(
        rng, stream, dur, S, cfg, cfg["ranges"],
        lambda lvl, k: rng.integers(0, n_ops, size=k, dtype=np.int64).astype(np.uint32))
    part = None
    part_rep = None
    eligible = np.ones(T, dtype=bool)
    return dict(stream=stream, name=name, dur=dur, start=start, part=part,
                part_rep=part_rep, eligible=eligible, ranges=ranges,
                planted=planted, n_names=cfg["names"], n_streams=S, n_ops=n_ops,
                n_parts=0, drop=cfg["drop"])


def _gen_gpt2(cfg, rng):
    L, J, I = cfg["layers"], cfg["per_layer"], cfg["iters"]
    T = L * J * I
    assert T == cfg["T"]
    # per-position template shared by every layer
    tmpl_name = rng.integers(0, cfg["names"], size=J, dtype=np.int64).astype(np.uint32)
    tmpl_stream = np.zeros(J, dtype=np.uint16)
    s1 = rng.choice(J, size=cfg["s1_positions"], replace=False)
    tmpl_stream[s1] = 1
    # op grouping of the stream-0 positions: 20 contiguous op groups + 2 uncovered
    n0 = int((tmpl_stream == 0).sum())
    n_groups = cfg["op_ranges_s0"]
    n_unc = cfg["uncovered_s0"]
    parts = n_groups + n_unc
    # random composition of n0 - n_unc kernels into n_groups positive sizes
    cuts = np.sort(rng.choice(np.arange(1, n0 - n_unc), size=n_groups - 1, replace=False))
    sizes = np.diff(np.concatenate([[0], cuts, [n0 - n_unc]]))
    kinds = np.concatenate([np.arange(n_groups), np.full(n_unc, -1)])
    lens = np.concatenate([sizes, np.ones(n_unc, dtype=np.int64)])
    order = rng.permutation(parts)
    kinds, lens = kinds[order], lens[order]
    grp0 = np.repeat(kinds, lens)                  # op group per stream-0 position
    tmpl_grp = np.full(J, -1, dtype=np.int64)
    tmpl_grp[tmpl_stream == 0] = grp0
    tmpl_grp[tmpl_stream == 1] = np.arange(int((tmpl_stream == 1).sum())) + 1000

    pos = np.tile(np.arange(J), L * I)
    layer = np.tile(np.repeat(np.arange(L), J), I)
    it = np.repeat(np.arange(I), L * J)
    name = tmpl_name[pos]
    stream = tmpl_stream[pos]
    dur = _durations(rng, *cfg["dur"], T)
    part = (it * L + layer).astype(np.int32)
    n_parts = I * L
    part_rep = (np.arange(n_parts) // L * L).astype(np.int32)
    eligible = layer == 0

    n_op_ids = cfg["n_op_ids"]
    n_ops = n_op_ids + 1 + L
    start = np.zeros(T, dtype=np.uint64)
    planted = np.full(T, -1, dtype=np.int64)
    rs, re, rstr, rop = [], [], [], []
    off = 0
    for s in range(2):
        idx = np.flatnonzero(stream == s)
        n = idx.size
        g = tmpl_grp[pos[idx]]
        d = np.where(g >= 0, 3, 2).astype(np.int64)
        t_k, l_k = it[idx], layer[idx]
        # common depth between consecutive kernels of this stream
        m = np.zeros(n + 1, dtype=np.int64)
        same_it = t_k[1:] == t_k[:-1]
        same_l = same_it & (l_k[1:] == l_k[:-1])
        same_g = same_l & (g[1:] == g[:-1]) & (g[1:] >= 0)
        m[1:n] = np.where(same_g, 3, np.where(same_l, 2, np.where(same_it, 1, 0)))
        d_prev = np.zeros(n + 1, dtype=np.int64)
        d_prev[1:] = d
        d_next = np.zeros(n + 1, dtype=np.int64)
        d_next[:n] = d
        c = d_prev - m
        o = d_next - m
        e = np.zeros(n + 1, dtype=np.int64)
        E = c + 2 * e + o
        st, gaplen, base = _stream_times(rng, n, E, dur[idx])
        r_s, r_e, lvl, rgap, pl = _build_stream_ranges(
            rng, d, c, e, o, m, gaplen, base, 1 << 62, False)
        first_layer = l_k[np.minimum(rgap, n - 1)]
        ops = np.where(lvl == 1, n_op_ids,
                       np.where(lvl == 2, n_op_ids + 1 + first_layer,
                                rng.integers(0, n_op_ids, size=lvl.size)))
        start[idx] = st
        planted[idx] = np.where(pl >= 0, pl + off, -1)
        rs.append(r_s)
        re.append(r_e)
        rstr.append(np.full(r_s.size, s, dtype=np.uint16))
        rop.append(ops.astype(np.uint32))
        off += r_s.size
    ranges = dict(start=np.concatenate(rs), end=np.concatenate(re),
                  stream=np.concatenate(rstr), op=np.concatenate(rop))
    return dict(stream=stream, name=name, dur=dur, start=start, part=part,
                part_rep=part_rep, eligible=eligible, ranges=ranges, planted=planted,
                n_names=cfg["names"], n_streams=2, n_ops=n_ops, n_parts=n_parts,
                drop=0.0)


def _gen_large(cfg, rng):
    I, L, J, K = cfg["iters"], cfg["layers"], cfg["per_layer"], cfg["classes"]
    pre, post, S = cfg["pre"], cfg["post"], cfg["streams"]
    per_it = pre + L * J + post
    T = I * per_it
    assert T == cfg["T"]
    nn, zs = cfg["names"], cfg["zipf"]
    # fixed templates: pre/post positions and one template per structural class
    pre_name, post_name = _zipf(rng, nn, zs, pre), _zipf(rng, nn, zs, post)
    pre_str = rng.integers(0, S, size=pre, dtype=np.int64)
    post_str = rng.integers(0, S, size=post, dtype=np.int64)
    cls_name = _zipf(rng, nn, zs, (K, J))
    cls_str = rng.integers(0, S, size=(K, J), dtype=np.int64)
    layer_cls = np.arange(L) % K
    it_name = np.concatenate([pre_name, cls_name[layer_cls].reshape(-1), post_name])
    it_str = np.concatenate([pre_str, cls_str[layer_cls].reshape(-1), post_str])
    it_layer = np.concatenate([np.full(pre, -1), np.repeat(np.arange(L), J),
                               np.full(post, -1)])
    name = np.tile(it_name, I).astype(np.uint32)
    stream = np.tile(it_str, I).astype(np.uint16)
    lay = np.tile(it_layer, I)
    it = np.repeat(np.arange(I, dtype=np.int64), per_it)
    part = np.where(lay >= 0, it * L + lay, -1).astype(np.int32)
    n_parts = I * L
    p_ids = np.arange(n_parts)
    part_rep = (p_ids // L * L + (p_ids % L) % K).astype(np.int32)
    eligible = (lay < 0) | (lay < K)
    dur = _durations(rng, *cfg["dur"], T)
    n_ops = cfg["n_ops"]
    rcfg = dict(depth=cfg["depth"], p_uncovered=cfg["p_uncovered"], root=False,
                empty_rate=cfg["empty_rate"])
    start, ranges, planted = _ranges_for_streams(
        rng, stream, dur, S, rcfg, cfg["ranges"],
        lambda lvl, k: rng.integers(0, n_ops, size=k, dtype=np.int64).astype(np.uint32))
    return dict(stream=stream, name=name, dur=dur, start=start, part=part,
                part_rep=part_rep, eligible=eligible, ranges=ranges, planted=planted,
                n_names=nn, n_streams=S, n_ops=n_ops, n_parts=n_parts, drop=0.0)


def generate(config="tiny", seed=None, emission="stream_major", **overrides):
    """Generate one synthetic trace.

    ``config`` is a key of CONFIGS or a dict of parameters; ``overrides`` replace
    entries (e.g. ``T`` for a smaller random trace). Returns a dict of numpy arrays
    in the requested emission order:

    kernels: seq u32, start_ns u64, dur_ns u32, stream_id u16, name_id u32,
             part_id i32 (or None)
    profiled: pf_name u32[P], counters f32[P, 20] (row-major)
    ranges: r_start u64, r_end u64, r_stream u16, r_op u32
    part_rep i32[n_parts] (or None), dims n_names / n_streams / n_ops / n_parts,
    labels planted_range i32[T], pf_src i64[P].
    """
    if emission not in EMISSIONS:
        raise ValueError(f"unknown emission {emission!r}")
    cfg = dict(CONFIGS[config]) if isinstance(config, str) else dict(config)
    cfg.update(overrides)
    if "ranges" in overrides and "T" in overrides and cfg["kind"] != "random":
        raise ValueError("size overrides apply to random configs only")
    if seed is None:
        seed = cfg["seed"]
    rng = _rng(seed)
    kind = cfg["kind"]
    if kind == "random":
        w = _gen_random(cfg, rng)
    elif kind == "gpt2":
        w = _gen_gpt2(cfg, rng)
    elif kind == "large":
        w = _gen_large(cfg, rng)
    else:
        raise ValueError(kind)

    T = w["name"].size
    seq = np.arange(T, dtype=np.uint32)
    # profiled rows: the replay of eligible launches, in launch order, minus drops
    pf_seq = np.flatnonzero(w["eligible"])
    if w["drop"] > 0:
        pf_seq = pf_seq[rng.random(pf_seq.size) >= w["drop"]]
    P = pf_seq.size
    pf_name = w["name"][pf_seq].astype(np.uint32)
    counters = rng.random((P, N_COUNTERS), dtype=np.float32)

    # emission order of kernels and ranges
    rg = w["ranges"]
    if emission == "stream_major":
        korder = np.argsort(w["stream"], kind="stable")
        rorder = np.lexsort((rg["start"], rg["stream"]))
    elif emission == "seq":
        korder = seq.astype(np.int64)
        rorder = np.lexsort((rg["stream"], rg["start"]))
    else:
        prng = _rng(seed + 1)
        korder = prng.permutation(T)
        rorder = prng.permutation(rg["start"].size)
    rinv = np.empty(rorder.size, dtype=np.int64)
    rinv[rorder] = np.arange(rorder.size)
    kinv = np.empty(T, dtype=np.int64)
    kinv[korder] = np.arange(T)
    planted = w["planted"][korder]
    planted = np.where(planted >= 0, rinv[np.maximum(planted, 0)], -1).astype(np.int32)
    out = dict(
        seq=seq[korder].copy(),
        start_ns=w["start"][korder].copy(),
        dur_ns=w["dur"][korder].copy(),
        stream_id=w["stream"][korder].copy(),
        name_id=w["name"][korder].copy(),
        part_id=None if w["part"] is None else w["part"][korder].copy(),
        pf_name=pf_name,
        counters=counters,
        r_start=rg["start"][rorder].copy(),
        r_end=rg["end"][rorder].copy(),
        r_stream=rg["stream"][rorder].copy(),
        r_op=rg["op"][rorder].copy(),
        part_rep=w["part_rep"],
        n_names=int(w["n_names"]), n_streams=int(w["n_streams"]),
        n_ops=int(w["n_ops"]), n_parts=int(w["n_parts"]),
        planted_range=planted,
        pf_src=kinv[pf_seq],
        config=config if isinstance(config, str) else "custom",
        emission=emission, seed=int(seed),
    )
    return out


def summary(tr) -> dict:
    """Sizes of a generated trace (for logs and DESIGN tables)."""
    return dict(T=int(tr["seq"].size), P=int(tr["pf_name"].size), R=int(tr["r_start"].size),
                n_names=tr["n_names"], n_streams=tr["n_streams"], n_ops=tr["n_ops"],
                n_parts=tr["n_parts"])


def with_range_kinds(tr, seed=5, p_skip=0.2):
    """A copy of ``tr`` whose ranges carry enclosure-walk kinds (r_kind u8):
    every outermost range of its stream (contained in no other, like a
    profiler step) is a boundary (1); of the others a fraction ``p_skip`` is
    skipped (2, namespaces the walk passes over) and the rest are operators
    (0)."""
    rng = _rng(seed)
    R = tr["r_start"].size
    kind = np.where(rng.random(R) < p_skip, 2, 0).astype(np.uint8)
    if R:
        rs, re, st = tr["r_start"], tr["r_end"], tr["r_stream"]
        order = np.lexsort((np.arange(R), -re.astype(np.int64), rs, st))
        st_o, re_o = st[order], re[order].astype(np.int64)
        cuts = np.flatnonzero(np.diff(st_o.astype(np.int64))) + 1
        root = np.zeros(R, dtype=bool)
        for a, b in zip(np.r_[0, cuts], np.r_[cuts, R]):
            seg = re_o[a:b]
            prev = np.maximum.accumulate(np.r_[np.int64(-1), seg[:-1]])
            root[a:b] = seg > prev  # ends beyond every earlier range of the stream
        kind[order[root]] = 1
    out = dict(tr)
    out["r_kind"] = kind
    return out


def _range_parents(tr):
    """Per range: the innermost range of its stream that contains it (the
    nearest earlier range in nesting order whose end is not before its own),
    -1 for a root."""
    R = tr["r_start"].size
    rs, re, st = tr["r_start"], tr["r_end"], tr["r_stream"]
    order = np.lexsort((np.arange(R), -re.astype(np.int64), rs, st))
    parent = np.full(R, -1, dtype=np.int64)
    stack = []
    cur = None
    for x in order:
        if st[x] != cur:
            stack, cur = [], st[x]
        while stack and re[stack[-1]] < re[x]:
            stack.pop()
        if stack:
            parent[x] = stack[-1]
        stack.append(x)
    return parent


def with_attribution_maps(tr, seed=7, p_corr=0.4, p_mismatch=0.1, p_none=0.02, p_fmap=0.3,
                          max_fused=3, p_bad=0.0, shuffle=False):
    """A copy of ``tr`` with the two maps of the tiered attribution:

    * a correlation map (``corr_name`` u32, ``corr_op`` i32), as the
      torch.profiler pass would record it: for a fraction ``p_corr`` of the
      kernel names, one entry per launch in launch order, whose operator is
      the one that dispatched the launch: the op of its planted innermost
      range, or with range kinds the first op range outward from it (past
      skipped ranges; none past a boundary), and for a launch no op range
      covers a fixed random op of its kernel name;
      a fraction ``p_none`` of the entries record no operator (-1); for a
      fraction ``p_mismatch`` of those names the last entry is missing (a
      count mismatch); ``shuffle`` interleaves the names at random while
      keeping each name's entries in order;
    * a fusion map (``fmap_off`` u32[n_names + 1], ``fmap_op`` i32): for a
      fraction ``p_fmap`` of the names, 1..``max_fused`` random operators.

    ``p_bad`` of the map entries get an operator id out of range."""
    rng = _rng(seed)
    NN, NOPS = int(tr["n_names"]), int(tr["n_ops"])
    T = tr["seq"].size
    name = np.asarray(tr["name_id"])
    order = np.lexsort((np.arange(T), tr["seq"]))
    order = order[name[order] < NN]
    nm = name[order].astype(np.int64)
    op = rng.integers(0, max(NOPS, 1), size=NN).astype(np.int64)[nm]
    pl = tr.get("planted_range")
    if pl is not None and order.size:
        pr = np.asarray(pl)[order].astype(np.int64)
        kinds = tr.get("r_kind")
        if kinds is not None and pr.size:
            kinds = np.asarray(kinds)
            parent = _range_parents(tr)
            for _ in range(256):  # outward past skipped ranges
                up = (pr >= 0) & (kinds[np.maximum(pr, 0)] == 2)
                if not up.any():
                    break
                pr = np.where(up, parent[np.maximum(pr, 0)], pr)
            pr = np.where((pr >= 0) & (kinds[np.maximum(pr, 0)] == 1), -1, pr)
        op = np.where(pr >= 0, np.asarray(tr["r_op"], dtype=np.int64)[np.maximum(pr, 0)], op)
    covered = rng.random(NN) < p_corr
    keep = covered[nm]
    cn, co = nm[keep], op[keep]
    co = np.where(rng.random(co.size) < p_none, -1, co)
    mism = covered & (rng.random(NN) < p_mismatch)
    last = np.full(NN, -1, dtype=np.int64)
    if cn.size:
        np.maximum.at(last, cn, np.arange(cn.size))
    drop = last[mism]
    sel = np.ones(cn.size, dtype=bool)
    sel[drop[drop >= 0]] = False
    cn, co = cn[sel], co[sel]
    if shuffle and cn.size:
        # a random order of the names, each name's entries still in order
        names_new = cn[rng.permutation(cn.size)]
        by_name = np.argsort(cn, kind="stable")
        start = np.searchsorted(cn[by_name], names_new)
        pos_new = np.argsort(names_new, kind="stable")
        occ = np.empty(cn.size, dtype=np.int64)
        occ[pos_new] = np.arange(cn.size) - np.searchsorted(names_new[pos_new], names_new[pos_new])
        co = co[by_name][start + occ]
        cn = names_new
    if p_bad:
        co = np.where(rng.random(co.size) < p_bad, NOPS + 3, co)
    nf = np.where(rng.random(NN) < p_fmap, rng.integers(1, max_fused + 1, size=NN), 0)
    off = np.zeros(NN + 1, dtype=np.uint32)
    off[1:] = np.cumsum(nf)
    fop = rng.integers(0, max(NOPS, 1), size=int(off[-1])).astype(np.int64)
    if p_bad:
        fop = np.where(rng.random(fop.size) < p_bad, -5, fop)
    out = dict(tr)
    out.update(corr_name=cn.astype(np.uint32), corr_op=co.astype(np.int32), fmap_off=off,
               fmap_op=fop.astype(np.int32))
    return out
