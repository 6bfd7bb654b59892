"""Pins of the oracle against what the paper and mathematics fix.

The oracle is checked against: brute-force restatements of each definition on
tiny inputs (tests/brute.py), values printed in the paper (tests/golden/),
closed forms, labels the generator planted by construction, and invariants.
"""
import json
import math
import os

import numpy as np
import pytest

import brute
import cases
from oracle import oracle as O
from paper_2609_11938_amd import tracegen as tg

GOLD = os.path.join(os.path.dirname(__file__), "golden")


@pytest.fixture(scope="module", autouse=True)
def _built():
    O.build(force=False)


# --------------------------------------------------------------------------- #
# invocation-order matching (Alg. 1)                                           #
# --------------------------------------------------------------------------- #

@pytest.mark.parametrize("seed", range(40))
def test_iom_matches_brute_force(seed):
    tr = cases.random_trace(seed, T=50, drop=0.15 if seed % 3 else 0.0,
                            extra_pf=0.1 if seed % 4 == 1 else 0.0,
                            dedup=seed % 5 == 2, seq_gaps=seed % 2 == 1)
    for policy in (O.PREFIX, O.SKIP_NAME, O.STRICT):
        got = O.attribute(tr, policy=policy, stages=["match"])
        want = brute.iom(tr, policy=1 if policy == O.SKIP_NAME else 0)
        np.testing.assert_array_equal(got["match_iom"], want)


def test_iom_closed_form_identity():
    """Profiled list = every launch in launch order: the k-th launch of a name
    takes the k-th row of that name, which is row seq itself."""
    for cfg in ("tiny", "sdpa"):
        tr = tg.generate(cfg)
        out = O.attribute(tr, stages=["match"])
        np.testing.assert_array_equal(out["match"], tr["seq"].astype(np.int32))


def test_iom_planted_source_rows():
    """Without drops each profiled row matches the launch that produced it."""
    tr = tg.generate("gpt2")
    m = O.attribute(tr, stages=["match"])["match_iom"]
    want = np.full(m.size, -1)
    want[tr["pf_src"]] = np.arange(tr["pf_src"].size)
    np.testing.assert_array_equal(m, want)


def test_iom_prefix_with_drops_independent_path():
    """With replay rows missing (LSTM-shaped trace, at a smaller size) each name
    matches its first min(tl, pf) launches to its rows in order."""
    tr = tg.generate("lstm", T=50_000, ranges=500)
    out = O.attribute(tr, stages=["match"])
    m = out["match_iom"]
    order = np.argsort(tr["seq"], kind="stable")
    want = np.full(m.size, -1)
    for n in range(tr["n_names"]):
        ks = order[tr["name_id"][order] == n]
        rows = np.flatnonzero(tr["pf_name"] == n)
        k = min(ks.size, rows.size)
        want[ks[:k]] = rows[:k]
    np.testing.assert_array_equal(m, want)
    tl = np.bincount(tr["name_id"], minlength=tr["n_names"])
    pf = np.bincount(tr["pf_name"], minlength=tr["n_names"])
    d = out["diag"]
    assert d["names_mismatched"] == int((tl != pf).sum()) > 0
    assert d["tl_unmatched"] == int(np.maximum(tl - pf, 0).sum())
    assert d["pf_unmatched"] == int(np.maximum(pf - tl, 0).sum())
    np.testing.assert_array_equal(out["name_counts"][:, 0], tl)
    np.testing.assert_array_equal(out["name_counts"][:, 1], pf)
    assert d["status"] == 0
    strict = O.attribute(tr, policy=O.STRICT, stages=["match"])
    assert strict["diag"]["status"] == -4
    np.testing.assert_array_equal(strict["match_iom"], m)


def test_iom_invariants():
    tr = tg.generate("lstm", T=40_000, ranges=400)
    m = O.attribute(tr, stages=["match"])["match_iom"]
    ok = m >= 0
    # the matched row always carries the launch's name
    np.testing.assert_array_equal(tr["pf_name"][m[ok]], tr["name_id"][ok])
    # per name, matches = min(tl, pf)
    tl = np.bincount(tr["name_id"], minlength=tr["n_names"])
    pf = np.bincount(tr["pf_name"], minlength=tr["n_names"])
    got = np.bincount(tr["name_id"][ok], minlength=tr["n_names"])
    np.testing.assert_array_equal(got, np.minimum(tl, pf))
    # injective, and increasing in launch order within a name
    assert np.unique(m[ok]).size == ok.sum()
    for n in range(tr["n_names"]):
        sel = np.flatnonzero(ok & (tr["name_id"] == n))
        o = np.argsort(tr["seq"][sel])
        assert np.all(np.diff(m[sel][o]) > 0)


def test_iom_timestamp_independence_figure():
    """Figure 'fig:clockdomain': five launches of one kernel name whose replay
    clock drifts. The nearest-timestamp join assigns K_D the row of K_C; IOM
    pairs by name and position and is untouched by any timestamp change."""
    fig = json.load(open(os.path.join(GOLD, "fig_clockdomain.json")))
    nsys = np.array(fig["nsys_t"])
    ncu = np.array(fig["ncu_t"])
    nearest = np.abs(nsys[:, None] - ncu[None, :]).argmin(axis=1)
    i_d = fig["kernels"].index(fig["timestamp_join_wrong"]["nsys"])
    assert fig["kernels"][nearest[i_d]] == fig["timestamp_join_wrong"]["ncu"]
    T = nsys.size
    tr = dict(seq=np.arange(T, dtype=np.uint32), start_ns=(nsys * 1000).astype(np.uint64),
              dur_ns=np.full(T, 10, np.uint32), stream_id=np.zeros(T, np.uint16),
              name_id=np.zeros(T, np.uint32), part_id=None, pf_name=np.zeros(T, np.uint32),
              counters=np.zeros((T, 20), np.float32), r_start=np.zeros(0, np.uint64),
              r_end=np.zeros(0, np.uint64), r_stream=np.zeros(0, np.uint16),
              r_op=np.zeros(0, np.uint32), part_rep=None, n_names=1, n_streams=1, n_ops=1)
    m = O.attribute(tr, stages=["match"])["match"]
    np.testing.assert_array_equal(m, np.arange(T))
    tr["start_ns"] = (ncu * 1000).astype(np.uint64)[::-1].copy()
    np.testing.assert_array_equal(O.attribute(tr, stages=["match"])["match"], np.arange(T))


def test_iom_timestamps_irrelevant_on_generated_trace():
    tr = tg.generate("lstm", T=20_000, ranges=200)
    m0 = O.attribute(tr, stages=["match"])["match"]
    rng = np.random.default_rng(7)
    tr2 = dict(tr, start_ns=rng.integers(0, 2**40, size=tr["seq"].size).astype(np.uint64))
    np.testing.assert_array_equal(O.attribute(tr2, stages=["match"])["match"], m0)


def test_iom_duplicate_seq_is_order_error():
    tr = cases.random_trace(3, T=30)
    tr["seq"] = tr["seq"].copy()
    tr["seq"][5] = tr["seq"][6]
    d = O.attribute(tr)["diag"]
    assert d["flags"] & O.F_ORDER and d["status"] == -8


# --------------------------------------------------------------------------- #
# layer dedup (Sec. 3.7)                                                       #
# --------------------------------------------------------------------------- #

@pytest.mark.parametrize("seed", range(30))
def test_dedup_matches_brute_force(seed):
    tr = cases.random_trace(100 + seed, T=60, dedup=True, drop=0.1 if seed % 2 else 0.0,
                            seq_gaps=seed % 3 == 1)
    out = O.attribute(tr, stages=["match", "dedup"])
    base = brute.iom(tr)
    want, errs = brute.dedup(tr, base)
    np.testing.assert_array_equal(out["match"], want)
    assert out["diag"]["dedup_errors"] == errs


def test_dedup_gpt2_profile_is_one_twelfth_and_planted():
    tr = tg.generate("gpt2")
    T, P = tr["seq"].size, tr["pf_name"].size
    assert P * 12 == T  # N/K = 12 replay reduction
    out = O.attribute(tr)
    m = out["match"]
    assert (m >= 0).all() and out["diag"]["dedup_errors"] == 0
    # every launch inherits the row replayed for the same position of layer 0
    # of its own iteration; the generator knows which launch produced each row
    seq = tr["seq"].astype(np.int64)
    per_layer, layers = 40, 12
    it, pos = seq // (per_layer * layers), seq % per_layer
    src_seq = it * per_layer * layers + pos
    kernel_of_seq = np.empty(T, dtype=np.int64)
    kernel_of_seq[seq] = np.arange(T)
    row_of_kernel = np.full(T, -1)
    row_of_kernel[tr["pf_src"]] = np.arange(P)
    np.testing.assert_array_equal(m, row_of_kernel[kernel_of_seq[src_seq]])
    np.testing.assert_array_equal(tr["pf_name"][m], tr["name_id"])


def test_dedup_k_equals_n_reduces_to_no_dedup():
    tr = cases.random_trace(11, T=80, dedup=True)
    tr2 = dict(tr, part_rep=np.arange(tr["n_parts"], dtype=np.int32))
    # with every partition its own class, every launch is replayed
    order = np.argsort(tr2["seq"])
    tr2["pf_name"] = tr2["name_id"][order]
    tr2["counters"] = np.zeros((tr2["pf_name"].size, 20), np.float32)
    a = O.attribute(tr2)["match"]
    tr3 = dict(tr2, part_id=None, part_rep=None, n_parts=0)
    b = O.attribute(tr3)["match"]
    np.testing.assert_array_equal(a, b)


def _dedup_case():
    # launch order: [rep p0: names 1 2 3][dup p1: names 1 2 3][dup p2: 1 2 3]
    T = 9
    tr = dict(seq=np.arange(T, dtype=np.uint32), start_ns=np.arange(T, dtype=np.uint64) * 10,
              dur_ns=np.ones(T, np.uint32), stream_id=np.zeros(T, np.uint16),
              name_id=np.array([1, 2, 3] * 3, np.uint32),
              part_id=np.repeat(np.arange(3), 3).astype(np.int32),
              pf_name=np.array([1, 2, 3], np.uint32), counters=np.zeros((3, 20), np.float32),
              r_start=np.zeros(0, np.uint64), r_end=np.zeros(0, np.uint64),
              r_stream=np.zeros(0, np.uint16), r_op=np.zeros(0, np.uint32),
              part_rep=np.zeros(3, np.int32), n_names=4, n_streams=1, n_ops=1, n_parts=3)
    return tr


def test_dedup_error_cases():
    tr = _dedup_case()
    out = O.attribute(tr)
    np.testing.assert_array_equal(out["match"], [0, 1, 2] * 3)
    assert out["diag"]["status"] == 0
    # a duplicate whose name differs from the representative at its position
    t2 = dict(tr, name_id=tr["name_id"].copy())
    t2["name_id"][4] = 0
    out = O.attribute(t2)
    assert out["match"][4] == -1 and out["diag"]["dedup_errors"] == 1
    assert out["diag"]["status"] == -6
    # a duplicate partition longer than its representative
    t3 = dict(tr, part_id=tr["part_id"].copy())
    t3["part_id"][2] = 1  # rep p0 now has 2 kernels; p1 has 4
    out = O.attribute(t3)
    assert out["diag"]["dedup_errors"] >= 1
    # a representative that is itself a duplicate (not a fixed point)
    t4 = dict(tr, part_rep=np.array([0, 0, 1], np.int32))
    out = O.attribute(t4)
    np.testing.assert_array_equal(out["match"][6:], [-1, -1, -1])
    assert out["diag"]["dedup_errors"] == 3
    # a partition whose launches are not one contiguous run
    t5 = dict(tr, part_id=np.array([0, 0, 0, 1, 2, 1, 2, 1, 2], np.int32))
    out = O.attribute(t5)
    assert out["diag"]["flags"] & O.F_PARTITION and out["diag"]["status"] == -7
    np.testing.assert_array_equal(out["match"][3:], [-1] * 6)


def test_counters_out_inherited_by_position():
    """Sec. 3.7: a duplicate layer's launches carry the counters of the
    representative's launch at the same position. Planted: row j of the
    profile holds 1000 * j + c, and the representative's launches are rows
    0, 1, 2 in launch order."""
    tr = _dedup_case()
    tr["counters"] = (1000 * np.arange(3)[:, None] + np.arange(20)[None, :]).astype(np.float32)
    rows = tr["counters"]
    out = O.attribute(tr, stages=["match", "dedup"])
    got = O.counters_out(tr, out["match"])
    np.testing.assert_array_equal(got, rows[[0, 1, 2] * 3])
    # counters absent from the capture are NaN for every launch
    got = O.counters_out(tr, out["match"], absent_mask=(1 << 3) | (1 << 19))
    assert np.isnan(got[:, [3, 19]]).all()
    keep = [c for c in range(20) if c not in (3, 19)]
    np.testing.assert_array_equal(got[:, keep], rows[[0, 1, 2] * 3][:, keep])
    # a duplicate whose name differs at its position inherits nothing
    t2 = dict(tr, name_id=tr["name_id"].copy())
    t2["name_id"][4] = 0
    got = O.counters_out(t2, O.attribute(t2, stages=["match", "dedup"])["match"])
    assert np.isnan(got[4]).all()
    np.testing.assert_array_equal(got[[3, 5]], rows[[0, 2]])
    # rows out of range and unmatched launches are NaN; strides are honoured
    m = np.array([2, -1, 3, 0], np.int32)
    t3 = dict(tr, counters=np.asfortranarray(rows))
    got = O.counters_out(t3, m)
    np.testing.assert_array_equal(got[[0, 3]], rows[[2, 0]])
    assert np.isnan(got[[1, 2]]).all()


def test_counters_out_gpt2_layers_equal_by_position():
    """The GPT-2-shaped trace (12 identical layers, one profiled): every
    launch of a duplicate layer carries the same counters as the launch at
    its position in its class representative, with positions taken from the
    partition tags in launch order."""
    tr = tg.generate("gpt2")
    out = O.attribute(tr, stages=["match", "dedup"])
    assert out["diag"]["dedup_errors"] == 0
    got = O.counters_out(tr, out["match"])
    order = np.argsort(tr["seq"], kind="stable")
    part = tr["part_id"][order]
    members = {q: order[part == q] for q in np.unique(part[part >= 0])}
    checked = 0
    for q, idx in members.items():
        r = int(tr["part_rep"][q])
        if r == q:
            continue
        src = members[r]
        assert src.size == idx.size
        np.testing.assert_array_equal(got[idx], got[src])
        checked += idx.size
    assert checked > 0.9 * tr["seq"].size * 11 / 12 * 0.9
    # the representative's launches carry rows of their own name
    reps = np.concatenate([members[q] for q in members if tr["part_rep"][q] == q])
    m = out["match"][reps]
    assert (m >= 0).all() and (tr["pf_name"][m] == tr["name_id"][reps]).all()
    np.testing.assert_array_equal(got[reps], tr["counters"][m])


def test_dedup_contiguity_is_in_launch_order():
    """A partition is a window of launches (Sec. 3.7): with gaps between the
    launch ordinals it is still contiguous when no other launch falls inside."""
    tr = _dedup_case()
    tr = dict(tr, seq=(np.arange(9) * 10 + 3).astype(np.uint32))
    out = O.attribute(tr)
    assert out["diag"]["status"] == 0
    np.testing.assert_array_equal(out["match"], [0, 1, 2] * 3)
    # an unpartitioned launch inside partition 1's window breaks it
    t2 = dict(tr, seq=np.array([0, 10, 20, 30, 40, 55, 60, 70, 80], np.uint32),
              part_id=np.array([0, 0, 0, 1, 1, 1, 2, 2, 2], np.int32))
    t2["seq"] = t2["seq"].copy()
    t2["part_id"] = np.concatenate([t2["part_id"], [-1]]).astype(np.int32)
    t2["seq"] = np.concatenate([t2["seq"], [45]]).astype(np.uint32)
    for key in ("start_ns", "dur_ns", "stream_id"):
        t2[key] = np.concatenate([t2[key], t2[key][:1]])
    t2["name_id"] = np.concatenate([t2["name_id"], [3]]).astype(np.uint32)
    t2["pf_name"] = np.array([1, 2, 3, 3], np.uint32)
    t2["counters"] = np.zeros((4, 20), np.float32)
    out = O.attribute(t2)
    assert out["diag"]["flags"] & O.F_PARTITION
    assert (out["match"][3:6] == -1).all()


def test_bad_ids_are_data_errors():
    tr = _dedup_case()
    t = dict(tr, name_id=tr["name_id"].copy())
    t["name_id"][0] = 99
    out = O.attribute(t)
    assert out["diag"]["bad_records"] == 1 and out["diag"]["status"] == -9
    assert out["match"][0] == -1


# --------------------------------------------------------------------------- #
# enclosure (Alg. 2)                                                           #
# --------------------------------------------------------------------------- #

@pytest.mark.parametrize("seed", range(60))
def test_enclose_matches_brute_force(seed):
    tr = cases.random_trace(200 + seed, T=70, R=25, S=1 + seed % 3, t_max=40,
                            nested=seed % 4 != 3)
    out = O.attribute(tr, stages=["match", "enclose"])
    np.testing.assert_array_equal(out["range_id"], brute.enclose(tr))
    np.testing.assert_array_equal(out["range_depth"], np.minimum(brute.depth(tr), 255))
    assert out["diag"]["nesting_errors"] == len(brute.crossing_streams(tr))


def test_enclose_ties_and_edges():
    # one stream; ranges: 0=[10,20] 1=[10,20] (identical: 1 is inner) 2=[20,30]
    # (touches 0/1 at 20) 3=[25,25] (point) 4=[40,50]; kernels at 5 (before all),
    # 10 (= s), 20 (touching point), 25 (point range), 30 (= e), 35 (gap), 60 (after)
    q = np.array([5, 10, 20, 25, 30, 35, 60], np.uint64)
    T = q.size
    tr = dict(seq=np.arange(T, dtype=np.uint32), start_ns=q, dur_ns=np.ones(T, np.uint32),
              stream_id=np.zeros(T, np.uint16), name_id=np.zeros(T, np.uint32), part_id=None,
              pf_name=np.zeros(0, np.uint32), counters=np.zeros((0, 20), np.float32),
              r_start=np.array([10, 10, 20, 25, 40], np.uint64),
              r_end=np.array([20, 20, 30, 25, 50], np.uint64),
              r_stream=np.zeros(5, np.uint16), r_op=np.arange(5, dtype=np.uint32),
              part_rep=None, n_names=1, n_streams=1, n_ops=5)
    out = O.attribute(tr)
    np.testing.assert_array_equal(out["range_id"], [-1, 1, 2, 3, 2, -1, -1])
    np.testing.assert_array_equal(out["range_id"], brute.enclose(tr))
    np.testing.assert_array_equal(out["range_depth"], [1, 2, 1, 2, 1])
    assert out["diag"]["nesting_errors"] == 0
    # the query point, when given, replaces the start time
    tr["query_ns"] = np.array([45] * T, np.uint64)
    np.testing.assert_array_equal(O.attribute(tr)["range_id"], [4] * T)


def test_enclose_crossing_ranges_flagged():
    T = 3
    tr = dict(seq=np.arange(T, dtype=np.uint32), start_ns=np.array([1, 4, 9], np.uint64),
              dur_ns=np.ones(T, np.uint32), stream_id=np.zeros(T, np.uint16),
              name_id=np.zeros(T, np.uint32), part_id=None, pf_name=np.zeros(0, np.uint32),
              counters=np.zeros((0, 20), np.float32),
              r_start=np.array([0, 3], np.uint64), r_end=np.array([5, 8], np.uint64),
              r_stream=np.zeros(2, np.uint16), r_op=np.zeros(2, np.uint32), part_rep=None,
              n_names=1, n_streams=1, n_ops=1)
    out = O.attribute(tr)
    assert out["diag"]["nesting_errors"] == 1 and out["diag"]["status"] == -5
    np.testing.assert_array_equal(out["range_id"], brute.enclose(tr))


def _with_kinds(tr, seed, p_bad=0.0):
    return cases.with_kinds(tr, seed, p_bad=p_bad)


@pytest.mark.parametrize("seed", range(12))
def test_enclose_walk_matches_brute_force(seed):
    """Alg. 2's walk with range kinds (op / structural boundary / skipped
    namespace) against its definition written out per kernel."""
    tr = cases.random_trace(700 + seed, T=70, R=30, S=1 + seed % 3, t_max=40, max_depth=5)
    tr = _with_kinds(tr, seed, p_bad=0.05 if seed % 4 == 3 else 0.0)
    out = O.enclose_walk(tr)
    rid, fused, rany, par = brute.enclose_walk(tr)
    np.testing.assert_array_equal(out["range_id"], rid)
    np.testing.assert_array_equal(out["fused"], fused)
    np.testing.assert_array_equal(out["range_any"], rany)
    np.testing.assert_array_equal(out["range_parent"], par)
    assert out["diag"]["nesting_errors"] == 0


def test_enclose_walk_all_ops_is_innermost():
    """Without kinds every range is an op: the walk returns the innermost
    enclosing range, and a kernel is fused exactly when that range has a
    parent (a second op encloses it)."""
    tr = tg.generate("tiny")
    out = O.enclose_walk(tr)
    np.testing.assert_array_equal(out["range_id"], tr["planted_range"])
    np.testing.assert_array_equal(out["range_any"], out["range_id"])
    has = out["range_any"] >= 0
    want = np.zeros_like(out["fused"])
    want[has] = out["range_parent"][out["range_any"][has]] >= 0
    np.testing.assert_array_equal(out["fused"], want)
    # parents are one level up
    d = out["range_depth"].astype(np.int64)
    ok = out["range_parent"] >= 0
    np.testing.assert_array_equal(d[ok], d[out["range_parent"][ok]] + 1)
    assert (d[~ok] <= 1).all()


def test_enclose_walk_hand_shaped():
    """A profiler step (structural boundary) encloses aten::linear (op), which
    encloses prims::view (skipped) enclosing aten::addmm (op); a second step
    holds aten::relu directly. Kernels: inside addmm (op addmm, fused: linear
    is also collected), inside view only (op linear, not fused), inside linear
    only, inside the step only (no op: the walk stops at the boundary), inside
    relu, and outside everything."""
    #          0=step1   1=linear  2=view    3=addmm   4=step2   5=relu
    rs = np.array([0, 10, 20, 30, 100, 110], np.uint64)
    re = np.array([90, 80, 70, 40, 190, 120], np.uint64)
    kind = np.array([1, 0, 2, 0, 1, 0], np.uint8)
    q = np.array([35, 50, 75, 5, 115, 95], np.uint64)
    T = q.size
    tr = dict(seq=np.arange(T, dtype=np.uint32), start_ns=q, dur_ns=np.ones(T, np.uint32),
              stream_id=np.zeros(T, np.uint16), name_id=np.zeros(T, np.uint32), part_id=None,
              pf_name=np.zeros(0, np.uint32), counters=np.zeros((0, 20), np.float32),
              r_start=rs, r_end=re, r_stream=np.zeros(6, np.uint16),
              r_op=np.arange(6, dtype=np.uint32), r_kind=kind, part_rep=None,
              n_names=1, n_streams=1, n_ops=6)
    out = O.enclose_walk(tr)
    np.testing.assert_array_equal(out["range_id"], [3, 1, 1, -1, 5, -1])
    np.testing.assert_array_equal(out["fused"], [1, 0, 0, 0, 0, 0])
    np.testing.assert_array_equal(out["range_any"], [3, 2, 1, 0, 5, -1])
    np.testing.assert_array_equal(out["range_parent"], [-1, 0, 1, 2, -1, 4])
    # the aggregation follows the walk: the step's own kernel is unattributed
    agg = O.attribute(tr, stages=["match", "enclose", "aggregate"])
    np.testing.assert_array_equal(agg["range_id"], out["range_id"])
    assert agg["table"]["kernel_count"][6] == 2


def _class_trace(seed, T=90, n_parts=9, noncontig=False, bad=False):
    return cases.class_trace(seed, T=T, n_parts=n_parts, noncontig=noncontig, bad=bad)


@pytest.mark.parametrize("seed", range(10))
def test_dedup_classes_match_brute_force(seed):
    """Class discovery against its definition: pairwise comparison of the
    partitions' (name, stream) sequences in launch order."""
    tr = _class_trace(seed, noncontig=seed % 3 == 1, bad=seed % 4 == 3)
    out = O.dedup_classes(tr)
    rep, has_noncontig = brute.dedup_classes(tr)
    np.testing.assert_array_equal(out["part_rep"], rep)
    assert bool(out["diag"]["flags"] & 16) == has_noncontig


def test_dedup_classes_empty_partitions_form_one_class():
    """Partitions without launches all have the empty sequence."""
    tr = _class_trace(4)
    part = tr["part_id"].copy()
    part[(part == 3) | (part == 5)] = -1
    tr["part_id"] = part
    out = O.dedup_classes(tr)
    rep, _ = brute.dedup_classes(tr)
    np.testing.assert_array_equal(out["part_rep"], rep)
    assert out["part_rep"][5] == 3 and out["part_rep"][3] == 3
    empty = cases.random_trace(0, T=0, S=1, n_names=2)
    empty.update(part_id=np.zeros(0, np.int32), n_parts=3, part_rep=None)
    np.testing.assert_array_equal(O.dedup_classes(empty)["part_rep"], [0, 0, 0])


def test_dedup_classes_duplicate_seq_ties_by_index():
    """Equal seq values rank by input index (as in the matching) and raise
    ORDER: launches 0 and 1 share seq 5, so partition 0 = (a, b) in index
    order and partition 1 = (a, b) too; swapping the indices of partition 1's
    launches would reverse it."""
    tr = cases.random_trace(0, T=4, S=1, n_names=2)
    tr.update(seq=np.array([5, 5, 7, 8], np.uint32), name_id=np.array([0, 1, 0, 1], np.uint32),
              stream_id=np.zeros(4, np.uint16), part_id=np.array([0, 0, 1, 1], np.int32),
              n_parts=2, part_rep=None)
    out = O.dedup_classes(tr)
    np.testing.assert_array_equal(out["part_rep"], [0, 0])
    assert out["diag"]["flags"] & 2 and out["diag"]["status"] == -8
    tr["name_id"] = np.array([1, 0, 0, 1], np.uint32)
    np.testing.assert_array_equal(O.dedup_classes(tr)["part_rep"], [0, 1])
    np.testing.assert_array_equal(brute.dedup_classes(tr)[0], [0, 1])
    tr["seq"] = np.array([5, 6, 7, 8], np.uint32)
    assert not O.dedup_classes(tr)["diag"]["flags"] & 2


@pytest.mark.parametrize("cfg", ["gpt2", "large"])
def test_dedup_classes_recover_the_generated_templates(cfg):
    """The generator copies class templates into every layer instance: GPT-2
    has one class (every layer is the same 40-kernel template), the large
    trace three (layer l of every iteration belongs to class l mod 3), so
    discovery finds the first instances as representatives. The planted
    per-iteration representatives are members of those classes."""
    tr = tg.generate(cfg)
    out = O.dedup_classes(tr)
    q = np.arange(tr["n_parts"])
    want = np.zeros_like(q) if cfg == "gpt2" else (q % 48) % 3
    np.testing.assert_array_equal(out["part_rep"], want)
    np.testing.assert_array_equal(out["part_rep"][tr["part_rep"]], out["part_rep"])
    assert out["diag"]["status"] == 0


@pytest.mark.parametrize("cfg", ["tiny", "gpt2", "sdpa", "lstm"])
def test_enclose_planted_labels(cfg):
    tr = tg.generate(cfg)
    out = O.attribute(tr, stages=["match", "enclose"])
    np.testing.assert_array_equal(out["range_id"], tr["planted_range"])
    assert out["diag"]["nesting_errors"] == 0


def test_enclose_invariants_and_depth():
    tr = tg.generate("tiny")
    out = O.attribute(tr, stages=["match", "enclose"])
    rid, dep = out["range_id"], out["range_depth"].astype(np.int64)
    q = tr["start_ns"]
    ok = rid >= 0
    # the chosen range holds the query point and lies on the kernel's stream
    assert np.all(tr["r_start"][rid[ok]] <= q[ok]) and np.all(q[ok] <= tr["r_end"][rid[ok]])
    assert np.all(tr["r_stream"][rid[ok]] == tr["stream_id"][ok])
    # its depth is the maximum among all ranges containing the query point
    for i in np.flatnonzero(ok)[::7]:
        cont = (tr["r_stream"] == tr["stream_id"][i]) & (tr["r_start"] <= q[i]) & (q[i] <= tr["r_end"])
        assert dep[rid[i]] == dep[cont].max()
    # kernels before the first range of their stream fall through
    first = tr["r_start"].min()
    assert np.all(rid[q < first] == -1)
    # depth = number of containing ranges (properly nested, no touching here)
    small = cases.random_trace(5, T=10, R=40, S=2, t_max=200)
    small_out = O.attribute(small, stages=["match", "enclose"])
    np.testing.assert_array_equal(small_out["range_depth"], brute.depth(small))
    assert out["range_depth"].min() >= 1 and out["range_depth"].max() <= 4


def test_depth_equals_container_count_without_touching():
    for seed in range(10):
        tr = cases.random_trace(300 + seed, T=5, R=30, S=2, t_max=1000)
        # drop ranges sharing an endpoint so containment is a tree
        ends = np.concatenate([tr["r_start"], tr["r_end"]])
        vals, cnt = np.unique(ends, return_counts=True)
        dup = set(vals[cnt > 1].tolist())
        keep = np.array([(a not in dup and b not in dup) for a, b in zip(tr["r_start"], tr["r_end"])],
                        dtype=bool)
        for k in ("r_start", "r_end", "r_stream", "r_op"):
            tr[k] = tr[k][keep]
        out = O.attribute(tr, stages=["match", "enclose"])
        np.testing.assert_array_equal(out["range_depth"], brute.containers(tr))


# --------------------------------------------------------------------------- #
# aggregation (Eq. 1)                                                          #
# --------------------------------------------------------------------------- #

def _table_dicts(table):
    return [dict(kernel_count=int(r["kernel_count"]), total_ns=int(r["total_ns"]),
                 matched_count=int(r["matched_count"]), matched_ns=int(r["matched_ns"]),
                 value=[float(v) for v in r["value"]]) for r in table]


def _assert_rows(got, want, rtol):
    for a, b in zip(got, want):
        for f in ("kernel_count", "total_ns", "matched_count", "matched_ns"):
            assert a[f] == b[f]
        for x, y in zip(a["value"], b["value"]):
            if math.isnan(y):
                assert math.isnan(x)
            else:
                assert abs(x - y) <= rtol * max(abs(x), abs(y)), (x, y)


def golden_kinds():
    """The Agg. column of the counter reference table (tests/golden)."""
    code = {"SUM": O.SUM, "DW-mean": O.DWMEAN, "MAX": O.MAX}
    rows = [ln.split() for ln in open(os.path.join(GOLD, "counter_agg.txt"))
            if ln.strip() and not ln.startswith("#")]
    assert [int(r[0]) for r in rows] == list(range(1, 21))
    return np.array([code[r[2]] for r in rows], np.uint8)


def test_default_kinds_are_the_counter_table():
    """The default aggregation kinds equal the transcribed Agg. column: the
    Python constant, the brute-force copy, and the C oracle's own table
    (the default gives the same table as passing the column explicitly, and
    a different one as soon as any single counter's kind changes)."""
    want = golden_kinds()
    np.testing.assert_array_equal(O.DEFAULT_KIND, want)
    np.testing.assert_array_equal(np.array(brute.DEFAULT_KIND, np.uint8), want)
    tr = cases.random_trace(31, T=400, R=60, n_ops=9, t_max=500)
    base = O.attribute(tr)["table"]
    same = O.attribute(tr, agg_kind=want)["table"]
    assert base.tobytes() == same.tobytes()
    for c in range(20):
        k = want.copy()
        k[c] = (k[c] + 1) % 3
        assert O.attribute(tr, agg_kind=k)["table"].tobytes() != base.tobytes(), c


def test_single_kernel_identity_from_profile_excerpt():
    """The appendix excerpt: one kernel attributed to aten::mm_26 gives
    kernel_count 1, total_duration_ns = its duration, and every aggregated
    counter equal to that kernel's own value; the counter absent on the
    capture's architecture is null."""
    g = json.load(open(os.path.join(GOLD, "profile_excerpt.json")))
    cnt = np.zeros((1, 20), np.float32)
    for v in g["counters"].values():
        cnt[0, v["index"]] = v["value"]
    absent = 0
    for v in g["absent"].values():
        absent |= 1 << v["index"]
    tr = dict(seq=np.zeros(1, np.uint32), start_ns=np.array([100], np.uint64),
              dur_ns=np.array([g["duration_ns"]], np.uint32), stream_id=np.zeros(1, np.uint16),
              name_id=np.zeros(1, np.uint32), part_id=None, pf_name=np.zeros(1, np.uint32),
              counters=cnt, r_start=np.array([50], np.uint64), r_end=np.array([200], np.uint64),
              r_stream=np.zeros(1, np.uint16), r_op=np.zeros(1, np.uint32), part_rep=None,
              n_names=1, n_streams=1, n_ops=1)
    out = O.attribute(tr, absent_mask=absent)
    row = out["table"][0]
    assert int(row["kernel_count"]) == g["kernel_count"]
    assert int(row["total_ns"]) == g["total_duration_ns"]
    for v in g["counters"].values():
        assert row["value"][v["index"]] == float(np.float32(v["value"]))
    for v in g["absent"].values():
        assert math.isnan(row["value"][v["index"]])
    assert out["summary"]["attributed_fraction"] == 1.0


@pytest.mark.parametrize("seed", range(20))
def test_aggregate_matches_fsum(seed):
    tr = cases.random_trace(400 + seed, T=120, R=30, drop=0.2, dedup=seed % 2 == 0)
    kind = None if seed % 3 else np.array([1] * 20, np.uint8)
    absent = 0 if seed % 4 else (1 << 5) | (1 << 17)
    out = O.attribute(tr, agg_kind=kind, absent_mask=absent)
    want = brute.aggregate(tr, out["match"], out["range_id"], kind, absent)
    _assert_rows(_table_dicts(out["table"]), want, 1e-13)


@pytest.mark.parametrize("cfg", ["tiny", "gpt2"])
def test_aggregate_matches_fsum_on_configs(cfg):
    tr = tg.generate(cfg)
    out = O.attribute(tr)
    want = brute.aggregate(tr, out["match"], out["range_id"])
    _assert_rows(_table_dicts(out["table"]), want, 1e-12)


def test_aggregate_closed_forms():
    tr = tg.generate("tiny")
    # equal durations: the duration-weighted mean is the arithmetic mean
    t = dict(tr, dur_ns=np.full(tr["seq"].size, 777, np.uint32))
    t["counters"] = tr["counters"].copy()
    t["counters"][:, 7] = np.float32(0.625)  # a constant counter: DW = constant
    out = O.attribute(t)
    for g, row in enumerate(out["table"]):
        if row["matched_count"] == 0:
            assert math.isnan(row["value"][3])
            continue
        sel = np.flatnonzero((np.where(out["range_id"] >= 0, t["r_op"][out["range_id"]],
                                       t["n_ops"]) == g) & (out["match"] >= 0))
        ms = t["counters"][out["match"][sel], 3].astype(np.float64)
        assert abs(row["value"][3] - ms.mean()) <= 1e-12 * abs(ms.mean())
        assert row["value"][7] == 0.625
        # MAX is the plain maximum, exactly
        assert row["value"][17] == t["counters"][out["match"][sel], 17].max()
    # totals are exact and complete
    tab, sm = out["table"], out["summary"]
    assert int(tab["kernel_count"].sum()) == t["seq"].size
    assert int(tab["total_ns"].sum(dtype=np.uint64)) == int(t["dur_ns"].sum(dtype=np.uint64))
    assert sm["attributed_ns"] + sm["unattributed_ns"] == sm["total_ns"]
    assert sm["unattributed_ns"] == int(tab["total_ns"][-1])


def test_coverage_of_shaped_configs():
    assert O.attribute(tg.generate("sdpa"))["summary"]["attributed_fraction"] == 1.0
    tr = tg.generate("lstm", T=200_000, ranges=2_000)
    f = O.attribute(tr)["summary"]["attributed_fraction"]
    assert 0.10 < f < 0.20


def test_emission_orders_agree():
    base = None
    for em in ("stream_major", "seq", "shuffled"):
        tr = tg.generate("gpt2", emission=em)
        out = O.attribute(tr)
        # map outputs back to launch order and ranges to a canonical key
        o = np.argsort(tr["seq"])
        key = np.stack([tr["r_stream"].astype(np.uint64), tr["r_start"]], 1)
        rid = out["range_id"][o]
        rk = np.where(rid[:, None] >= 0, key[np.maximum(rid, 0)], -1)
        res = (out["match"][o], rk, out["table"])
        if base is None:
            base = res
            continue
        np.testing.assert_array_equal(res[0], base[0])
        np.testing.assert_array_equal(res[1], base[1])
        _assert_rows(_table_dicts(res[2]), _table_dicts(base[2]), 1e-14)


def _tier_trace(seed, T=120, dedup=False, shuffle=False, p_bad=0.0):
    tr = cases.random_trace(500 + seed, T=T, R=40, S=2, t_max=80, max_depth=4, dedup=dedup)
    tr = cases.with_kinds(tr, seed)
    return tg.with_attribution_maps(tr, seed=seed, p_corr=0.6, p_mismatch=0.3, p_none=0.1,
                                    p_fmap=0.5, p_bad=p_bad, shuffle=shuffle)


@pytest.mark.parametrize("seed", range(8))
@pytest.mark.parametrize("policy", [0, 1, 2])
def test_tiers_match_brute_force(seed, policy):
    """The decision tree written out per kernel (brute.tiers) against the
    oracle: random traces with range kinds, partitions (which the
    correlation index ignores), maps with missing entries, count mismatches,
    interleaved names and bad operator ids."""
    tr = _tier_trace(seed, dedup=seed % 2 == 0, shuffle=seed % 3 == 1,
                     p_bad=0.05 if seed % 4 == 3 else 0.0)
    out = O.tiers(tr, corr_policy=policy)
    tier, op, fused, cnt, ns = brute.tiers(tr, 1 if policy == 1 else 0)
    np.testing.assert_array_equal(out["tier"], tier)
    np.testing.assert_array_equal(out["op"], op)
    np.testing.assert_array_equal(out["fused"], fused)
    assert list(out["coverage"]["count"]) == cnt and list(out["coverage"]["ns"]) == ns
    assert out["coverage"]["ns"].sum() == tr["dur_ns"].astype(np.int64).sum()
    assert math.isclose(out["coverage"]["frac"].sum(), 1.0, rel_tol=1e-12)
    co = tr["corr_op"].astype(np.int64)
    bad = int(((co < -1) | (co >= tr["n_ops"])).sum())
    assert out["diag"]["bad_records"] == bad and bool(out["diag"]["flags"] & 1) == (bad > 0)
    if policy == 2 and out["diag"]["flags"] & 64 and not bad:
        assert out["diag"]["status"] == -4


def test_tiers_decision_tree_example():
    """One kernel per branch of the decision-tree figure, on one stream with
    one op range around launches 0, 1 and 5:
      0  name 0, invocation 0: map entry op 3 -> HIGH 3 (pre-empts the range);
         the fusion map lists two ops for name 0 -> fused
      1  name 1 (no map entries) inside the range -> NVTX, the range's op 1
      2  name 2 outside the range, fusion map [4] -> FUSION 4, not fused
      3  name 3 outside, nothing -> UNATTRIBUTED
      4  name 2 again -> FUSION 4
      5  name 0, invocation 1: the entry records no operator -> the range, NVTX 1
    """
    tr = cases.random_trace(0, T=6, S=1, n_names=4, R=1)
    tr.update(seq=np.arange(6, dtype=np.uint32),
              start_ns=np.array([10, 20, 50, 60, 70, 30], np.uint64),
              dur_ns=np.array([1, 2, 4, 8, 16, 32], np.uint32),
              stream_id=np.zeros(6, np.uint16), name_id=np.array([0, 1, 2, 3, 2, 0], np.uint32),
              part_id=None, part_rep=None, query_ns=None,
              r_start=np.array([5], np.uint64), r_end=np.array([40], np.uint64),
              r_stream=np.zeros(1, np.uint16), r_op=np.array([1], np.uint32), r_kind=None,
              n_ops=8, n_names=4, n_streams=1,
              corr_name=np.array([0, 0], np.uint32), corr_op=np.array([3, -1], np.int32),
              fmap_off=np.array([0, 2, 2, 3, 3], np.uint32), fmap_op=np.array([5, 6, 4], np.int32))
    out = O.tiers(tr)
    np.testing.assert_array_equal(out["tier"], [1, 2, 3, 0, 3, 2])
    np.testing.assert_array_equal(out["op"], [3, 1, 4, -1, 4, 1])
    np.testing.assert_array_equal(out["fused"], [1, 0, 0, 0, 0, 1])
    np.testing.assert_array_equal(out["coverage"]["count"], [1, 1, 2, 2])
    np.testing.assert_array_equal(out["coverage"]["ns"], [8, 1, 34, 20])
    np.testing.assert_allclose(out["coverage"]["frac"], np.array([8, 1, 34, 20]) / 63)


def test_tiers_full_correlation_map_is_all_high():
    """A correlation map recorded from the same run for every name (no gaps,
    no mismatches): every launch with a valid name is HIGH, with the op of
    its planted innermost range where it has one."""
    tr = tg.with_attribution_maps(tg.generate("tiny"), seed=3, p_corr=1.0, p_mismatch=0.0,
                                  p_none=0.0, p_fmap=0.0)
    out = O.tiers(tr)
    assert np.all(out["tier"] == 1)
    enc = tr["planted_range"] >= 0
    np.testing.assert_array_equal(out["op"][enc], tr["r_op"][tr["planted_range"][enc]])
    assert out["coverage"]["frac"][1] == 1.0 and out["diag"]["status"] == 0


def test_tiers_without_maps_reduce_to_the_walk():
    tr = cases.with_kinds(tg.generate("tiny"), 2)
    out = O.tiers(tr)
    walk = O.enclose_walk(tr)
    rid = walk["range_id"]
    np.testing.assert_array_equal(out["tier"], np.where(rid >= 0, 2, 0))
    r_op = tr["r_op"].astype(np.int64)
    np.testing.assert_array_equal(out["op"], np.where(rid >= 0, r_op[np.maximum(rid, 0)], -1))
    np.testing.assert_array_equal(out["fused"], walk["fused"])


def test_tiers_count_policies():
    """Name 0 has 5 launches and 4 entries: PREFIX gives HIGH to its first
    four invocations, SKIP_NAME to none of them, STRICT like PREFIX with
    status COUNT_MISMATCH."""
    tr = cases.random_trace(1, T=10, S=1, n_names=2, R=0)
    tr.update(seq=np.arange(10, dtype=np.uint32), name_id=np.array([0, 1] * 5, np.uint32),
              part_id=None, part_rep=None, n_ops=9,
              corr_name=np.array([0, 0, 1, 0, 1, 1, 0, 1, 1], np.uint32),
              corr_op=np.array([0, 1, 5, 2, 6, 7, 3, 8, 8], np.int32))
    pre = O.tiers(tr, corr_policy=0)
    np.testing.assert_array_equal(pre["tier"], [1, 1, 1, 1, 1, 1, 1, 1, 0, 1])
    np.testing.assert_array_equal(pre["op"], [0, 5, 1, 6, 2, 7, 3, 8, -1, 8])
    skip = O.tiers(tr, corr_policy=1)
    np.testing.assert_array_equal(skip["tier"], [0, 1] * 5)
    strict = O.tiers(tr, corr_policy=2)
    np.testing.assert_array_equal(strict["tier"], pre["tier"])
    assert pre["diag"]["status"] == 0 and strict["diag"]["status"] == -4
    assert pre["diag"]["names_mismatched"] == 1


def test_aggregate_ops_equals_range_aggregation():
    """Given each kernel's op as the op of its range, the aggregation by op
    is the aggregation by range (Eq. 1 pinned elsewhere)."""
    tr = tg.generate("tiny")
    full = O.attribute(tr)
    rid = full["range_id"]
    op = np.where(rid >= 0, tr["r_op"].astype(np.int64)[np.maximum(rid, 0)], -1).astype(np.int32)
    out = O.aggregate_ops(tr, full["match"], op)
    for f in ("kernel_count", "total_ns", "matched_count", "matched_ns"):
        np.testing.assert_array_equal(out["table"][f], full["table"][f])
    np.testing.assert_array_equal(out["table"]["value"], full["table"]["value"])
    bad = op.copy()
    bad[:3] = [tr["n_ops"], -2, 0]
    out = O.aggregate_ops(tr, full["match"], bad)
    assert out["diag"]["bad_records"] == 2 and out["diag"]["status"] == -9


def _dispatch_case(seed):
    tr = _tier_trace(seed, T=150, dedup=seed % 2 == 0)
    match = O.attribute(tr, stages=["match", "dedup"])["match"]
    t = O.tiers(tr)
    return tr, match, t


@pytest.mark.parametrize("seed", range(6))
def test_dispatch_table_matches_brute_force(seed):
    """Per-dispatch rows (a range when the kernel's tier operator is the
    range's, else per operator, else unattributed) against the fsum
    reduction over the same groups written out."""
    tr, match, t = _dispatch_case(seed)
    op = t["op"] if seed % 3 else None
    out = O.aggregate_dispatch(tr, match, t["range_id"], op)
    R = tr["r_start"].size
    keys = brute.dispatch_keys(tr, t["range_id"], op)
    want = brute.aggregate_groups(tr, match, keys, R + tr["n_ops"] + 1)
    for a, b in zip(out["table"], want):
        for f in ("kernel_count", "total_ns", "matched_count", "matched_ns"):
            assert int(a[f]) == b[f]
        for x, y in zip(a["value"], b["value"]):
            assert (math.isnan(x) and math.isnan(y)) or math.isclose(x, y, rel_tol=1e-12)


@pytest.mark.parametrize("seed", range(4))
def test_dispatch_rows_add_up_to_operator_rows(seed):
    """Every kernel of operator o lies in a dispatch of o or in o's own row
    R + o, so the per-dispatch rows of o add up to o's row of the operator
    table: counts and ns exactly, SUM by addition, MAX by max, the
    duration-weighted mean as the matched-ns weighted mean of the rows."""
    tr, match, t = _dispatch_case(10 + seed)
    disp = O.aggregate_dispatch(tr, match, t["range_id"], t["op"])["table"]
    ops = O.aggregate_ops(tr, match, t["op"])["table"]
    R, NOPS = tr["r_start"].size, tr["n_ops"]
    owner = np.concatenate([tr["r_op"].astype(np.int64), np.arange(NOPS), [NOPS]])
    kinds = O.DEFAULT_KIND
    for o in range(NOPS + 1):
        rows = disp[owner == o]
        for f in ("kernel_count", "total_ns", "matched_count", "matched_ns"):
            assert rows[f].sum() == ops[o][f]
        mk = rows[rows["matched_count"] > 0]
        for c in range(O.NC):
            want = ops[o]["value"][c]
            if not len(mk):
                assert math.isnan(want)
                continue
            v = mk["value"][:, c]
            if kinds[c] == O.SUM:
                got = math.fsum(v)
            elif kinds[c] == O.MAX:
                got = v.max()
            else:
                w = mk["matched_ns"].astype(np.float64)
                got = math.fsum(v * w) / w.sum()
            assert math.isclose(got, want, rel_tol=1e-9), (o, c, got, want)
    # without tier operators every kernel sits in its range's row
    plain = O.aggregate_dispatch(tr, match, t["range_id"])["table"]
    cnt = np.bincount(t["range_id"][t["range_id"] >= 0], minlength=R)
    np.testing.assert_array_equal(plain["kernel_count"][:R], cnt)
    assert plain["kernel_count"][R:R + NOPS].sum() == 0


@pytest.mark.parametrize("seed", range(8))
def test_enclose_all_matches_brute_force(seed):
    """Every enclosing range of every kernel, innermost first, against the
    containment test written out per kernel; coarse timestamps put many
    launches on range edges (closed intervals: a range ending at the point
    contains it). The walk's outputs are read off the same lists: range_any
    is the first entry, range_id the first op before a boundary, fused more
    than one op before it."""
    tr = cases.random_trace(960 + seed, T=120, R=60, S=1 + seed % 3, t_max=40 + 20 * (seed % 3),
                            max_depth=5)
    tr = cases.with_kinds(tr, seed, p_bad=0.05 if seed % 4 == 3 else 0.0)
    out = O.enclose_all(tr)
    want = brute.enclosing_lists(tr)
    off, ids = out["off"], out["ids"]
    assert off[0] == 0 and off[-1] == sum(len(w) for w in want)
    for i, w in enumerate(want):
        assert list(ids[off[i]:off[i + 1]]) == w, i
    walk = O.enclose_walk(tr)
    kind = tr["r_kind"]
    for i, w in enumerate(want):
        assert walk["range_any"][i] == (w[0] if w else -1)
        ops = []
        for r in w:
            if kind[r] == 1:
                break
            if kind[r] == 0:
                ops.append(r)
        assert walk["range_id"][i] == (ops[0] if ops else -1)
        assert walk["fused"][i] == (1 if len(ops) > 1 else 0)


@pytest.mark.parametrize("seed", range(6))
def test_enclose_all_reports_crossing_ranges(seed):
    """Crossing ranges (Alg. 2 assumes proper nesting): the list call counts
    the streams that have them, as the walk does, and the status says so."""
    tr = cases.random_trace(990 + seed, T=60, R=30, S=1 + seed % 3, t_max=40, nested=False)
    out = O.enclose_all(tr)
    n = len(brute.crossing_streams(tr))
    assert out["diag"]["nesting_errors"] == n
    assert out["diag"]["nesting_errors"] == O.enclose_walk(tr)["diag"]["nesting_errors"]
    assert (out["diag"]["status"] == -5) == (n > 0)


def test_enclose_all_capacity():
    """With a smaller capacity the offsets are still complete and exactly the
    lists that end within it are written."""
    tr = cases.random_trace(7, T=80, R=40, S=2, t_max=60, max_depth=4)
    full = O.enclose_all(tr)
    off = full["off"]
    cap = int(off[-1]) // 2
    import ctypes as C
    x = O._Inputs(tr)
    o2 = np.empty_like(off)
    ids = np.full(max(cap, 1), -7, np.int32)
    dg = O.Diag()
    assert O.lib().oref_enclose_all(C.byref(x.k), C.byref(x.r), C.byref(x.d), O._ptr(o2),
                                    O._ptr(ids), cap, C.byref(dg)) == 0
    np.testing.assert_array_equal(o2, off)
    last = np.searchsorted(off, cap, side="right") - 1  # lists 0..last-1 end within cap
    np.testing.assert_array_equal(ids[:off[last]], full["ids"][:off[last]])
    assert np.all(ids[off[last]:cap] == -7)
