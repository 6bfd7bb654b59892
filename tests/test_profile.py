"""profile.json export (App. A.4 schema) from the attribution's outputs, on
the host: the appendix excerpt reproduced field by field, and the document's
invariants (every kernel listed once, per-dispatch aggregates equal to the
table rows, call indices per operator, methods per tier)."""
import json
import os

import numpy as np

import brute
import cases
from oracle import oracle as O
from paper_2609_11938_amd import profile, tracegen as tg

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _outputs(tr, absent_mask=0):
    match = O.attribute(tr, stages=["match", "dedup"])["match"]
    t = O.tiers(tr)
    walk = O.enclose_walk(tr)
    disp = O.aggregate_dispatch(tr, match, t["range_id"], t["op"], absent_mask=absent_mask)
    row = np.array(brute.dispatch_keys(tr, t["range_id"], t["op"]))
    return match, t, walk, disp, row


def test_profile_reproduces_the_appendix_excerpt():
    """One kernel (seq 880, stream 7) inside the 27th aten::mm range: the
    operator entry carries the excerpt's identity fields, the kernel record
    its method and confidence, and the aggregated block its counter values
    with the architecture's absent counter as null."""
    g = json.load(open(os.path.join(GOLD, "profile_excerpt.json")))
    lst = g["listing"]
    cnt = np.zeros((1, 20), np.float32)
    for v in g["counters"].values():
        cnt[0, v["index"]] = v["value"]
    absent = 0
    for v in g["absent"].values():
        absent |= 1 << v["index"]
    R = lst["call_index"] + 1
    starts = np.arange(R, dtype=np.uint64) * 1000
    tr = dict(seq=np.array([880], np.uint32), start_ns=np.array([starts[-1] + 10], np.uint64),
              dur_ns=np.array([g["duration_ns"]], np.uint32),
              stream_id=np.array([lst["stream_id"]], np.uint16), name_id=np.zeros(1, np.uint32),
              part_id=None, pf_name=np.zeros(1, np.uint32), counters=cnt, r_start=starts,
              r_end=starts + 500, r_stream=np.full(R, lst["stream_id"], np.uint16),
              r_op=np.zeros(R, np.uint32), part_rep=None, n_names=1, n_streams=8, n_ops=1)
    match, t, walk, disp, row = _outputs(tr, absent)
    doc = profile.build(tr, match, t["tier"], t["op"], t["fused"], row, disp["table"],
                        op_names=[lst["operator_name"]], kernel_names=[lst["kernel_name"]],
                        absent_mask=absent)
    assert doc["schema_version"] == "1.0" and doc["unattributed_kernels"] == []
    (entry,) = doc["operators"]
    for f in ("operator_id", "operator_name", "call_index", "is_fused", "fused_with"):
        assert entry[f] == lst[f], f
    (k,) = entry["kernels"]
    for f in ("kernel_id", "kernel_name", "attribution_method", "confidence", "stream_id"):
        assert k[f] == lst[f], f
    assert k["duration_ns"] == g["duration_ns"]
    agg = entry["aggregated"]
    assert agg["total_duration_ns"] == g["total_duration_ns"]
    assert agg["kernel_count"] == g["kernel_count"]
    for f, v in g["counters"].items():
        assert agg[f] == float(np.float32(v["value"])), f
        assert k["metrics"][f] == float(np.float32(v["value"])), f
    for f in g["absent"]:
        assert agg[f] is None and k["metrics"][f] is None
    json.dumps(doc, allow_nan=False)


def test_profile_invariants():
    """GPT-2 with range kinds and both maps: every kernel listed exactly once;
    each operator's aggregated block is its dispatch row (kernel count,
    total ns = the sum of its kernels' durations); call indices distinct per
    operator name; each kernel's method is its tier's."""
    tr = tg.with_attribution_maps(cases.with_kinds(tg.generate("gpt2"), 2, p_boundary=0.0,
                                                   roots_boundary=True))
    match, t, walk, disp, row = _outputs(tr)
    doc = profile.build(tr, match, t["tier"], t["op"], t["fused"], row, disp["table"],
                        range_any=walk["range_any"], range_parent=walk["range_parent"])
    ids = [k["kernel_id"] for e in doc["operators"] for k in e["kernels"]]
    ids += [k["kernel_id"] for k in doc["unattributed_kernels"]]
    assert len(ids) == len(set(ids)) == tr["seq"].size
    by_id = {f"k_{int(s):05d}": i for i, s in enumerate(tr["seq"])}
    seen = {}
    for e in doc["operators"]:
        agg = e["aggregated"]
        assert agg["kernel_count"] == len(e["kernels"])
        assert agg["total_duration_ns"] == sum(k["duration_ns"] for k in e["kernels"])
        key = (e["operator_name"], e["call_index"])
        assert key not in seen
        seen[key] = True
        assert e["operator_id"] == f"{e['operator_name']}_{e['call_index']}"
        for k in e["kernels"]:
            i = by_id[k["kernel_id"]]
            assert k["attribution_method"] == profile.TIER_METHOD[int(t["tier"][i])]
            assert e["operator_name"] == f"aten::op{int(t['op'][i])}"
        assert e["is_fused"] == any(bool(t["fused"][by_id[k["kernel_id"]]]) for k in e["kernels"])
    for k in doc["unattributed_kernels"]:
        assert t["tier"][by_id[k["kernel_id"]]] == 0 and k["confidence"] is None
    assert any(e["fused_with"] for e in doc["operators"])
    json.dumps(doc, allow_nan=False)
