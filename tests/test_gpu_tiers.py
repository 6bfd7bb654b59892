"""Tiered attribution on the GPU against the oracle, through the C ABI: the
tier, operator and fused flag of every launch, the coverage record and the
diagnostics, on random traces (range kinds, partitions, correlation maps
with gaps, count mismatches, interleaved names and bad operator ids, fusion
maps), the generated workloads in every emission order, the 10M-launch
trace, and the operator table by tier operator (Eq. 1)."""
import numpy as np
import pytest

import cases
import parity
from oracle import oracle as O
from paper_2609_11938_amd import opattr, tracegen as tg

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
HINTS = opattr.KERNELS_STREAM_MAJOR | opattr.SEQ_DENSE | opattr.RANGES_NESTED
DIAG = ("status", "flags", "bad_records", "names_mismatched", "tl_unmatched", "pf_unmatched")


@pytest.fixture(scope="module", autouse=True)
def _setup():
    import torch

    assert torch.cuda.is_available(), "GPU tests need a GPU"
    opattr.library()
    O.build(force=False)


def _gpu_tiers(tr, policy=1, flags=0, walk_from_oracle=None):
    import torch

    dt = opattr.to_device(tr, DEV)
    if walk_from_oracle is None:
        w = opattr.opattr_enclose_walk(dt, flags=flags)
        rid, wf = w["range_id"], w["fused"]
    else:
        rid = torch.from_numpy(walk_from_oracle["range_id"]).to(DEV)
        wf = torch.from_numpy(walk_from_oracle["walk_fused"]).to(DEV)
    out = opattr.opattr_tiers(dt, rid, wf, corr_policy=policy, flags=flags)
    torch.cuda.synchronize()
    return out, opattr.read_diag(out["diag"])


def _assert_tiers(out, diag, want):
    for f in ("tier", "op", "fused"):
        np.testing.assert_array_equal(parity.host(out[f]), want[f], err_msg=f)
    cov = out.coverage_host()
    np.testing.assert_array_equal(cov["count"], want["coverage"]["count"])
    np.testing.assert_array_equal(cov["ns"], want["coverage"]["ns"])
    np.testing.assert_array_equal(cov["frac"], want["coverage"]["frac"])
    for f in DIAG:
        assert diag[f] == want["diag"][f], (f, diag, want["diag"])


def _tier_trace(seed, T=400, dedup=False, shuffle=False, p_bad=0.0):
    tr = cases.random_trace(600 + seed, T=T, R=120, S=1 + seed % 4, t_max=300, max_depth=6,
                            dedup=dedup)
    tr = cases.with_kinds(tr, seed)
    return tg.with_attribution_maps(tr, seed=seed, p_corr=0.6, p_mismatch=0.3, p_none=0.1,
                                    p_fmap=0.5, p_bad=p_bad, shuffle=shuffle)


@pytest.mark.parametrize("seed", range(8))
@pytest.mark.parametrize("policy", [0, 1, 2])
def test_tiers_parity(seed, policy):
    print(f"case tiers seed={seed} policy={policy}", flush=True)
    tr = _tier_trace(seed, dedup=seed % 2 == 0, shuffle=seed % 3 == 1,
                     p_bad=0.05 if seed % 4 == 3 else 0.0)
    want = O.tiers(tr, corr_policy=policy)
    out, diag = _gpu_tiers(tr, policy)
    _assert_tiers(out, diag, want)


@pytest.mark.parametrize("cfg", ["tiny", "gpt2", "sdpa", "lstm"])
@pytest.mark.parametrize("emission", ["stream_major", "seq", "shuffled"])
def test_tiers_generated(cfg, emission):
    """The generated workloads with range kinds and maps; layout hints where
    the emission keeps them."""
    print(f"case tiers {cfg}/{emission}", flush=True)
    tr = cases.with_kinds(parity.trace(cfg, emission), 4, p_boundary=0.0, p_skip=0.2,
                          roots_boundary=True)
    tr = tg.with_attribution_maps(tr, seed=11, shuffle=emission == "shuffled")
    flags = {"stream_major": HINTS, "seq": opattr.SEQ_DENSE, "shuffled": 0}[emission]
    want = O.tiers(tr)
    out, diag = _gpu_tiers(tr, flags=flags, walk_from_oracle=want)
    _assert_tiers(out, diag, want)


def test_tiers_large():
    """The 10M-launch trace with profiler-step boundaries, skipped ranges, a
    correlation map for 40% of the names and a fusion map; the whole GPU
    chain (walk, then tiers)."""
    print("case tiers large", flush=True)
    tr = tg.with_attribution_maps(tg.with_range_kinds(parity.trace("large", "stream_major")))
    want = O.tiers(tr)
    out, diag = _gpu_tiers(tr, flags=HINTS)
    _assert_tiers(out, diag, want)
    assert want["coverage"]["frac"][opattr.TIER_HIGH] > 0.2


def test_tiers_without_maps_and_empty():
    print("case tiers no maps", flush=True)
    tr = cases.with_kinds(parity.trace("tiny", "stream_major"), 2)
    want = O.tiers(tr)
    out, diag = _gpu_tiers(tr, flags=HINTS)
    _assert_tiers(out, diag, want)
    # maps present but empty: no entries, every fusion list empty
    tr = dict(tr, corr_name=np.zeros(0, np.uint32), corr_op=np.zeros(0, np.int32),
              fmap_off=np.zeros(tr["n_names"] + 1, np.uint32), fmap_op=np.zeros(0, np.int32))
    want = O.tiers(tr, corr_policy=0)
    out, diag = _gpu_tiers(tr, policy=0, flags=HINTS)
    _assert_tiers(out, diag, want)


@pytest.mark.parametrize("cfg", ["tiny", "gpt2"])
def test_aggregate_ops_parity(cfg):
    """Eq. 1 by tier operator: the oracle's table given the oracle's match
    and ops, on the GPU; a few operators out of range are bad records."""
    import torch

    print(f"case aggregate_ops {cfg}", flush=True)
    tr = tg.with_attribution_maps(cases.with_kinds(parity.trace(cfg, "stream_major"), 1))
    match = O.attribute(tr, stages=["match", "dedup"])["match"]
    op = O.tiers(tr)["op"].copy()
    op[:2] = [tr["n_ops"] + 4, -3]
    want = O.aggregate_ops(tr, match, op)
    dt = opattr.to_device(tr, DEV)
    out = opattr.opattr_aggregate_ops(dt, torch.from_numpy(match).to(DEV),
                                      torch.from_numpy(op).to(DEV))
    torch.cuda.synchronize()
    diag = opattr.read_diag(out["diag"])
    parity.assert_table(out.table_host(), want["table"])
    assert diag["bad_records"] == want["diag"]["bad_records"] == 2
    assert diag["status"] == want["diag"]["status"]


@pytest.mark.parametrize("T", [2_000_000, 9_000_000])
def test_aggregate_ops_heavy_rows(T):
    """Rows whose items span hundreds of thousands of windows: every launch
    alternates between the UNATTRIBUTED row and operator 0 (one item each),
    so both rows are reduced in chunks of 256 windows; at 9M launches each
    row has more than 256 chunks. Random matches, some unmatched."""
    import torch

    print(f"case aggregate_ops heavy rows T={T}", flush=True)
    rng = np.random.default_rng(T)
    tr = cases.random_trace(5, T=64, R=8, n_ops=3)
    P = 200_000
    tr.update(seq=np.arange(T, dtype=np.uint32), start_ns=np.arange(T, dtype=np.uint64) * 10,
              dur_ns=rng.integers(1, 5000, size=T).astype(np.uint32),
              stream_id=np.zeros(T, np.uint16), name_id=np.zeros(T, np.uint32), part_id=None,
              pf_name=np.zeros(P, np.uint32),
              counters=rng.random((P, 20), dtype=np.float32), part_rep=None, n_parts=0)
    match = rng.integers(-1, P, size=T).astype(np.int32)
    op = np.where(np.arange(T) % 2 == 0, -1, 0).astype(np.int32)
    want = O.aggregate_ops(tr, match, op)
    dt = opattr.to_device(tr, DEV)
    out = opattr.opattr_aggregate_ops(dt, torch.from_numpy(match).to(DEV),
                                      torch.from_numpy(op).to(DEV))
    torch.cuda.synchronize()
    diag = opattr.read_diag(out["diag"])
    parity.assert_table(out.table_host(), want["table"])
    assert diag["status"] == want["diag"]["status"] == 0


def test_attribute_tiered_pipeline():
    """The tiered pipeline as library calls (match + dedup broadcast, walk,
    tiers, table by tier operator) against the oracle's stages on GPT-2
    (layer dedup on)."""
    import torch

    print("case tiered pipeline gpt2", flush=True)
    tr = tg.with_attribution_maps(cases.with_kinds(parity.trace("gpt2", "stream_major"), 3,
                                                   p_boundary=0.0, roots_boundary=True))
    match = O.attribute(tr, stages=["match", "dedup"])["match"]
    wt = O.tiers(tr)
    want = O.aggregate_ops(tr, match, wt["op"])
    dt = opattr.to_device(tr, DEV)
    res = opattr.attribute_tiered(dt, flags=HINTS)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(parity.host(res["match"]["match"]), match)
    _assert_tiers(res["tiers"], opattr.read_diag(res["tiers"]["diag"]), wt)
    parity.assert_table(res["aggregate"].table_host(), want["table"])


def _gpu_dispatch(tr, match, range_id, op, flags=0):
    import torch

    dt = opattr.to_device(tr, DEV)
    out = opattr.opattr_aggregate_dispatch(
        dt, torch.from_numpy(np.ascontiguousarray(match, np.int32)).to(DEV),
        torch.from_numpy(np.ascontiguousarray(range_id, np.int32)).to(DEV),
        None if op is None else torch.from_numpy(np.ascontiguousarray(op, np.int32)).to(DEV),
        flags=flags)
    torch.cuda.synchronize()
    return out, opattr.read_diag(out["diag"])


@pytest.mark.parametrize("seed", range(6))
def test_dispatch_parity(seed):
    """The per-dispatch table (ranges, then per-operator rows, then the
    unattributed row) against the oracle, with tier operators and without;
    a few bad range ids and operators."""
    print(f"case dispatch seed={seed}", flush=True)
    tr = _tier_trace(seed, dedup=seed % 2 == 0)
    match = O.attribute(tr, stages=["match", "dedup"])["match"]
    t = O.tiers(tr)
    rid, op = t["range_id"].copy(), t["op"].copy()
    if seed % 3 == 2:
        rid[:2] = [tr["r_start"].size + 1, -4]
        op[2:4] = [tr["n_ops"], -2]
    for o in (op, None):
        want = O.aggregate_dispatch(tr, match, rid, o)
        out, diag = _gpu_dispatch(tr, match, rid, o)
        parity.assert_table(out.table_host(), want["table"])
        assert diag["bad_records"] == want["diag"]["bad_records"]
        assert diag["status"] == want["diag"]["status"]
        parity.assert_summary(out.summary_host(), want["summary"])


@pytest.mark.parametrize("cfg", ["gpt2", "sdpa", "large"])
def test_dispatch_generated(cfg):
    """Tens of thousands to half a million dispatch rows (one radix sort of
    the items by row): the tiered pipeline's dispatch table against the
    oracle's."""
    print(f"case dispatch {cfg}", flush=True)
    tr = tg.with_attribution_maps(tg.with_range_kinds(parity.trace(cfg, "stream_major")))
    match = O.attribute(tr, stages=["match", "dedup"])["match"]
    t = O.tiers(tr)
    want = O.aggregate_dispatch(tr, match, t["range_id"], t["op"])
    out, diag = _gpu_dispatch(tr, match, t["range_id"], t["op"], flags=HINTS)
    parity.assert_table(out.table_host(), want["table"])
    parity.assert_summary(out.summary_host(), want["summary"])
    assert diag["status"] == want["diag"]["status"] == 0


def _same_doc(a, b, path="doc"):
    """Equal JSON-like values, floats within the aggregation tolerance."""
    if isinstance(a, dict):
        assert isinstance(b, dict) and a.keys() == b.keys(), path
        for k in a:
            _same_doc(a[k], b[k], f"{path}.{k}")
    elif isinstance(a, list):
        assert isinstance(b, list) and len(a) == len(b), path
        for i, (x, y) in enumerate(zip(a, b)):
            _same_doc(x, y, f"{path}[{i}]")
    elif isinstance(a, float) and isinstance(b, float):
        assert abs(a - b) <= parity.RTOL * max(abs(a), abs(b)), (path, a, b)
    else:
        assert a == b, (path, a, b)


def test_profile_from_gpu_outputs():
    """profile.json built from the GPU pipeline's outputs (tiers, the walk's
    range links, the per-dispatch rows and table) equals the one built from
    the oracle's, GPT-2 with range kinds and both maps."""
    import torch

    from paper_2609_11938_amd import profile

    print("case profile.json gpt2", flush=True)
    tr = tg.with_attribution_maps(cases.with_kinds(parity.trace("gpt2", "stream_major"), 2,
                                                   p_boundary=0.0, roots_boundary=True))
    dt = opattr.to_device(tr, DEV)
    res = opattr.attribute_tiered(dt, flags=HINTS, dispatch=True)
    torch.cuda.synchronize()
    h = parity.host
    got = profile.build(tr, h(res["match"]["match"]), h(res["tiers"]["tier"]),
                        h(res["tiers"]["op"]), h(res["tiers"]["fused"]), h(res["dispatch"]["row"]),
                        res["dispatch"].table_host(), range_any=h(res["walk"]["range_any"]),
                        range_parent=h(res["walk"]["range_parent"]))
    match = O.attribute(tr, stages=["match", "dedup"])["match"]
    t = O.tiers(tr)
    walk = O.enclose_walk(tr)
    disp = O.aggregate_dispatch(tr, match, t["range_id"], t["op"])
    import brute
    row = np.array(brute.dispatch_keys(tr, t["range_id"], t["op"]))
    np.testing.assert_array_equal(h(res["dispatch"]["row"]), row)
    want = profile.build(tr, match, t["tier"], t["op"], t["fused"], row, disp["table"],
                         range_any=walk["range_any"], range_parent=walk["range_parent"])
    _same_doc(got, want)


def _empty_trace(T, R):
    tr = cases.random_trace(31, T=max(T, 1), R=max(R, 1), S=2, n_names=3)
    if T == 0:
        for f in ("seq", "start_ns", "dur_ns", "stream_id", "name_id", "part_id", "query_ns"):
            if tr.get(f) is not None:
                tr[f] = tr[f][:0]
    if R == 0:
        for f in ("r_start", "r_end", "r_stream", "r_op", "r_kind"):
            if tr.get(f) is not None:
                tr[f] = tr[f][:0]
    return tr


@pytest.mark.parametrize("T,R", [(0, 5), (7, 0), (0, 0)])
def test_next_rows_on_empty_inputs(T, R):
    """No launches and/or no ranges: tiers (with an empty correlation map and
    an empty fusion map), the table by operator, the per-dispatch table and
    the CSR lists all equal the oracle's."""
    import torch

    print(f"case next rows empty T={T} R={R}", flush=True)
    tr = _empty_trace(T, R)
    tr.update(corr_name=np.zeros(0, np.uint32), corr_op=np.zeros(0, np.int32),
              fmap_off=np.zeros(tr["n_names"] + 1, np.uint32), fmap_op=np.zeros(0, np.int32))
    want = O.tiers(tr, corr_policy=0)
    out, diag = _gpu_tiers(tr, policy=0)
    _assert_tiers(out, diag, want)
    match = np.full(T, -1, np.int32)
    dt = opattr.to_device(tr, DEV)
    agg = opattr.opattr_aggregate_ops(dt, torch.from_numpy(match).to(DEV), out["op"])
    torch.cuda.synchronize()
    parity.assert_table(agg.table_host(), O.aggregate_ops(tr, match, want["op"])["table"])
    dout, ddiag = _gpu_dispatch(tr, match, want["range_id"], want["op"])
    dwant = O.aggregate_dispatch(tr, match, want["range_id"], want["op"])
    parity.assert_table(dout.table_host(), dwant["table"])
    assert ddiag["status"] == dwant["diag"]["status"]
    aw = O.enclose_all(tr)
    ao = opattr.opattr_enclose_all(dt)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(parity.host(ao["off"]), aw["off"])
    assert int(ao["ids"].numel()) == 0


@pytest.mark.parametrize("case", ["random0", "random1", "gpt2", "large"])
def test_attribute_tiered_one_call(case):
    """opattr_attribute_tiered against the oracle's stages: matching with the
    dedup broadcast, the walk's range ids and fused flags, the tiers and
    coverage, the table by tier operator; the diag record covers both
    matchings, the walk and the tiers."""
    import torch

    print(f"case attribute_tiered {case}", flush=True)
    if case.startswith("random"):
        seed = int(case[-1])
        tr = _tier_trace(40 + seed, dedup=seed == 0, shuffle=seed == 1,
                         p_bad=0.05 if seed == 1 else 0.0)
        flags = 0
    else:
        tr = tg.with_attribution_maps(tg.with_range_kinds(parity.trace(case, "stream_major")))
        flags = HINTS
    att = O.attribute(tr, stages=["match", "dedup"])
    t = O.tiers(tr)
    walk = O.enclose_walk(tr)
    agg = O.aggregate_ops(tr, att["match"], t["op"])
    dt = opattr.to_device(tr, DEV)
    out = opattr.opattr_attribute_tiered(dt, flags=flags)
    torch.cuda.synchronize()
    h = parity.host
    np.testing.assert_array_equal(h(out["match"]), att["match"])
    np.testing.assert_array_equal(h(out["range_id"]), walk["range_id"])
    _assert_tiers(out, opattr.read_diag(out["diag"]) | {f: t["diag"][f] for f in DIAG}, t)
    parity.assert_table(out.table_host(), agg["table"])
    parity.assert_summary(out.summary_host(), agg["summary"])
    diag = opattr.read_diag(out["diag"])
    bad = att["diag"]["bad_records"] + t["diag"]["bad_records"] + walk["diag"]["bad_records"]
    assert diag["bad_records"] == bad
    ok = att["diag"]["status"] == t["diag"]["status"] == walk["diag"]["status"] == 0
    assert (diag["status"] == 0) == ok


@pytest.mark.parametrize("n_names,n_ops", [(4096, 6143), (4097, 6144)])
def test_attribute_tiered_at_path_boundaries(n_names, n_ops):
    """Either side of the LDS-ranking limit on names (4096) and of the
    per-tile item histograms on operator rows (6144): the one-call tiered
    attribution still equals the oracle's stages."""
    import torch

    print(f"case tiered names={n_names} ops={n_ops}", flush=True)
    tr = cases.random_trace(77, T=30_000, S=3, n_names=n_names, R=5_000, n_ops=n_ops,
                            t_max=300_000, max_depth=5, dedup=True)
    tr = tg.with_attribution_maps(cases.with_kinds(tr, 3), seed=5)
    att = O.attribute(tr, stages=["match", "dedup"])
    t = O.tiers(tr)
    agg = O.aggregate_ops(tr, att["match"], t["op"])
    out = opattr.opattr_attribute_tiered(opattr.to_device(tr, DEV))
    torch.cuda.synchronize()
    np.testing.assert_array_equal(parity.host(out["match"]), att["match"])
    for f in ("tier", "op", "fused"):
        np.testing.assert_array_equal(parity.host(out[f]), t[f], err_msg=f)
    parity.assert_table(out.table_host(), agg["table"])


@pytest.mark.parametrize("side", ["profiled", "corr"])
@pytest.mark.parametrize("policy,corr_policy", [(0, 2), (2, 1), (2, 2), (1, 0)])
def test_attribute_tiered_policy_mix(side, policy, corr_policy):
    """The two matchings of the one-call tiered attribution under different
    count policies, with a count mismatch in the correlation map (entries
    missing at the end of some names) and, or not, in the profiled rows
    (missing rows): outputs
    as the oracle's stages, the count diagnostics of both matchings added up,
    and COUNT_MISMATCH exactly when either policy is STRICT and either side
    has a mismatch."""
    import torch

    print(f"case tiered policy mix side={side} policy={policy} corr={corr_policy}", flush=True)
    tr = cases.random_trace(901, T=3000, S=2, n_names=12, R=400, n_ops=30, t_max=6000,
                            max_depth=4, drop=0.1 if side == "profiled" else 0.0)
    tr = tg.with_attribution_maps(cases.with_kinds(tr, 1), seed=3, p_corr=0.6,
                                  p_mismatch=0.4 if side == "corr" else 0.0, p_none=0.1,
                                  p_fmap=0.4)
    att = O.attribute(tr, policy=policy, stages=["match", "dedup"])
    t = O.tiers(tr, corr_policy=corr_policy)
    assert bool(att["diag"]["flags"] & O.F_COUNT) == (side == "profiled")
    assert bool(t["diag"]["flags"] & O.F_COUNT)
    out = opattr.opattr_attribute_tiered(opattr.to_device(tr, DEV), policy=policy,
                                         corr_policy=corr_policy)
    torch.cuda.synchronize()
    diag = opattr.read_diag(out["diag"])
    np.testing.assert_array_equal(parity.host(out["match"]), att["match"])
    for f in ("tier", "op", "fused"):
        np.testing.assert_array_equal(parity.host(out[f]), t[f], err_msg=f)
    for f in ("names_mismatched", "tl_unmatched", "pf_unmatched"):
        assert diag[f] == att["diag"][f] + t["diag"][f], f
    strict = opattr.MISMATCH_STRICT in (policy, corr_policy)
    assert (diag["status"] == -4) == strict, diag
    assert bool(diag["flags"] & O.F_COUNT)
