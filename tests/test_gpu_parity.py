"""Parity of the HIP library with the oracle, element by element, through the
C ABI (the Python binding only marshals pointers).

Covers the five workload shapes in the three emission orders (layout hints
given only where the emission fulfils them), random small traces full of
ties, each public stage on its own, the mismatch policies, data errors, and
run-to-run determinism."""
import numpy as np
import pytest

import cases
import parity
from oracle import oracle as O
from paper_2609_11938_amd import opattr, tracegen as tg

pytestmark = pytest.mark.gpu

HINTS = opattr.KERNELS_STREAM_MAJOR | opattr.SEQ_DENSE | opattr.RANGES_NESTED
DEV = "cuda:0"


@pytest.fixture(scope="module", autouse=True)
def _setup():
    import torch

    assert torch.cuda.is_available(), "GPU tests need a GPU"
    opattr.library()
    O.build(force=False)


_CACHE = {}


def _trace(cfg, emission):
    return parity.trace(cfg, emission)


def _oracle(cfg, emission):
    key = ("oracle", cfg, emission)
    if key not in _CACHE:
        _CACHE[key] = O.attribute(_trace(cfg, emission))
    return _CACHE[key]


def _run(tr, flags=0, policy=0, agg_kind=None, absent_mask=0, **kw):
    import torch

    dt = opattr.to_device(tr, DEV)
    out = opattr.opattr_attribute(dt, policy=policy, flags=flags, agg_kind=agg_kind,
                                  absent_mask=absent_mask, raise_strict=False, **kw)
    torch.cuda.synchronize()
    return out, opattr.read_diag(out["diag"])


@pytest.mark.parametrize("S,hinted", [(700, True), (1500, True), (1500, False)])
def test_many_streams(S, hinted):
    """More streams than the range stage's parent search finds tile bases for
    in each tile (1024): the bases then come from a kernel of their own.
    Nested ranges with depth on every stream, stream blocks for every
    stream, the depths written by the enclosure's extra blocks; hinted
    (stream-major, nesting order promised) and not (sorted on the device)."""
    tr = cases.random_trace(7100 + S, T=40_000, S=S, n_names=11, R=6000, n_ops=40,
                            t_max=200_000, max_depth=6, dedup=True)
    flags = 0
    if hinted:
        tr, _, _ = cases.stream_major(tr)
        flags = HINTS
    print(f"case many streams S={S} hinted={hinted} R={tr['r_start'].size}", flush=True)
    want = O.attribute(tr)
    out, diag = _run(tr, flags=flags)
    parity.assert_attribute(out, want, diag)


@pytest.mark.parametrize("cfg", ["tiny", "gpt2", "sdpa", "lstm"])
@pytest.mark.parametrize("emission", ["stream_major", "seq", "shuffled"])
def test_config_parity(cfg, emission):
    print(f"case config={cfg} emission={emission}", flush=True)
    tr = _trace(cfg, emission)
    flags = HINTS if emission == "stream_major" else (opattr.SEQ_DENSE if emission == "seq" else 0)
    want = _oracle(cfg, emission)
    out, diag = _run(tr, flags=flags)
    parity.assert_attribute(out, want, diag)


@pytest.mark.parametrize("emission,flags", [
    ("stream_major", HINTS),
    ("seq", opattr.SEQ_DENSE),
    ("shuffled", 0),
    ("stream_major", HINTS | opattr.VALIDATE),
], ids=["stream_major", "seq", "shuffled", "stream_major_validate"])
def test_large_parity_full_size(emission, flags):
    """The 10M-launch, 16-stream, dedup 48/3 trace, every output compared:
    in the benchmark's launch configuration (stream-major with every layout
    hint), in launch order (the launch-order view is a scatter), shuffled
    (no hints: the seq sort, the kernel sort by stream and query point, the
    500k-range nesting sort), and with the hints checked (VALIDATE)."""
    print(f"case config=large emission={emission} flags={flags:#x}", flush=True)
    tr = _trace("large", emission)
    want = _oracle("large", emission)
    out, diag = _run(tr, flags=flags)
    parity.assert_attribute(out, want, diag)
    assert diag["status"] == 0 and diag["order_violations"] == 0


def test_many_names_full_size():
    """More names than the LDS counters hold (5000) on the 10M-launch trace
    with dedup 48/3: the tile radix sort ranks every tile and a separate pass
    broadcasts to the duplicates."""
    print("case config=large names=5000", flush=True)
    tr = tg.generate("large", emission="stream_major", names=5000)
    assert tr["n_names"] == 5000 and int(tr["name_id"].max()) >= 4096
    want = O.attribute(tr)
    out, diag = _run(tr, flags=HINTS)
    parity.assert_attribute(out, want, diag)
    assert diag["status"] == 0


@pytest.mark.parametrize("seed", range(24))
def test_random_traces_with_ties(seed):
    tr = cases.random_trace(1000 + seed, T=3000 + 517 * seed, S=1 + seed % 5, n_names=7 + seed,
                            R=300 + 40 * seed, n_ops=13, t_max=4000, max_depth=1 + seed % 7,
                            nested=seed % 6 != 5, dedup=seed % 3 == 0,
                            drop=0.1 if seed % 4 == 1 else 0.0,
                            extra_pf=0.05 if seed % 4 == 2 else 0.0, seq_gaps=seed % 5 == 4)
    print(f"case random seed={seed} T={tr['seq'].size}", flush=True)
    want = O.attribute(tr)
    out, diag = _run(tr)  # no hints: every order accepted
    parity.assert_attribute(out, want, diag)
    if seed % 5 != 4:  # dense seq: also the hinted path on the same trace re-emitted
        sm, _, _ = cases.stream_major(tr)
        want2 = O.attribute(sm)
        out2, diag2 = _run(sm, flags=HINTS)
        parity.assert_attribute(out2, want2, diag2)


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_fused_path_random_times(seed):
    """The fused path (stream-major launches with dense seq, ranges at most
    one per 16 launches) on launches whose start times jump back and forth
    along each stream: the enclosure searches from each block's range window
    whatever the order of the query points."""
    tr = cases.random_trace(9100 + seed, T=40_000 + 997 * seed, S=2 + seed, n_names=30,
                            R=2000 + 100 * seed, n_ops=50, t_max=400_000, max_depth=5,
                            dedup=seed == 1)
    sm, _, _ = cases.stream_major(tr)
    T, R = sm["seq"].size, sm["r_start"].size
    assert R * 16 <= T
    print(f"case fused random times seed={seed} T={T} R={R}", flush=True)
    out, diag = _run(sm, flags=HINTS)
    parity.assert_attribute(out, O.attribute(sm), diag)


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_dense_seq_in_any_order(seed):
    """Launches in random storage order with seq promised dense (and ranges
    at most one per 16 launches): opattr_attribute permutes them into
    stream-major order through the launch-order view, runs the fused path and
    permutes match and range_id back."""
    tr = cases.random_trace(9300 + seed, T=40_000 + 1013 * seed, S=2 + 2 * seed, n_names=40,
                            R=2000 + 90 * seed, n_ops=60, t_max=400_000, max_depth=5,
                            dedup=seed != 1, drop=0.1 if seed == 2 else 0.0)
    T, R = tr["seq"].size, tr["r_start"].size
    assert R * 16 <= T
    print(f"case dense seq any order seed={seed} T={T} R={R}", flush=True)
    out, diag = _run(tr, flags=opattr.SEQ_DENSE)
    parity.assert_attribute(out, O.attribute(tr), diag)


@pytest.mark.parametrize("kind", ["shared_seq", "bad_stream"])
def test_dense_seq_any_order_broken(kind):
    """The permuted path on a false density promise (one seq value on two
    launches) stays within its buffers; a launch on a stream past the last
    one is counted as a bad record, as on the other paths."""
    import numpy as np

    tr = dict(cases.random_trace(9400, T=30_000, S=3, n_names=20, R=1500, n_ops=30,
                                 t_max=300_000, max_depth=4))
    if kind == "shared_seq":
        seq = tr["seq"].copy()
        seq[int(np.argmax(seq == 7))] = 8
        tr["seq"] = seq
    else:
        st = tr["stream_id"].copy()
        st[123] = 3  # n_streams is 3
        tr["stream_id"] = st
    print(f"case dense seq any order broken kind={kind}", flush=True)
    out, diag = _run(tr, flags=opattr.SEQ_DENSE)
    if kind == "bad_stream":
        assert diag["bad_records"] >= 1 and diag["status"] == -9
    else:
        assert diag["status"] <= 0  # any status: the outputs are unspecified


@pytest.mark.parametrize("R,S,t_max,nested,min_r", [(2049, 1, 300, True, 2049),
                                                    (6143, 3, 200, False, 6143),
                                                    (9001, 2, 40, False, 9001),
                                                    (20000, 5, 3000, True, 16000)])
def test_unordered_ranges_past_one_sort_tile(R, S, t_max, nested, min_r):
    """Ranges in random order, more of them than one sorting tile holds
    (2048): the merge passes of the nesting-order sort, a ragged last run,
    and (with a short time span) many identical intervals, which nest by
    index. Checked through the innermost ranges against the oracle."""
    tr = cases.random_trace(7100 + R, T=30_000, S=S, n_names=40, R=R, n_ops=31, t_max=t_max,
                            max_depth=6, nested=nested)
    print(f"case unordered ranges R={tr['r_start'].size} S={S} t_max={t_max}", flush=True)
    assert tr["r_start"].size >= min_r
    want = O.attribute(tr)
    out, diag = _run(tr)
    parity.assert_attribute(out, want, diag)


@pytest.mark.parametrize("n_names,n_ops", [(5000, 50), (7000, 7000), (4096, 6143), (4097, 6144)])
def test_many_names_and_rows(n_names, n_ops):
    """Name and operator-row counts past the LDS-counter limits take the
    tile radix sort instead; both must agree with the oracle."""
    tr = cases.random_trace(4242 + n_names, T=40_000, S=4, n_names=n_names, R=6_000,
                            n_ops=n_ops, t_max=400_000, max_depth=5, dedup=True)
    print(f"case many names={n_names} ops={n_ops} T={tr['seq'].size}", flush=True)
    want = O.attribute(tr)
    out, diag = _run(tr)
    parity.assert_attribute(out, want, diag)
    sm, _, _ = cases.stream_major(tr)
    out2, diag2 = _run(sm, flags=HINTS)
    parity.assert_attribute(out2, O.attribute(sm), diag2)


def test_layout_promises_validated():
    """Under VALIDATE a kept promise changes nothing and a broken kernel
    layout promise is reported as an order error."""
    tr = _trace("gpt2", "stream_major")
    want = _oracle("gpt2", "stream_major")
    out, diag = _run(tr, flags=HINTS | opattr.VALIDATE)
    assert diag["status"] == 0 and diag["order_violations"] == 0
    parity.assert_attribute(out, want, diag)
    bad = _trace("gpt2", "shuffled")
    _, diag2 = _run(bad, flags=HINTS | opattr.VALIDATE)
    assert diag2["status"] == -8 and diag2["order_violations"] > 0


@pytest.mark.parametrize("cfg,emission,hints", [("gpt2", "stream_major", "all"),
                                                 ("lstm", "stream_major", "all"),
                                                 ("gpt2", "seq", "dense")])
@pytest.mark.parametrize("kind", ["past_n", "shared"])
def test_broken_density_validated(cfg, emission, hints, kind):
    """Launches whose seq is not a permutation of [0, n) (every other
    promise kept): under VALIDATE the density check reports an order error
    -- a seq past n, or one seq value on two launches of different streams
    (their neighbours on each stream keep their order). Covers the segment
    path (GPT-2 shape), the fused one (LSTM shape, few ranges) and, with
    only SEQ_DENSE promised, the launch-order view."""
    import numpy as np

    tr = dict(_trace(cfg, emission))
    seq = tr["seq"].astype(np.int64).copy()
    st = tr["stream_id"]
    if kind == "past_n":
        seq[int(np.argmax(seq))] = seq.size + 5  # the largest seq: still last on its stream
    else:
        order = np.argsort(seq, kind="stable")
        k = next(j for j in range(1, order.size) if st[order[j]] != st[order[j - 1]])
        seq[order[k]] = seq[order[k - 1]]  # v + 1 on another stream becomes v
    tr["seq"] = seq.astype(np.uint32)
    flags = (HINTS if hints == "all" else opattr.SEQ_DENSE) | opattr.VALIDATE
    print(f"case broken density cfg={cfg} emission={emission} kind={kind}", flush=True)
    _, diag = _run(tr, flags=flags)
    assert diag["status"] == -8 and diag["order_violations"] > 0


def test_graph_replay_matches_eager():
    """A captured opattr_attribute (both stream branches) replays to the eager
    outputs bit for bit, replay after replay, with eager work in between."""
    import torch

    tr = _trace("gpt2", "stream_major")
    dt = opattr.to_device(tr, DEV)
    ws = opattr.Workspace(DEV)
    T, R = tr["seq"].size, tr["r_start"].size

    def outs():
        return opattr.Outputs(
            match=torch.empty(T, dtype=torch.int32, device=DEV),
            range_id=torch.empty(T, dtype=torch.int32, device=DEV),
            range_depth=torch.empty(R, dtype=torch.uint8, device=DEV),
            name_counts=torch.empty((tr["n_names"], 2), dtype=torch.int32, device=DEV),
            table=torch.empty((tr["n_ops"] + 1) * 192, dtype=torch.uint8, device=DEV),
            summary=torch.empty(40, dtype=torch.uint8, device=DEV))

    eager = opattr.opattr_attribute(dt, flags=HINTS, ws=ws, outputs=outs(), raise_strict=False)
    torch.cuda.synchronize()
    ref = {k: v.clone() for k, v in eager.items() if v is not None}
    o = outs()
    side = torch.cuda.Stream()
    with torch.cuda.stream(side):  # warm-up on the capture stream
        opattr.opattr_attribute(dt, flags=HINTS, ws=ws, outputs=o, raise_strict=False)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=side):
        opattr.opattr_attribute(dt, flags=HINTS, ws=ws, outputs=o, raise_strict=False)
    for rep in range(4):
        for k in ("match", "range_id", "table", "summary", "range_depth", "name_counts"):
            o[k].fill_(0x5A if o[k].dtype == torch.uint8 else -7)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        print(f"case graph replay {rep}", flush=True)
        for k, v in ref.items():
            if k == "diag":
                continue
            assert torch.equal(o[k], v), (rep, k)
        assert opattr.read_diag(o["diag"])["status"] == 0


@pytest.mark.parametrize("policy", [opattr.MISMATCH_SKIP_NAME, opattr.MISMATCH_STRICT])
def test_mismatch_policies(policy):
    tr = tg.generate("lstm", T=300_000, ranges=3_000, emission="stream_major")
    want = O.attribute(tr, policy=policy)
    out, diag = _run(tr, flags=HINTS, policy=policy)
    parity.assert_attribute(out, want, diag)
    if policy == opattr.MISMATCH_STRICT:
        assert diag["status"] == -4
        with pytest.raises(opattr.InvocationCountMismatchError):
            opattr.opattr_attribute(opattr.to_device(tr, DEV), policy=policy, flags=HINTS)


def test_agg_kinds_and_absent_counters():
    tr = tg.generate("gpt2", emission="seq")
    kind = np.array([opattr.AGG_DWMEAN] * 20, np.uint8)
    absent = (1 << 12) | (1 << 3)
    want = O.attribute(tr, agg_kind=kind, absent_mask=absent)
    out, diag = _run(tr, flags=opattr.SEQ_DENSE, agg_kind=kind, absent_mask=absent)
    parity.assert_attribute(out, want, diag)


def test_stages_one_by_one():
    import torch

    tr = tg.generate("gpt2", emission="shuffled")
    want = O.attribute(tr)
    dt = opattr.to_device(tr, DEV)
    m = opattr.opattr_match(dt)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(parity.host(m["match"]), want["match_iom"])
    np.testing.assert_array_equal(parity.host(m["name_counts"]).view(np.uint32),
                                  want["name_counts"])
    dd = opattr.opattr_dedup_broadcast(dt, m["match"], counters_out=True)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(parity.host(m["match"]), want["match"])
    assert opattr.read_diag(dd["diag"])["dedup_errors"] == 0
    np.testing.assert_array_equal(parity.host(dd["counters_out"]),
                                  O.counters_out(tr, want["match"]))
    e = opattr.opattr_enclose(dt)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(parity.host(e["range_id"]), want["range_id"])
    np.testing.assert_array_equal(parity.host(e["range_depth"]), want["range_depth"])
    a = opattr.opattr_aggregate(dt, m["match"], e["range_id"])
    torch.cuda.synchronize()
    parity.assert_table(a.table_host(), want["table"])
    parity.assert_summary(a.summary_host(), want["summary"])


def test_stage_dedup_and_aggregate_on_given_inputs():
    """Dedup and aggregate fed with the oracle's own intermediate outputs."""
    import torch

    tr = _trace("large", "stream_major")
    want = _oracle("large", "stream_major")
    dt = opattr.to_device(tr, DEV)
    mt = torch.from_numpy(want["match_iom"].copy()).to(DEV)
    absent = 1 << 9
    dd = opattr.opattr_dedup_broadcast(dt, mt, flags=opattr.SEQ_DENSE, counters_out=True,
                                       absent_mask=absent)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(parity.host(mt), want["match"])
    # the 10M x 20 inherited counters: every launch of a sample, one by one
    rng = np.random.default_rng(11)
    idx = np.sort(rng.choice(tr["seq"].size, 200_000, replace=False))
    got = parity.host(dd["counters_out"][torch.from_numpy(idx).to(DEV)])
    ref = O.counters_out(tr, want["match"][idx], absent_mask=absent)
    np.testing.assert_array_equal(got, ref)
    co = dd["counters_out"]
    assert int(torch.isnan(co[:, 9]).sum()) == tr["seq"].size
    unmatched = torch.from_numpy(want["match"] < 0).to(DEV)
    assert int(torch.isnan(co[unmatched]).logical_not().sum()) == 0
    del dd, co
    a = opattr.opattr_aggregate(dt, torch.from_numpy(want["match"]).to(DEV),
                                torch.from_numpy(want["range_id"]).to(DEV))
    torch.cuda.synchronize()
    parity.assert_table(a.table_host(), want["table"])


def test_determinism_and_poisoned_outputs():
    import torch

    tr = tg.generate("sdpa", emission="stream_major")
    dt = opattr.to_device(tr, DEV)
    runs = []
    for poison in (0x5A, 0xA7):
        outs = opattr.Outputs(
            match=torch.full((tr["seq"].size,), poison, dtype=torch.int32, device=DEV),
            range_id=torch.full((tr["seq"].size,), poison, dtype=torch.int32, device=DEV),
            range_depth=torch.full((tr["r_start"].size,), poison, dtype=torch.uint8, device=DEV),
            name_counts=torch.full((tr["n_names"], 2), poison, dtype=torch.int32, device=DEV),
            table=torch.full(((tr["n_ops"] + 1) * 192,), poison, dtype=torch.uint8, device=DEV),
            summary=torch.full((40,), poison, dtype=torch.uint8, device=DEV))
        out = opattr.opattr_attribute(dt, flags=HINTS, outputs=outs)
        torch.cuda.synchronize()
        runs.append((parity.host(out["match"]).copy(), parity.host(out["range_id"]).copy(),
                     parity.host(out["range_depth"]).copy(), out.table_host().copy()))
    want = O.attribute(tr)
    for r in runs:
        np.testing.assert_array_equal(r[0], want["match"])
        np.testing.assert_array_equal(r[1], want["range_id"])
        np.testing.assert_array_equal(r[2], want["range_depth"])
        parity.assert_table(r[3], want["table"])
    for k in range(3):
        np.testing.assert_array_equal(runs[0][k], runs[1][k])
    for f in ("kernel_count", "total_ns", "matched_count", "matched_ns"):
        np.testing.assert_array_equal(runs[0][3][f], runs[1][3][f])


def test_timestamps_do_not_move_matches():
    tr = tg.generate("lstm", T=200_000, ranges=2_000)
    out0, _ = _run(tr, flags=HINTS)
    rng = np.random.default_rng(3)
    tr2 = dict(tr, start_ns=np.sort(rng.integers(0, 2**40, size=tr["seq"].size)).astype(np.uint64))
    out1, _ = _run(tr2)
    np.testing.assert_array_equal(parity.host(out0["match"]), parity.host(out1["match"]))


def _small(T=40):
    return cases.random_trace(77, T=T, S=2, R=12, t_max=50, dedup=True)


def test_error_classes_match_oracle():
    base = _small()
    variants = []
    t = dict(base, name_id=base["name_id"].copy())
    t["name_id"][3] = 10_000  # bad name
    variants.append(t)
    t = dict(base, r_op=base["r_op"].copy())
    t["r_op"][0] = 10_000  # bad op id
    variants.append(t)
    t = dict(base, seq=base["seq"].copy())
    t["seq"][0] = t["seq"][1]  # duplicate seq
    variants.append(t)
    t = dict(base, r_start=np.concatenate([base["r_start"], [5, 8]]).astype(np.uint64),
             r_end=np.concatenate([base["r_end"], [10, 20]]).astype(np.uint64),
             r_stream=np.concatenate([base["r_stream"], [0, 0]]).astype(np.uint16),
             r_op=np.concatenate([base["r_op"], [1, 2]]).astype(np.uint32))  # crossing
    variants.append(t)
    if base["part_id"] is not None:
        t = dict(base, part_id=base["part_id"].copy())
        order = np.argsort(t["seq"])
        p = t["part_id"][order]
        first = np.flatnonzero(p >= 0)[0]
        p[first], p[first + 1] = -1, p[first]  # a hole inside partition 0
        t["part_id"][order] = p
        variants.append(t)
    for k, tr in enumerate(variants):
        print(f"case error variant {k}", flush=True)
        want = O.attribute(tr)
        out, diag = _run(tr)
        assert diag["status"] == want["diag"]["status"] != 0, (k, diag, want["diag"])
        parity.assert_diag(diag, want["diag"])
        if want["diag"]["status"] not in (-8,):  # outputs are defined except for order errors
            parity.assert_attribute(out, want, diag)


def _walk_gpu(tr, flags=0):
    import torch

    dt = opattr.to_device(tr, DEV)
    out = opattr.opattr_enclose_walk(dt, flags=flags)
    torch.cuda.synchronize()
    return out, opattr.read_diag(out["diag"])


def _assert_walk(out, want, diag):
    for f in ("range_id", "fused", "range_any", "range_parent", "range_depth"):
        np.testing.assert_array_equal(parity.host(out[f]), want[f], err_msg=f)
    parity.assert_diag(diag, want["diag"])


@pytest.mark.parametrize("seed", range(10))
def test_enclose_walk_parity(seed):
    """Alg. 2's walk with range kinds: every output of the walk entry point
    against the oracle, on random nested traces (some with invalid kinds),
    in every emission order."""
    emission = ("stream_major", "seq", "shuffled")[seed % 3]
    print(f"case walk seed={seed} emission={emission}", flush=True)
    tr = cases.random_trace(900 + seed, T=400, R=120, S=1 + seed % 4, t_max=300, max_depth=6)
    tr = cases.with_kinds(tr, seed, p_bad=0.05 if seed % 5 == 4 else 0.0,
                          roots_boundary=seed % 2 == 0)
    flags = 0
    if emission == "stream_major":
        tr = cases.stream_major(tr)[0]
        flags = opattr.KERNELS_STREAM_MAJOR | opattr.RANGES_NESTED
    want = O.enclose_walk(tr)
    out, diag = _walk_gpu(tr, flags)
    _assert_walk(out, want, diag)


@pytest.mark.parametrize("seed", range(6))
def test_enclose_walk_touching_ranges(seed):
    """Coarse timestamps: many ranges end exactly where the next one starts
    and many launches sit on those points, where a range that only touches
    the innermost one still contains the launch (closed intervals): the walk
    must visit it (fused, the op chosen) as the oracle's stack does."""
    print(f"case walk touching seed={seed}", flush=True)
    tr = cases.random_trace(950 + seed, T=500, R=150, S=1 + seed % 2, t_max=60, max_depth=6)
    tr = cases.with_kinds(tr, seed, p_boundary=0.1 * (seed % 2), p_skip=0.3)
    flags = 0
    if seed % 3 == 0:
        tr = cases.stream_major(tr)[0]
        flags = opattr.KERNELS_STREAM_MAJOR | opattr.RANGES_NESTED
    want = O.enclose_walk(tr)
    out, diag = _walk_gpu(tr, flags)
    _assert_walk(out, want, diag)
    no_kinds = dict(tr, r_kind=None)
    want = O.enclose_walk(no_kinds)
    out, diag = _walk_gpu(no_kinds, flags)
    _assert_walk(out, want, diag)


def test_enclose_walk_large_with_kinds():
    """The 10M-launch trace with profiler-step roots (boundaries) and skipped
    namespaces: the walk outputs, and the whole attribution following the
    walk (operator rows from the innermost op before a boundary)."""
    print("case walk large", flush=True)
    tr = cases.with_kinds(_trace("large", "stream_major"), 5, p_boundary=0.0, p_skip=0.2,
                          roots_boundary=True)
    want = O.enclose_walk(tr)
    out, diag = _walk_gpu(tr, HINTS)
    _assert_walk(out, want, diag)
    want_all = O.attribute(tr)
    got, gdiag = _run(tr, flags=HINTS)
    parity.assert_attribute(got, want_all, gdiag)


def test_enclose_walk_without_kinds_is_innermost():
    print("case walk no kinds", flush=True)
    tr = _trace("gpt2", "stream_major")
    want = O.enclose_walk(tr)
    out, diag = _walk_gpu(tr, HINTS)
    _assert_walk(out, want, diag)
    np.testing.assert_array_equal(parity.host(out["range_id"]), tr["planted_range"])


def test_deep_nesting_limit():
    T, depth = 8, 300
    r_start = np.arange(depth, dtype=np.uint64)
    r_end = (10_000 - np.arange(depth)).astype(np.uint64)
    tr = dict(seq=np.arange(T, dtype=np.uint32), start_ns=np.full(T, 5000, np.uint64),
              dur_ns=np.ones(T, np.uint32), stream_id=np.zeros(T, np.uint16),
              name_id=np.zeros(T, np.uint32), part_id=None, pf_name=np.zeros(T, np.uint32),
              counters=np.ones((T, 20), np.float32), r_start=r_start, r_end=r_end,
              r_stream=np.zeros(depth, np.uint16), r_op=np.zeros(depth, np.uint32),
              part_rep=None, n_names=1, n_streams=1, n_ops=1)
    want = O.attribute(tr)
    out, diag = _run(tr, flags=HINTS)
    assert want["diag"]["status"] == diag["status"] == -10
    np.testing.assert_array_equal(parity.host(out["range_depth"]), want["range_depth"])


def test_empty_inputs():
    z = np.zeros(0)
    tr = dict(seq=z.astype(np.uint32), start_ns=z.astype(np.uint64), dur_ns=z.astype(np.uint32),
              stream_id=z.astype(np.uint16), name_id=z.astype(np.uint32), part_id=None,
              pf_name=z.astype(np.uint32), counters=np.zeros((0, 20), np.float32),
              r_start=z.astype(np.uint64), r_end=z.astype(np.uint64),
              r_stream=z.astype(np.uint16), r_op=z.astype(np.uint32), part_rep=None,
              n_names=3, n_streams=2, n_ops=4)
    want = O.attribute(tr)
    out, diag = _run(tr)
    parity.assert_attribute(out, want, diag)


def _assert_all(out, want):
    import torch

    torch.cuda.synchronize()
    np.testing.assert_array_equal(parity.host(out["off"]), want["off"])
    np.testing.assert_array_equal(parity.host(out["ids"]), want["ids"])
    diag = opattr.read_diag(out["diag"])
    for f in ("status", "bad_records", "nesting_errors"):
        assert diag[f] == want["diag"][f], (f, diag, want["diag"])


@pytest.mark.parametrize("seed", range(6))
def test_enclose_all_parity(seed):
    """Every enclosing range of every launch (CSR, innermost first) against
    the oracle's stack sweep, coarse timestamps (launches on range edges),
    some ranges with bad ids, each emission order."""
    print(f"case enclose_all seed={seed}", flush=True)
    tr = cases.random_trace(970 + seed, T=600, R=200, S=1 + seed % 3, t_max=80 + 200 * (seed % 2),
                            max_depth=6)
    tr = cases.with_kinds(tr, seed, p_bad=0.05 if seed % 3 == 2 else 0.0)
    flags = 0
    if seed % 2 == 0:
        tr = cases.stream_major(tr)[0]
        flags = opattr.KERNELS_STREAM_MAJOR | opattr.RANGES_NESTED
    want = O.enclose_all(tr)
    out = opattr.opattr_enclose_all(opattr.to_device(tr, DEV), flags=flags)
    _assert_all(out, want)


def test_enclose_all_bad_streams_and_capacity():
    """Launches on stream ids past n_streams get empty lists and count as
    bad records; a capacity below the total writes exactly the lists that
    end within it (the offsets stay complete)."""
    import torch

    print("case enclose_all bad streams", flush=True)
    tr = cases.random_trace(995, T=300, R=80, S=3, t_max=60, max_depth=5)
    tr["stream_id"] = tr["stream_id"].copy()
    tr["stream_id"][[3, 77, 150]] = 7
    want = O.enclose_all(tr)
    dt = opattr.to_device(tr, DEV)
    out = opattr.opattr_enclose_all(dt)
    torch.cuda.synchronize()
    off = parity.host(out["off"])
    np.testing.assert_array_equal(off, want["off"])
    np.testing.assert_array_equal(parity.host(out["ids"]), want["ids"])
    diag = opattr.read_diag(out["diag"])
    assert diag["bad_records"] == want["diag"]["bad_records"] == 3
    assert all(off[i + 1] == off[i] for i in (3, 77, 150))
    cap = int(off[-1]) // 2
    part = opattr.opattr_enclose_all(dt, ids=torch.full((max(cap, 1),), -7, dtype=torch.int32,
                                                          device=DEV))
    torch.cuda.synchronize()
    got = parity.host(part["ids"])
    last = np.searchsorted(off, cap, side="right") - 1
    np.testing.assert_array_equal(got[:off[last]], want["ids"][:off[last]])
    assert np.all(got[off[last]:cap] == -7)


def test_enclose_all_crossing_ranges_reported():
    """Crossing ranges: the list call reports them as the oracle does (count
    of streams with a crossing, NOT_NESTED status); the lists are then
    unspecified and only their offsets' consistency is checked."""
    import torch

    for seed in range(3):
        print(f"case enclose_all crossing seed={seed}", flush=True)
        tr = cases.random_trace(990 + seed, T=60, R=30, S=1 + seed % 3, t_max=40, nested=False)
        want = O.enclose_all(tr)
        out = opattr.opattr_enclose_all(opattr.to_device(tr, DEV))
        torch.cuda.synchronize()
        diag = opattr.read_diag(out["diag"])
        for f in ("status", "bad_records", "nesting_errors"):
            assert diag[f] == want["diag"][f], (f, diag, want["diag"])
        off = parity.host(out["off"])
        assert off[0] == 0 and np.all(np.diff(off) >= 0)


@pytest.mark.parametrize("cfg", ["sdpa", "large"])
def test_enclose_all_generated(cfg):
    """The generated workloads: one list per launch over up to 8 levels."""
    print(f"case enclose_all {cfg}", flush=True)
    tr = parity.trace(cfg, "stream_major")
    want = O.enclose_all(tr)
    out = opattr.opattr_enclose_all(opattr.to_device(tr, DEV), flags=HINTS)
    _assert_all(out, want)


@pytest.mark.parametrize("emission", ["stream_major", "seq"])
def test_default_kinds_are_the_counter_table(emission):
    """The library's default aggregation kinds equal the transcribed Agg.
    column of the counter reference table: passing the column explicitly
    gives the default's table (stream_major: the fused path; seq: the
    general one)."""
    import test_oracle

    tr = tg.generate("lstm" if emission == "stream_major" else "gpt2", emission=emission)
    flags = HINTS if emission == "stream_major" else opattr.SEQ_DENSE
    a, _ = _run(tr, flags=flags)
    b, _ = _run(tr, flags=flags, agg_kind=test_oracle.golden_kinds())
    parity.assert_table(a.table_host(), b.table_host(), rtol=1e-12)
