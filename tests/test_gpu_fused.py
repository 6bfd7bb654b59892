"""Parity of the fused attribution path (kernels stream-major with dense
seq, at most one range per 16 launches, at most 16384 operator rows): the
matching stops at the eligible launches, one pass resolves every launch's
match with the dedup broadcast, one pass reduces the runs of launches of one
operator row (block partials sorted by row bucket, then added per bucket).

Random traces with ties, partitions, drops, extra profiled rows, range kinds
and non-default aggregation kinds, sized so that some blocks hold more runs
than they keep (the rest go through the row accumulators)."""
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


def _run(tr, flags=HINTS, **kw):
    import torch

    out = opattr.opattr_attribute(opattr.to_device(tr, DEV), flags=flags, raise_strict=False, **kw)
    torch.cuda.synchronize()
    return out, opattr.read_diag(out["diag"])


@pytest.mark.parametrize("seed", range(16))
def test_fused_random(seed):
    T = 20_000 + 1777 * seed
    tr = cases.random_trace(5000 + seed, T=T, S=1 + seed % 6, n_names=7 + 3 * seed,
                            R=T // (17 + 7 * (seed % 4)), n_ops=13 + 50 * seed,
                            t_max=T * (3 + seed % 5), max_depth=1 + seed % 7,
                            dedup=seed % 2 == 0, drop=0.1 if seed % 4 == 1 else 0.0,
                            extra_pf=0.05 if seed % 4 == 2 else 0.0)
    tr, _, _ = cases.stream_major(tr)
    if seed % 5 == 3:
        tr = cases.with_kinds(tr, seed)
    kw = {}
    if seed % 3 == 1:
        kw["agg_kind"] = np.array([(c * 7 + seed) % 3 for c in range(20)], np.uint8)
    if seed % 7 == 2:
        kw["absent_mask"] = (1 << 5) | (1 << 17)
    print(f"case fused seed={seed} T={T} R={tr['r_start'].size} G={tr['n_ops'] + 1}", flush=True)
    want = O.attribute(tr, **kw)
    out, diag = _run(tr, **kw)
    parity.assert_attribute(out, want, diag)


@pytest.mark.parametrize("policy", [opattr.MISMATCH_PREFIX, opattr.MISMATCH_SKIP_NAME,
                                    opattr.MISMATCH_STRICT])
def test_fused_lstm_policies(policy):
    """The LSTM shape (5% of launches missing from the profiled list, 85% of
    kernel time outside every range) under the three count policies."""
    tr = tg.generate("lstm", emission="stream_major")
    want = O.attribute(tr, policy=policy)
    out, diag = _run(tr, policy=policy)
    parity.assert_attribute(out, want, diag)


def _regular_trace(T, run, n_ops, cycle, seed, with_ranges=True, NC=20):
    """One stream, launches 10 ns apart (5 ns long); each range covers `run`
    consecutive launches, the operators of consecutive ranges cycling over
    0 .. cycle-1; every launch has a profiled row in launch order."""
    rng = np.random.default_rng(seed)
    seq = np.arange(T, dtype=np.uint32)
    start = (np.arange(T, dtype=np.uint64) * 10).astype(np.uint64)
    dur = np.full(T, 5, dtype=np.uint32)
    name = (np.arange(T) % 7).astype(np.uint32)
    R = T // run if with_ranges else 0
    j = np.arange(R, dtype=np.uint64)
    r_start = (j * run * 10).astype(np.uint64)
    r_end = ((j * run + run - 1) * 10 + 5).astype(np.uint64)
    return dict(seq=seq, start_ns=start, dur_ns=dur, stream_id=np.zeros(T, np.uint16),
                name_id=name, part_id=None, pf_name=name.copy(),
                counters=rng.random((T, NC), dtype=np.float32), r_start=r_start, r_end=r_end,
                r_stream=np.zeros(R, np.uint16), r_op=(np.arange(R) % cycle).astype(np.uint32),
                part_rep=None, n_names=7, n_streams=1, n_ops=n_ops, n_parts=0)


def test_fused_combine_list_overflow():
    """More partial results for one bucket of operator rows in a combine
    wave's round than its LDS list holds: 64 operators of one bucket, each in
    every block, over more blocks than one round lists (the per-entry path)."""
    tr = _regular_trace(T=400_000, run=32, n_ops=16383, cycle=64, seed=91)
    print(f"case combine overflow T={tr['seq'].size} R={tr['r_start'].size}", flush=True)
    want = O.attribute(tr)
    out, diag = _run(tr)
    parity.assert_attribute(out, want, diag)


@pytest.mark.parametrize("with_ranges", [False, True])
def test_fused_unattributed(with_ranges):
    """No ranges at all (every launch in the unattributed row, which has a
    partial in every block and combine waves of its own), and ranges whose
    operator rows all fall in the unattributed row's bucket."""
    tr = _regular_trace(T=300_000, run=40, n_ops=3, cycle=3, seed=92, with_ranges=with_ranges)
    print(f"case unattributed ranges={with_ranges}", flush=True)
    want = O.attribute(tr)
    out, diag = _run(tr)
    parity.assert_attribute(out, want, diag)


def test_fused_dedup_errors():
    """Duplicates whose representative is shorter or has another name at a
    position, and a partition split in two: the same dedup errors, statuses
    and outputs as the oracle."""
    tr = cases.random_trace(4711, T=30_000, S=3, n_names=9, R=1_200, n_ops=40, t_max=90_000,
                            max_depth=4, dedup=True)
    tr, _, _ = cases.stream_major(tr)
    part = tr["part_id"].copy()
    names = tr["name_id"].copy()
    order = np.argsort(tr["seq"])
    ps = part[order]
    dup = np.flatnonzero(ps >= 0)
    # another name at some duplicate positions
    names[order[dup[5::97]]] = (names[order[dup[5::97]]] + 1) % tr["n_names"]
    t = dict(tr, name_id=names)
    want = O.attribute(t)
    out, diag = _run(t)
    assert want["diag"]["dedup_errors"] > 0
    parity.assert_attribute(out, want, diag)
    # a hole in one partition
    first = dup[0]
    ps2 = ps.copy()
    ps2[first + 1] = -1
    part2 = part.copy()
    part2[order] = ps2
    t2 = dict(tr, part_id=part2)
    want2 = O.attribute(t2)
    out2, diag2 = _run(t2)
    assert want2["diag"]["status"] == diag2["status"] != 0
    parity.assert_attribute(out2, want2, diag2)


def test_fused_graph_replay():
    """The fused path captured in a HIP graph (caller stream and both side
    streams) replays to the oracle's outputs, replay after replay, with the
    outputs poisoned and eager work in between."""
    import torch

    T = 60_000
    tr = cases.random_trace(808, T=T, S=4, n_names=31, R=T // 25, n_ops=300, t_max=4 * T,
                            max_depth=5, dedup=True)
    tr, _, _ = cases.stream_major(tr)
    want = O.attribute(tr)
    dt = opattr.to_device(tr, DEV)
    ws = opattr.Workspace(DEV)
    R = tr["r_start"].size
    o = opattr.Outputs(
        match=torch.empty(T, dtype=torch.int32, device=DEV),
        range_id=torch.empty(T, dtype=torch.int32, device=DEV),
        range_depth=torch.empty(R, dtype=torch.uint8, device=DEV),
        name_counts=torch.empty((tr["n_names"], 2), dtype=torch.int32, device=DEV),
        table=torch.empty((tr["n_ops"] + 1) * 192, dtype=torch.uint8, device=DEV),
        summary=torch.empty(40, dtype=torch.uint8, device=DEV))
    side = torch.cuda.Stream()
    with torch.cuda.stream(side):
        opattr.opattr_attribute(dt, flags=HINTS, ws=ws, outputs=o, raise_strict=False)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=side):
        opattr.opattr_attribute(dt, flags=HINTS, ws=ws, outputs=o, raise_strict=False)
    for rep in range(4):
        for k in ("match", "range_id", "table", "summary", "range_depth", "name_counts"):
            o[k].fill_(0x5A if o[k].dtype == torch.uint8 else -7)
        # eager work on the same workspace between replays
        opattr.opattr_attribute(dt, flags=HINTS, ws=ws, raise_strict=False)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        print(f"case fused graph replay {rep}", flush=True)
        parity.assert_attribute(o, want, opattr.read_diag(o["diag"]))
