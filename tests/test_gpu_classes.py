"""Layer class discovery (Sec. 3.7) on the GPU against the oracle, through
the C ABI: random class traces (consecutive and broken partitions, bad ids,
seq with gaps or dense, storage shuffled or stream-major), key collisions
forced by narrowing the class key (the exact search must decide), the
generated GPT-2 and 10M-launch traces, edge cases, and the discovered classes
driving the dedup broadcast of a full attribution."""
import numpy as np
import pytest

import cases
import parity
from oracle import oracle as O
from paper_2609_11938_amd import opattr

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
HINTS = opattr.KERNELS_STREAM_MAJOR | opattr.SEQ_DENSE | opattr.RANGES_NESTED


@pytest.fixture(scope="module", autouse=True)
def _setup():
    import torch

    assert torch.cuda.is_available(), "GPU tests need a GPU"
    opattr.library()
    O.build(force=False)


def _classes(tr, flags=0, bits=64):
    import torch

    dt = opattr.to_device(tr, DEV)
    opattr.set_class_key_bits(bits)
    try:
        out = opattr.opattr_dedup_classes(dt, flags=flags)
        torch.cuda.synchronize()
    finally:
        opattr.set_class_key_bits(64)
    return parity.host(out["part_rep"]), opattr.read_diag(out["diag"])


def _check(tr, flags=0, bits=64):
    want = O.dedup_classes(tr)
    got, diag = _classes(tr, flags, bits)
    np.testing.assert_array_equal(got, want["part_rep"])
    for f in ("status", "flags", "bad_records"):
        assert diag[f] == want["diag"][f], (f, diag, want["diag"])
    return got


def _dense(tr):
    s = np.sort(tr["seq"])
    return bool(np.array_equal(s, np.arange(s.size)))


@pytest.mark.parametrize("seed", range(10))
def test_dedup_classes_parity(seed):
    """Random class traces: exact copies, near copies (one stream differs),
    a partition with a hole, a launch with a bad name; seq dense or with
    gaps; storage shuffled, then stream-major."""
    print(f"case classes seed={seed}", flush=True)
    tr = cases.class_trace(seed, T=400, n_parts=12, noncontig=seed % 3 == 1, bad=seed % 4 == 3)
    _check(tr)
    if _dense(tr):
        _check(tr, flags=opattr.SEQ_DENSE)
        _check(tr, flags=opattr.SEQ_DENSE | opattr.VALIDATE)
    sm = cases.stream_major(tr)[0]
    _check(sm, flags=opattr.SEQ_DENSE if _dense(sm) else 0)


@pytest.mark.parametrize("bits", [1, 3, 12])
def test_dedup_classes_exact_under_key_collisions(bits):
    """With the class key cut to a few bits, partitions of different
    sequences (and lengths) share keys: the count check and the element-wise
    comparison reject the candidate and the exact search finds the lowest
    partition of the same sequence."""
    for seed in range(4):
        print(f"case classes collisions bits={bits} seed={seed}", flush=True)
        tr = cases.class_trace(100 + seed, T=3000, n_parts=60, noncontig=seed == 1, bad=seed == 2)
        _check(tr, bits=bits)


@pytest.mark.parametrize("n_parts", [20, 5000])
def test_dedup_classes_many_tiles(n_parts):
    """300k launches: partitions of ~15k launches (whole waves in one
    partition) or of 59 (waves across partition edges), in shuffled and
    stream-major storage, full and 10-bit keys."""
    print(f"case classes 300k n_parts={n_parts}", flush=True)
    tr = cases.class_trace(7, T=300_000, n_parts=n_parts, S=4, n_names=6, seq_gaps=False)
    _check(tr)
    sm = cases.stream_major(tr)[0]
    _check(sm, flags=opattr.SEQ_DENSE)
    _check(sm, flags=opattr.SEQ_DENSE, bits=10)


@pytest.mark.parametrize("cfg,emission", [("gpt2", "shuffled"), ("gpt2", "stream_major"),
                                          ("large", "stream_major")])
def test_dedup_classes_generated_traces(cfg, emission):
    """The generated traces copy one template per class into every layer:
    discovery recovers one class for GPT-2, three for the 10M-launch trace."""
    print(f"case classes {cfg}/{emission}", flush=True)
    tr = parity.trace(cfg, emission)
    got = _check(tr, flags=0 if emission == "shuffled" else opattr.SEQ_DENSE)
    assert np.unique(got).size == (1 if cfg == "gpt2" else 3)


def test_dedup_classes_duplicate_seq_and_edges():
    """Equal seq values (general path): ORDER, ranks tie by index. No
    launches: every partition empty, one class. No partitions: nothing to
    write. Every launch with a bad name: all partitions empty."""
    print("case classes edges", flush=True)
    tr = cases.class_trace(11, T=200, n_parts=8)
    tr["seq"] = tr["seq"].copy()
    tr["seq"][5] = tr["seq"][9]
    _check(tr)
    empty = dict(tr)
    for f in ("seq", "start_ns", "dur_ns", "stream_id", "name_id", "part_id"):
        empty[f] = tr[f][:0]
    np.testing.assert_array_equal(_check(empty), np.zeros(8, np.int32))
    _check(empty, flags=opattr.SEQ_DENSE)
    none = dict(tr, n_parts=0)
    none["part_id"] = np.full(tr["seq"].size, -1, np.int32)
    assert _check(none).size == 0
    bad = dict(tr)
    bad["name_id"] = np.full(tr["seq"].size, tr["n_names"] + 3, np.uint32)
    _check(bad)


def test_discovered_classes_drive_the_dedup():
    """Classes found on the GPU, handed to the full attribution as the class
    map: the same matches and table as the oracle given that map."""
    print("case classes -> attribute", flush=True)
    tr = parity.trace("gpt2", "stream_major")
    rep, _ = _classes(tr, flags=opattr.SEQ_DENSE)
    tr = dict(tr, part_rep=rep)
    want = O.attribute(tr)
    dt = opattr.to_device(tr, DEV)
    out = opattr.opattr_attribute(dt, flags=HINTS, raise_strict=False)
    parity.assert_attribute(out, want, opattr.read_diag(out["diag"]))
