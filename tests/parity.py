"""Element-wise comparison of the HIP library's outputs with the oracle's.

Bar: bit-exact for every id, count and integer nanosecond sum; relative 1e-9
for the fp64 counter aggregates (NaN equals NaN; MAX compared by value).
"""
from __future__ import annotations

import numpy as np

RTOL = 1e-9
DIAG_FIELDS = ("status", "names_mismatched", "nesting_errors", "tl_unmatched", "pf_unmatched",
               "dedup_errors", "bad_records")
COMMON_FLAGS = 0x7F


_TRACES = {}


def trace(cfg, emission):
    """A generated trace, made once per process (the 10M-launch one takes a
    while) and shared by the GPU test modules."""
    from paper_2609_11938_amd import tracegen

    key = (cfg, emission)
    if key not in _TRACES:
        _TRACES[key] = tracegen.generate(cfg, emission=emission)
    return _TRACES[key]


def host(t):
    return None if t is None else t.cpu().numpy()


def assert_values_close(a, b, rtol=RTOL, what="value"):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    na, nb = np.isnan(a), np.isnan(b)
    assert np.array_equal(na, nb), f"{what}: NaN pattern differs at {np.argwhere(na != nb)[:5]}"
    ok = nb | (np.abs(a - b) <= rtol * np.maximum(np.abs(a), np.abs(b)))
    assert ok.all(), f"{what}: {np.argwhere(~ok)[:5].tolist()} {a[~ok][:5]} vs {b[~ok][:5]}"


def assert_table(got_rows, want_rows, rtol=RTOL):
    for f in ("kernel_count", "total_ns", "matched_count", "matched_ns"):
        assert np.array_equal(got_rows[f], want_rows[f]), f"table.{f} differs"
    assert_values_close(got_rows["value"], want_rows["value"], rtol, "table.value")


def assert_summary(got, want):
    for f in ("total_ns", "attributed_ns", "unattributed_ns", "matched_ns"):
        assert got[f] == int(want[f]), f"summary.{f}: {got[f]} vs {want[f]}"
    assert_values_close([got["attributed_fraction"]], [want["attributed_fraction"]], 1e-15,
                        "summary.attributed_fraction")


def assert_diag(got, want, fields=DIAG_FIELDS):
    for f in fields:
        assert got[f] == want[f], f"diag.{f}: {got[f]} vs {want[f]}"
    assert (got["flags"] & COMMON_FLAGS) == want["flags"], \
        f"diag.flags: {got['flags']:#x} vs {want['flags']:#x}"


def assert_attribute(out, want, diag, check_depth=True):
    """Full comparison of an opattr_attribute result with oracle.attribute."""
    np.testing.assert_array_equal(host(out["match"]), want["match"], err_msg="match")
    np.testing.assert_array_equal(host(out["range_id"]), want["range_id"], err_msg="range_id")
    if check_depth and out.get("range_depth") is not None:
        np.testing.assert_array_equal(host(out["range_depth"]), want["range_depth"],
                                      err_msg="range_depth")
    if out.get("name_counts") is not None:
        np.testing.assert_array_equal(host(out["name_counts"]).view(np.uint32),
                                      want["name_counts"], err_msg="name_counts")
    assert_table(out.table_host(), want["table"])
    assert_summary(out.summary_host(), want["summary"])
    assert_diag(diag, want["diag"])
