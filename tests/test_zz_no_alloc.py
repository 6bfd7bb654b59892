"""opattr_attribute_noalloc (the entry point for callers that cannot
allocate device memory) against opattr_attribute on the same inputs: two
calls in a row on the library's scratch, the second with a smaller input
(the scratch then holds the first call's contents), one on the fused path
and one on the general path; a call that needs more than the scratch is
refused on the host."""
import numpy as np
import pytest

import cases
import parity
from paper_2609_11938_amd import opattr, tracegen as tg

pytestmark = pytest.mark.gpu

HINTS = opattr.KERNELS_STREAM_MAJOR | opattr.SEQ_DENSE | opattr.RANGES_NESTED
DEV = "cuda:0"


def _fused_trace():
    T = 240_000
    tr = cases.random_trace(77, T=T, S=5, n_names=40, R=T // 20, n_ops=900, t_max=4 * T,
                            max_depth=5, dedup=True)
    tr, _, _ = cases.stream_major(tr)
    return tr


def _both(tr, flags, **kw):
    import torch

    dt = opattr.to_device(tr, DEV)
    want = opattr.opattr_attribute(dt, flags=flags, raise_strict=False, **kw)
    torch.cuda.synchronize()
    got = opattr.opattr_attribute_noalloc(dt, flags=flags, raise_strict=False, **kw)
    torch.cuda.synchronize()
    return dt, got, want


def _same(got, want):
    for f in ("match", "range_id", "range_depth", "name_counts"):
        np.testing.assert_array_equal(parity.host(got[f]), parity.host(want[f]), err_msg=f)
    parity.assert_table(got.table_host(), want.table_host())
    gs, ws = got.summary_host(), want.summary_host()
    parity.assert_summary(gs, ws)
    gd, wd = opattr.read_diag(got["diag"]), opattr.read_diag(want["diag"])
    assert gd == wd, f"diag {gd} vs {wd}"


def test_noalloc_two_calls_second_smaller():
    import torch

    assert torch.cuda.is_available(), "GPU tests need a GPU"
    big = _fused_trace()
    small = tg.generate("gpt2")
    dt_big = opattr.to_device(big, DEV)
    dt_small = opattr.to_device(small, DEV)
    nb, ns = opattr.workspace_bytes(dt_big, HINTS), opattr.workspace_bytes(dt_small, 0)
    print(f"case noalloc fused T={big['seq'].size} ws={nb} then gpt2 T={small['seq'].size} "
          f"ws={ns}", flush=True)
    assert ns < nb <= opattr.NOALLOC_SCRATCH_BYTES
    kinds = np.array([(c * 5 + 1) % 3 for c in range(20)], np.uint8)
    _, got, want = _both(big, HINTS, agg_kind=kinds)
    _same(got, want)
    _, got, want = _both(small, 0)
    _same(got, want)


def test_noalloc_refuses_more_than_scratch():
    import torch

    tr = tg.generate("sdpa")
    dt = opattr.to_device(tr, DEV)
    need = opattr.workspace_bytes(dt, 0)
    print(f"case noalloc refuse T={tr['seq'].size} ws={need}", flush=True)
    assert need > opattr.NOALLOC_SCRATCH_BYTES
    with pytest.raises(RuntimeError, match=r"\(-11\)"):
        opattr.opattr_attribute_noalloc(dt)
    torch.cuda.synchronize()
