"""Python binding of libopattr (the MI355X attribution join).

Argument marshalling only: device tensors are handed to the C ABI declared in
``include/opattr.h`` by pointer, every stage runs in the library's HIP kernels,
and results come back as device tensors. PyTorch supplies device memory and the
current HIP stream. There is no CPU fallback: a missing library raises.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "_build", "libopattr.so")

NUM_COUNTERS = 20
MISMATCH_PREFIX, MISMATCH_SKIP_NAME, MISMATCH_STRICT = 0, 1, 2
AGG_SUM, AGG_DWMEAN, AGG_MAX = 0, 1, 2
KERNELS_STREAM_MAJOR, SEQ_DENSE, RANGES_NESTED, VALIDATE = 1, 2, 4, 8
F_DATA, F_ORDER, F_LIMIT, F_NOT_NESTED, F_PARTITION, F_DEDUP, F_COUNT = 1, 2, 4, 8, 16, 32, 64


class InvocationCountMismatchError(RuntimeError):
    """Per-name launch and profiled-row counts differ under the strict policy."""


class opattr_kernels(C.Structure):
    _fields_ = [("n", C.c_int64), ("seq", C.c_void_p), ("start_ns", C.c_void_p),
                ("dur_ns", C.c_void_p), ("stream_id", C.c_void_p), ("name_id", C.c_void_p),
                ("part_id", C.c_void_p), ("query_ns", C.c_void_p)]


class opattr_profiled(C.Structure):
    _fields_ = [("n", C.c_int64), ("name_id", C.c_void_p), ("counters", C.c_void_p),
                ("row_stride", C.c_int64), ("col_stride", C.c_int64),
                ("absent_mask", C.c_uint32)]


class opattr_ranges(C.Structure):
    _fields_ = [("n", C.c_int64), ("start_ns", C.c_void_p), ("end_ns", C.c_void_p),
                ("stream_id", C.c_void_p), ("op_id", C.c_void_p), ("kind", C.c_void_p)]


# range kinds of the enclosure walk (Alg. 2)
KIND_OP, KIND_BOUNDARY, KIND_SKIP = 0, 1, 2


class opattr_dims(C.Structure):
    _fields_ = [("n_names", C.c_uint32), ("n_streams", C.c_uint32), ("n_ops", C.c_uint32),
                ("n_parts", C.c_uint32), ("part_rep", C.c_void_p), ("flags", C.c_uint32)]


class opattr_corr_map(C.Structure):
    _fields_ = [("n", C.c_int64), ("name_id", C.c_void_p), ("op_id", C.c_void_p)]


class opattr_fusion_map(C.Structure):
    _fields_ = [("off", C.c_void_p), ("op_id", C.c_void_p)]


class opattr_coverage(C.Structure):
    _fields_ = [("count", C.c_uint64 * 4), ("ns", C.c_uint64 * 4), ("frac", C.c_double * 4)]


TIER_UNATTRIBUTED, TIER_HIGH, TIER_NVTX, TIER_FUSION = 0, 1, 2, 3


class opattr_diag(C.Structure):
    _fields_ = [("status", C.c_int32), ("flags", C.c_uint32), ("names_mismatched", C.c_uint32),
                ("nesting_errors", C.c_uint32), ("tl_unmatched", C.c_uint64),
                ("pf_unmatched", C.c_uint64), ("dedup_errors", C.c_uint64),
                ("bad_records", C.c_uint64), ("order_violations", C.c_uint64),
                ("strict", C.c_uint32), ("reserved", C.c_uint32)]


OP_ROW_DTYPE = np.dtype([("kernel_count", "<u8"), ("total_ns", "<u8"),
                         ("matched_count", "<u8"), ("matched_ns", "<u8"),
                         ("value", "<f8", (NUM_COUNTERS,))])
SUMMARY_DTYPE = np.dtype([("total_ns", "<u8"), ("attributed_ns", "<u8"),
                          ("unattributed_ns", "<u8"), ("matched_ns", "<u8"),
                          ("attributed_fraction", "<f8")])
assert OP_ROW_DTYPE.itemsize == 192 and SUMMARY_DTYPE.itemsize == 40
assert C.sizeof(opattr_diag) == 64

EXPORTS = ("opattr_workspace_bytes", "opattr_diag_clear", "opattr_read_diag", "opattr_match",
           "opattr_dedup_broadcast", "opattr_dedup_classes", "opattr_tiers_workspace_bytes",
           "opattr_tiers", "opattr_aggregate_ops", "opattr_dispatch_workspace_bytes",
           "opattr_aggregate_dispatch", "opattr_enclose_all",
           "opattr_attribute_tiered_workspace_bytes", "opattr_attribute_tiered", "opattr_enclose",
           "opattr_enclose_walk", "opattr_aggregate", "opattr_attribute",
           "opattr_attribute_noalloc", "opattr_set_probe_events", "opattr_set_class_key_bits",
           "opattr_strerror")
PROBES = ("seq_view", "tl_hist", "pf_hist", "col_scan", "pf_slot", "tl_match", "dedup",
          "ranges", "main_pass", "finalize", "aggregate", "agg_runs", "item_sort")

_lib = None


def library(path: str | None = None):
    """Load libopattr.so (or the library at ``path``) and declare its entry
    points. Raises when it is not built: this package has no CPU fallback."""
    global _lib
    if path is None:
        path = LIB_PATH
    if _lib is not None and path == LIB_PATH:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"libopattr is not built ({path}); run __graft_entry__.build()")
    L = C.CDLL(path)
    P = C.POINTER
    vp, i, sz = C.c_void_p, C.c_int, C.c_size_t
    L.opattr_workspace_bytes.argtypes = [P(opattr_kernels), P(opattr_profiled),
                                         P(opattr_ranges), P(opattr_dims)]
    L.opattr_workspace_bytes.restype = sz
    L.opattr_diag_clear.argtypes = [vp, vp]
    L.opattr_read_diag.argtypes = [vp, P(opattr_diag), vp]
    L.opattr_match.argtypes = [P(opattr_kernels), P(opattr_profiled), P(opattr_dims), i, vp, vp,
                               vp, vp, sz, vp]
    L.opattr_dedup_broadcast.argtypes = [P(opattr_kernels), P(opattr_dims), vp,
                                         P(opattr_profiled), vp, vp, vp, sz, vp]
    L.opattr_dedup_classes.argtypes = [P(opattr_kernels), P(opattr_dims), vp, vp, vp, sz, vp]
    L.opattr_enclose.argtypes = [P(opattr_kernels), P(opattr_ranges), P(opattr_dims), vp, vp,
                                 vp, vp, sz, vp]
    L.opattr_enclose_walk.argtypes = [P(opattr_kernels), P(opattr_ranges), P(opattr_dims), vp,
                                      vp, vp, vp, vp, vp, vp, sz, vp]
    L.opattr_aggregate.argtypes = [P(opattr_kernels), P(opattr_profiled), vp, vp,
                                   P(opattr_ranges), P(opattr_dims), vp, vp, vp, vp, vp, sz, vp]
    L.opattr_attribute.argtypes = [P(opattr_kernels), P(opattr_profiled), P(opattr_ranges),
                                   P(opattr_dims), i, vp, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]
    L.opattr_attribute_noalloc.argtypes = [P(opattr_kernels), P(opattr_profiled),
                                           P(opattr_ranges), P(opattr_dims), i, vp, vp, vp, vp,
                                           vp, vp, vp, vp, vp]
    for f in ("opattr_diag_clear", "opattr_read_diag", "opattr_match", "opattr_dedup_broadcast",
              "opattr_enclose", "opattr_enclose_walk", "opattr_aggregate", "opattr_attribute",
              "opattr_attribute_noalloc"):
        getattr(L, f).restype = C.c_int
    L.opattr_tiers_workspace_bytes.argtypes = [P(opattr_kernels), P(opattr_corr_map),
                                               P(opattr_ranges), P(opattr_dims)]
    L.opattr_tiers_workspace_bytes.restype = sz
    L.opattr_tiers.argtypes = [P(opattr_kernels), P(opattr_corr_map), P(opattr_fusion_map),
                               P(opattr_ranges), P(opattr_dims), i, vp, vp, vp, vp, vp, vp, vp,
                               vp, sz, vp]
    L.opattr_tiers.restype = C.c_int
    L.opattr_aggregate_ops.argtypes = [P(opattr_kernels), P(opattr_profiled), vp, vp,
                                       P(opattr_dims), vp, vp, vp, vp, vp, sz, vp]
    L.opattr_aggregate_ops.restype = C.c_int
    L.opattr_dispatch_workspace_bytes.argtypes = [P(opattr_kernels), P(opattr_profiled),
                                                  P(opattr_ranges), P(opattr_dims)]
    L.opattr_dispatch_workspace_bytes.restype = sz
    L.opattr_aggregate_dispatch.argtypes = [P(opattr_kernels), P(opattr_profiled), vp, vp, vp,
                                            P(opattr_ranges), P(opattr_dims), vp, vp, vp, vp, vp,
                                            vp, sz, vp]
    L.opattr_aggregate_dispatch.restype = C.c_int
    L.opattr_enclose_all.argtypes = [P(opattr_kernels), P(opattr_ranges), P(opattr_dims), vp, vp,
                                     C.c_int64, vp, vp, sz, vp]
    L.opattr_enclose_all.restype = C.c_int
    L.opattr_attribute_tiered_workspace_bytes.argtypes = [P(opattr_kernels), P(opattr_profiled),
                                                          P(opattr_ranges), P(opattr_corr_map),
                                                          P(opattr_dims)]
    L.opattr_attribute_tiered_workspace_bytes.restype = sz
    L.opattr_attribute_tiered.argtypes = [P(opattr_kernels), P(opattr_profiled), P(opattr_ranges),
                                          P(opattr_corr_map), P(opattr_fusion_map), P(opattr_dims),
                                          i, i, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]
    L.opattr_attribute_tiered.restype = C.c_int
    L.opattr_set_class_key_bits.argtypes = [i]
    L.opattr_set_class_key_bits.restype = C.c_int
    L.opattr_set_probe_events.argtypes = [vp, i]
    L.opattr_set_probe_events.restype = C.c_int
    L.opattr_strerror.argtypes = [i]
    L.opattr_strerror.restype = C.c_char_p
    if path == LIB_PATH:
        _lib = L
    return L


def set_probe_events(events) -> None:
    """events: None, or a list of 2*n torch.cuda.Event (timing enabled, already
    recorded once so that the HIP event exists), start/stop per probe in the
    order of PROBES; a None entry leaves that event unrecorded."""
    L = library()
    if not events:
        _check(L.opattr_set_probe_events(None, 0), "opattr_set_probe_events")
        return
    arr = (C.c_void_p * len(events))(*[e.cuda_event if e is not None else None
                                       for e in events])
    _check(L.opattr_set_probe_events(arr, len(events) // 2), "opattr_set_probe_events")


def strerror(status: int) -> str:
    return library().opattr_strerror(status).decode()


# --------------------------------------------------------------------------- #
# device trace                                                                #
# --------------------------------------------------------------------------- #

_KERNEL_FIELDS = {"seq": np.uint32, "start_ns": np.uint64, "dur_ns": np.uint32,
                  "stream_id": np.uint16, "name_id": np.uint32, "part_id": np.int32,
                  "query_ns": np.uint64}
_MAP_FIELDS = {"corr_name": np.uint32, "corr_op": np.int32, "fmap_off": np.uint32,
               "fmap_op": np.int32}
_RANGE_FIELDS = {"r_start": np.uint64, "r_end": np.uint64, "r_stream": np.uint16,
                 "r_op": np.uint32, "r_kind": np.uint8}


def to_device(tr: dict, device="cuda:0") -> dict:
    """Copy a host trace (dict of numpy arrays, see tracegen.generate) to device
    tensors. Dimension entries are kept as Python ints."""
    import torch

    out = {}
    for k, dt in {**_KERNEL_FIELDS, **_RANGE_FIELDS, **_MAP_FIELDS, "pf_name": np.uint32,
                  "part_rep": np.int32}.items():
        a = tr.get(k)
        out[k] = None if a is None else torch.from_numpy(
            np.ascontiguousarray(a, dtype=dt)).to(device)
    cnt = tr["counters"]
    if cnt.dtype != np.float32 or cnt.ndim != 2:
        raise TypeError("counters must be a 2-D float32 array")
    out["counters"] = torch.from_numpy(np.ascontiguousarray(cnt)).to(device)
    for k in ("n_names", "n_streams", "n_ops", "n_parts"):
        out[k] = int(tr.get(k, 0) or 0)
    return out


def _p(t):
    return None if t is None else C.c_void_p(t.data_ptr())


class _Marshal:
    """ctypes structs pointing at a device trace's tensors."""

    def __init__(self, dt: dict, flags: int, absent_mask: int = 0):
        T = 0 if dt["seq"] is None else int(dt["seq"].numel())
        self.k = opattr_kernels(T, _p(dt["seq"]), _p(dt["start_ns"]), _p(dt["dur_ns"]),
                                _p(dt["stream_id"]), _p(dt["name_id"]), _p(dt.get("part_id")),
                                _p(dt.get("query_ns")))
        cnt = dt["counters"]
        P = int(dt["pf_name"].numel())
        rs, cs = (cnt.stride(0), cnt.stride(1)) if cnt.dim() == 2 else (NUM_COUNTERS, 1)
        self.p = opattr_profiled(P, _p(dt["pf_name"]), _p(cnt) if P else None, rs, cs,
                                 absent_mask)
        R = int(dt["r_start"].numel())
        self.r = opattr_ranges(R, _p(dt["r_start"]), _p(dt["r_end"]), _p(dt["r_stream"]),
                               _p(dt["r_op"]), _p(dt.get("r_kind")))
        rep = dt.get("part_rep")
        self.d = opattr_dims(dt["n_names"], dt["n_streams"], dt["n_ops"],
                             dt.get("n_parts", 0) if rep is not None else 0, _p(rep), flags)
        self.T, self.P, self.R = T, P, R


class Workspace:
    """Device scratch reused across calls (grown on demand)."""

    def __init__(self, device="cuda:0"):
        self.device = device
        self.buf = None

    def get(self, nbytes: int):
        import torch

        if self.buf is None or self.buf.numel() < nbytes:
            self.buf = torch.empty(max(nbytes, 1), dtype=torch.uint8, device=self.device)
        return self.buf


def _stream_handle(stream):
    import torch

    s = torch.cuda.current_stream() if stream is None else stream
    return C.c_void_p(s.cuda_stream)


def _check(rc: int, fn: str):
    if rc != 0:
        raise RuntimeError(f"{fn}: {strerror(rc)} ({rc})")


def read_diag(diag_dev, stream=None) -> dict:
    L = library()
    h = opattr_diag()
    _check(L.opattr_read_diag(_p(diag_dev), C.byref(h), _stream_handle(stream)),
           "opattr_read_diag")
    return {f: int(getattr(h, f)) for f, _ in opattr_diag._fields_}


def _new_diag(device, stream):
    import torch

    d = torch.empty(C.sizeof(opattr_diag), dtype=torch.uint8, device=device)
    _check(library().opattr_diag_clear(_p(d), _stream_handle(stream)), "opattr_diag_clear")
    return d


def workspace_bytes(dt: dict, flags: int = 0) -> int:
    m = _Marshal(dt, flags)
    return int(library().opattr_workspace_bytes(C.byref(m.k), C.byref(m.p), C.byref(m.r),
                                                C.byref(m.d)))


def _kinds(agg_kind):
    if agg_kind is None:
        return None, None
    k = np.ascontiguousarray(agg_kind, dtype=np.uint8)
    if k.size != NUM_COUNTERS:
        raise ValueError("agg_kind needs 20 entries")
    return k, C.c_void_p(k.ctypes.data)


class Outputs(dict):
    """Device outputs of a call plus host copies made on demand."""

    def table_host(self):
        return self["table"].cpu().numpy().view(OP_ROW_DTYPE).reshape(-1)

    def coverage_host(self):
        c = opattr_coverage.from_buffer_copy(self["coverage"].cpu().numpy().tobytes())
        return {"count": np.array(c.count[:], dtype=np.uint64),
                "ns": np.array(c.ns[:], dtype=np.uint64),
                "frac": np.array(c.frac[:], dtype=np.float64)}

    def summary_host(self):
        a = self["summary"].cpu().numpy().view(SUMMARY_DTYPE)[0]
        return {f: (float(a[f]) if f == "attributed_fraction" else int(a[f]))
                for f in SUMMARY_DTYPE.names}


def _attribute_outputs(dt: dict, m: _Marshal, want_depth: bool, want_name_counts: bool):
    import torch

    dev = dt["counters"].device
    return Outputs(
        match=torch.empty(m.T, dtype=torch.int32, device=dev),
        range_id=torch.empty(m.T, dtype=torch.int32, device=dev),
        range_depth=torch.empty(m.R, dtype=torch.uint8, device=dev) if want_depth else None,
        name_counts=torch.empty((dt["n_names"], 2), dtype=torch.int32, device=dev)
        if want_name_counts else None,
        table=torch.empty((dt["n_ops"] + 1) * 192, dtype=torch.uint8, device=dev),
        summary=torch.empty(40, dtype=torch.uint8, device=dev),
    )


def _raise_strict(outputs: Outputs, stream):
    d = read_diag(outputs["diag"], stream)
    if d["status"] == -4:
        raise InvocationCountMismatchError(
            f"{d['names_mismatched']} kernel names have different launch and profiled counts")


def opattr_attribute(dt: dict, policy=MISMATCH_PREFIX, agg_kind=None, flags=0, absent_mask=0,
                     want_depth=True, want_name_counts=True, ws: Workspace | None = None,
                     stream=None, outputs: Outputs | None = None, raise_strict=True) -> Outputs:
    """All four stages in one call (see opattr_attribute in include/opattr.h)."""
    L = library()
    m = _Marshal(dt, flags, absent_mask)
    dev = dt["counters"].device
    if outputs is None:
        outputs = _attribute_outputs(dt, m, want_depth, want_name_counts)
    outputs["diag"] = _new_diag(dev, stream)
    ws = ws or Workspace(dev)
    need = L.opattr_workspace_bytes(C.byref(m.k), C.byref(m.p), C.byref(m.r), C.byref(m.d))
    buf = ws.get(need)
    _, kp = _kinds(agg_kind)
    k_keep = _kinds(agg_kind)[0]
    rc = L.opattr_attribute(C.byref(m.k), C.byref(m.p), C.byref(m.r), C.byref(m.d), policy, kp,
                            _p(outputs["match"]), _p(outputs["range_id"]),
                            _p(outputs["range_depth"]), _p(outputs["name_counts"]),
                            _p(outputs["table"]), _p(outputs["summary"]), _p(outputs["diag"]),
                            _p(buf), C.c_size_t(buf.numel()), _stream_handle(stream))
    del k_keep
    _check(rc, "opattr_attribute")
    if raise_strict and policy == MISMATCH_STRICT:
        _raise_strict(outputs, stream)
    return outputs


NOALLOC_SCRATCH_BYTES = 64 << 20


def opattr_attribute_noalloc(dt: dict, policy=MISMATCH_PREFIX, agg_kind=None, flags=0,
                             absent_mask=0, want_depth=True, want_name_counts=True, stream=None,
                             outputs: Outputs | None = None, raise_strict=True) -> Outputs:
    """opattr_attribute on the library's own scratch (see opattr_attribute_noalloc
    in include/opattr.h): the call itself allocates nothing; pass ``outputs``
    (from an earlier call) to allocate nothing here either."""
    L = library()
    m = _Marshal(dt, flags, absent_mask)
    dev = dt["counters"].device
    if outputs is None:
        outputs = _attribute_outputs(dt, m, want_depth, want_name_counts)
    if outputs.get("diag") is None:
        outputs["diag"] = _new_diag(dev, stream)
    else:
        _check(L.opattr_diag_clear(_p(outputs["diag"]), _stream_handle(stream)),
               "opattr_diag_clear")
    k_keep, kp = _kinds(agg_kind)
    rc = L.opattr_attribute_noalloc(C.byref(m.k), C.byref(m.p), C.byref(m.r), C.byref(m.d),
                                    policy, kp, _p(outputs["match"]), _p(outputs["range_id"]),
                                    _p(outputs["range_depth"]), _p(outputs["name_counts"]),
                                    _p(outputs["table"]), _p(outputs["summary"]),
                                    _p(outputs["diag"]), _stream_handle(stream))
    del k_keep
    _check(rc, "opattr_attribute_noalloc")
    if raise_strict and policy == MISMATCH_STRICT:
        _raise_strict(outputs, stream)
    return outputs


def opattr_match(dt: dict, policy=MISMATCH_PREFIX, flags=0, ws: Workspace | None = None,
                 stream=None) -> Outputs:
    import torch

    L = library()
    m = _Marshal(dt, flags)
    dev = dt["counters"].device
    out = Outputs(match=torch.empty(m.T, dtype=torch.int32, device=dev),
                  name_counts=torch.empty((dt["n_names"], 2), dtype=torch.int32, device=dev),
                  diag=_new_diag(dev, stream))
    ws = ws or Workspace(dev)
    buf = ws.get(L.opattr_workspace_bytes(C.byref(m.k), C.byref(m.p), C.byref(m.r), C.byref(m.d)))
    _check(L.opattr_match(C.byref(m.k), C.byref(m.p), C.byref(m.d), policy, _p(out["match"]),
                          _p(out["name_counts"]), _p(out["diag"]), _p(buf),
                          C.c_size_t(buf.numel()), _stream_handle(stream)), "opattr_match")
    return out


def opattr_dedup_broadcast(dt: dict, match, flags=0, ws: Workspace | None = None,
                           stream=None, counters_out=None, absent_mask=0) -> Outputs:
    """Dedup broadcast of ``match`` in place; with ``counters_out`` (True for a
    new [T, 20] float32 tensor, or such a tensor) also every launch's
    inherited counter row."""
    import torch

    L = library()
    m = _Marshal(dt, flags, absent_mask)
    dev = dt["counters"].device
    if counters_out is True:
        counters_out = torch.empty((m.T, NUM_COUNTERS), dtype=torch.float32, device=dev)
    if counters_out is not None and (counters_out.shape != (m.T, NUM_COUNTERS)
                                     or counters_out.dtype != torch.float32
                                     or not counters_out.is_contiguous()):
        raise ValueError("counters_out must be a contiguous [T, 20] float32 tensor")
    out = Outputs(match=match, diag=_new_diag(dev, stream), counters_out=counters_out)
    ws = ws or Workspace(dev)
    buf = ws.get(L.opattr_workspace_bytes(C.byref(m.k), None, None, C.byref(m.d)))
    _check(L.opattr_dedup_broadcast(C.byref(m.k), C.byref(m.d), _p(match),
                                    C.byref(m.p) if counters_out is not None else None,
                                    _p(counters_out), _p(out["diag"]), _p(buf),
                                    C.c_size_t(buf.numel()), _stream_handle(stream)),
           "opattr_dedup_broadcast")
    return out


def opattr_dedup_classes(dt: dict, flags=0, ws: Workspace | None = None,
                         stream=None) -> Outputs:
    """Layer class discovery (Sec. 3.7): part_rep for ``dt["n_parts"]``
    partitions from the launches' (name, stream) sequences; ``dt["part_rep"]``
    is not read."""
    import torch

    L = library()
    m = _Marshal(dt, flags)
    NP = int(dt.get("n_parts", 0) or 0)
    m.d.n_parts = NP
    m.d.part_rep = None
    dev = dt["seq"].device
    out = Outputs(part_rep=torch.empty(NP, dtype=torch.int32, device=dev),
                  diag=_new_diag(dev, stream))
    ws = ws or Workspace(dev)
    buf = ws.get(L.opattr_workspace_bytes(C.byref(m.k), None, None, C.byref(m.d)))
    _check(L.opattr_dedup_classes(C.byref(m.k), C.byref(m.d), _p(out["part_rep"]),
                                  _p(out["diag"]), _p(buf), C.c_size_t(buf.numel()),
                                  _stream_handle(stream)), "opattr_dedup_classes")
    return out


def _maps(dt: dict):
    """ctypes views of a device trace's correlation and fusion maps (None
    when absent); keeps a placeholder for an empty fusion list alive."""
    import torch

    corr = fm = None
    keep = []
    if dt.get("corr_name") is not None:
        corr = opattr_corr_map(int(dt["corr_name"].numel()), _p(dt["corr_name"]),
                               _p(dt["corr_op"]))
    if dt.get("fmap_off") is not None:
        fop = dt["fmap_op"]
        if fop.numel() == 0:
            fop = torch.zeros(1, dtype=torch.int32, device=dt["fmap_off"].device)
            keep.append(fop)
        fm = opattr_fusion_map(_p(dt["fmap_off"]), _p(fop))
    return corr, fm, keep


def opattr_tiers(dt: dict, range_id, walk_fused=None, corr_policy=MISMATCH_SKIP_NAME, flags=0,
                 ws: Workspace | None = None, stream=None) -> Outputs:
    """Tiered attribution (see opattr_tiers in include/opattr.h): tier, op
    and fused per launch, and the coverage record, from the enclosure walk's
    range_id / fused and the maps in ``dt`` (corr_name/corr_op,
    fmap_off/fmap_op)."""
    import torch

    L = library()
    m = _Marshal(dt, flags)
    corr, fm, keep = _maps(dt)
    dev = dt["seq"].device
    out = Outputs(tier=torch.empty(m.T, dtype=torch.uint8, device=dev),
                  op=torch.empty(m.T, dtype=torch.int32, device=dev),
                  fused=torch.empty(m.T, dtype=torch.uint8, device=dev),
                  coverage=torch.empty(C.sizeof(opattr_coverage), dtype=torch.uint8, device=dev),
                  diag=_new_diag(dev, stream))
    cp = C.byref(corr) if corr is not None else None
    fp = C.byref(fm) if fm is not None else None
    ws = ws or Workspace(dev)
    buf = ws.get(L.opattr_tiers_workspace_bytes(C.byref(m.k), cp, C.byref(m.r), C.byref(m.d)))
    rc = L.opattr_tiers(C.byref(m.k), cp, fp, C.byref(m.r), C.byref(m.d), corr_policy,
                        _p(range_id), _p(walk_fused), _p(out["tier"]), _p(out["op"]),
                        _p(out["fused"]), _p(out["coverage"]), _p(out["diag"]), _p(buf),
                        C.c_size_t(buf.numel()), _stream_handle(stream))
    del keep
    _check(rc, "opattr_tiers")
    return out


def opattr_aggregate_ops(dt: dict, match, op, agg_kind=None, flags=0, absent_mask=0,
                         ws: Workspace | None = None, stream=None) -> Outputs:
    """Eq. 1 by a given operator per launch (see opattr_aggregate_ops)."""
    import torch

    L = library()
    m = _Marshal(dt, flags, absent_mask)
    dev = dt["counters"].device
    out = Outputs(table=torch.empty((dt["n_ops"] + 1) * 192, dtype=torch.uint8, device=dev),
                  summary=torch.empty(40, dtype=torch.uint8, device=dev),
                  diag=_new_diag(dev, stream))
    ws = ws or Workspace(dev)
    buf = ws.get(L.opattr_workspace_bytes(C.byref(m.k), C.byref(m.p), None, C.byref(m.d)))
    k_keep, kp = _kinds(agg_kind)
    rc = L.opattr_aggregate_ops(C.byref(m.k), C.byref(m.p), _p(match), _p(op), C.byref(m.d), kp,
                                _p(out["table"]), _p(out["summary"]), _p(out["diag"]), _p(buf),
                                C.c_size_t(buf.numel()), _stream_handle(stream))
    del k_keep
    _check(rc, "opattr_aggregate_ops")
    return out


def opattr_aggregate_dispatch(dt: dict, match, range_id, op=None, agg_kind=None, flags=0,
                              absent_mask=0, ws: Workspace | None = None,
                              stream=None) -> Outputs:
    """Eq. 1 per operator dispatch (see opattr_aggregate_dispatch): R range
    rows, then n_ops per-operator rows, then the unattributed row."""
    import torch

    L = library()
    m = _Marshal(dt, flags, absent_mask)
    dev = dt["counters"].device
    G = m.R + dt["n_ops"] + 1
    out = Outputs(table=torch.empty(G * 192, dtype=torch.uint8, device=dev),
                  summary=torch.empty(40, dtype=torch.uint8, device=dev),
                  row=torch.empty(m.T, dtype=torch.int32, device=dev),
                  diag=_new_diag(dev, stream))
    ws = ws or Workspace(dev)
    nbytes = L.opattr_dispatch_workspace_bytes(C.byref(m.k), C.byref(m.p), C.byref(m.r),
                                               C.byref(m.d))
    if nbytes == 0:
        raise RuntimeError("opattr_aggregate_dispatch: too many ranges and operators")
    buf = ws.get(nbytes)
    k_keep, kp = _kinds(agg_kind)
    rc = L.opattr_aggregate_dispatch(C.byref(m.k), C.byref(m.p), _p(match), _p(range_id), _p(op),
                                     C.byref(m.r), C.byref(m.d), kp, _p(out["table"]),
                                     _p(out["summary"]), _p(out["row"]), _p(out["diag"]), _p(buf),
                                     C.c_size_t(buf.numel()), _stream_handle(stream))
    del k_keep
    _check(rc, "opattr_aggregate_dispatch")
    return out


def opattr_attribute_tiered(dt: dict, policy=MISMATCH_PREFIX, corr_policy=MISMATCH_SKIP_NAME,
                            agg_kind=None, flags=0, absent_mask=0, ws: Workspace | None = None,
                            stream=None) -> Outputs:
    """Tiered attribution in one library call (see opattr_attribute_tiered):
    match, range_id, tier, op, fused per launch, the table by tier operator,
    the summary and the coverage record."""
    import torch

    L = library()
    m = _Marshal(dt, flags, absent_mask)
    corr, fm, keep = _maps(dt)
    dev = dt["counters"].device
    T = m.T
    out = Outputs(match=torch.empty(T, dtype=torch.int32, device=dev),
                  range_id=torch.empty(T, dtype=torch.int32, device=dev),
                  tier=torch.empty(T, dtype=torch.uint8, device=dev),
                  op=torch.empty(T, dtype=torch.int32, device=dev),
                  fused=torch.empty(T, dtype=torch.uint8, device=dev),
                  table=torch.empty((dt["n_ops"] + 1) * 192, dtype=torch.uint8, device=dev),
                  summary=torch.empty(40, dtype=torch.uint8, device=dev),
                  coverage=torch.empty(C.sizeof(opattr_coverage), dtype=torch.uint8, device=dev),
                  diag=_new_diag(dev, stream))
    cp = C.byref(corr) if corr is not None else None
    fp = C.byref(fm) if fm is not None else None
    ws = ws or Workspace(dev)
    buf = ws.get(L.opattr_attribute_tiered_workspace_bytes(C.byref(m.k), C.byref(m.p),
                                                           C.byref(m.r), cp, C.byref(m.d)))
    k_keep, kp = _kinds(agg_kind)
    rc = L.opattr_attribute_tiered(
        C.byref(m.k), C.byref(m.p), C.byref(m.r), cp, fp, C.byref(m.d), policy, corr_policy, kp,
        _p(out["match"]), _p(out["range_id"]), _p(out["tier"]), _p(out["op"]), _p(out["fused"]),
        _p(out["table"]), _p(out["summary"]), _p(out["coverage"]), _p(out["diag"]), _p(buf),
        C.c_size_t(buf.numel()), _stream_handle(stream))
    del k_keep, keep
    _check(rc, "opattr_attribute_tiered")
    return out


def attribute_tiered(dt: dict, policy=MISMATCH_PREFIX, corr_policy=MISMATCH_SKIP_NAME,
                     agg_kind=None, flags=0, dispatch=False, ws: Workspace | None = None,
                     stream=None) -> dict:
    """The tiered pipeline as a sequence of library calls on one stream:
    matching (with the dedup broadcast when a class map is given), the
    enclosure walk, the tiers, the operator table by tier operator and,
    with ``dispatch``, the per-dispatch table. Returns each call's
    outputs."""
    ws = ws or Workspace(dt["seq"].device)
    m = opattr_match(dt, policy=policy, flags=flags, ws=ws, stream=stream)
    res = {"match": m}
    if dt.get("part_rep") is not None and dt.get("part_id") is not None:
        res["dedup"] = opattr_dedup_broadcast(dt, m["match"], flags=flags, ws=ws, stream=stream)
    w = opattr_enclose_walk(dt, flags=flags, ws=ws, stream=stream)
    t = opattr_tiers(dt, w["range_id"], w["fused"], corr_policy=corr_policy, flags=flags, ws=ws,
                     stream=stream)
    a = opattr_aggregate_ops(dt, m["match"], t["op"], agg_kind=agg_kind, flags=flags, ws=ws,
                             stream=stream)
    res.update(walk=w, tiers=t, aggregate=a)
    if dispatch:
        res["dispatch"] = opattr_aggregate_dispatch(dt, m["match"], w["range_id"], t["op"],
                                                    agg_kind=agg_kind, flags=flags, ws=ws,
                                                    stream=stream)
    return res


def set_class_key_bits(bits: int = 64):
    """Test support: keep only ``bits`` bits of the class keys on this thread
    (see opattr_set_class_key_bits)."""
    _check(library().opattr_set_class_key_bits(int(bits)), "opattr_set_class_key_bits")


def opattr_enclose(dt: dict, flags=0, want_depth=True, ws: Workspace | None = None,
                   stream=None) -> Outputs:
    import torch

    L = library()
    m = _Marshal(dt, flags)
    dev = dt["counters"].device
    out = Outputs(range_id=torch.empty(m.T, dtype=torch.int32, device=dev),
                  range_depth=torch.empty(m.R, dtype=torch.uint8, device=dev)
                  if want_depth else None,
                  diag=_new_diag(dev, stream))
    ws = ws or Workspace(dev)
    buf = ws.get(L.opattr_workspace_bytes(C.byref(m.k), C.byref(m.p), C.byref(m.r), C.byref(m.d)))
    _check(L.opattr_enclose(C.byref(m.k), C.byref(m.r), C.byref(m.d), _p(out["range_id"]),
                            _p(out["range_depth"]), _p(out["diag"]), _p(buf),
                            C.c_size_t(buf.numel()), _stream_handle(stream)), "opattr_enclose")
    return out


def opattr_enclose_walk(dt: dict, flags=0, ws: Workspace | None = None, stream=None) -> Outputs:
    """The full enclosure walk of Alg. 2 (range kinds from ``dt["r_kind"]``):
    range_id, fused and range_any per launch; range_parent and range_depth
    per range."""
    import torch

    L = library()
    m = _Marshal(dt, flags)
    dev = dt["counters"].device
    out = Outputs(range_id=torch.empty(m.T, dtype=torch.int32, device=dev),
                  fused=torch.empty(m.T, dtype=torch.uint8, device=dev),
                  range_any=torch.empty(m.T, dtype=torch.int32, device=dev),
                  range_parent=torch.empty(m.R, dtype=torch.int32, device=dev),
                  range_depth=torch.empty(m.R, dtype=torch.uint8, device=dev),
                  diag=_new_diag(dev, stream))
    ws = ws or Workspace(dev)
    buf = ws.get(L.opattr_workspace_bytes(C.byref(m.k), C.byref(m.p), C.byref(m.r), C.byref(m.d)))
    _check(L.opattr_enclose_walk(C.byref(m.k), C.byref(m.r), C.byref(m.d), _p(out["range_id"]),
                                 _p(out["fused"]), _p(out["range_any"]), _p(out["range_parent"]),
                                 _p(out["range_depth"]), _p(out["diag"]), _p(buf),
                                 C.c_size_t(buf.numel()), _stream_handle(stream)),
           "opattr_enclose_walk")
    return out


def opattr_enclose_all(dt: dict, flags=0, ids=None, ws: Workspace | None = None,
                       stream=None) -> Outputs:
    """Every enclosing range of every launch as CSR lists (see
    opattr_enclose_all): one call for the offsets, one for the lists; with
    ``ids`` given (an int32 device tensor), one call filling it up to its
    size."""
    import torch

    L = library()
    m = _Marshal(dt, flags)
    dev = dt["counters"].device
    out = Outputs(off=torch.empty(m.T + 1, dtype=torch.int64, device=dev),
                  diag=_new_diag(dev, stream))
    ws = ws or Workspace(dev)
    buf = ws.get(L.opattr_workspace_bytes(C.byref(m.k), None, C.byref(m.r), C.byref(m.d)))

    def call(ids, cap):
        _check(L.opattr_enclose_all(C.byref(m.k), C.byref(m.r), C.byref(m.d), _p(out["off"]),
                                    _p(ids), C.c_int64(cap), _p(out["diag"]), _p(buf),
                                    C.c_size_t(buf.numel()), _stream_handle(stream)),
               "opattr_enclose_all")

    if ids is not None:
        out["ids"] = ids
        call(ids, int(ids.numel()))
        return out
    call(None, 0)
    total = int(out["off"][-1].item())
    out["ids"] = torch.empty(max(total, 1), dtype=torch.int32, device=dev)
    out["diag"] = _new_diag(dev, stream)
    call(out["ids"], total)
    out["ids"] = out["ids"][:total]
    return out


def opattr_aggregate(dt: dict, match, range_id, agg_kind=None, flags=0, absent_mask=0,
                     ws: Workspace | None = None, stream=None) -> Outputs:
    import torch

    L = library()
    m = _Marshal(dt, flags, absent_mask)
    dev = dt["counters"].device
    out = Outputs(table=torch.empty((dt["n_ops"] + 1) * 192, dtype=torch.uint8, device=dev),
                  summary=torch.empty(40, dtype=torch.uint8, device=dev),
                  diag=_new_diag(dev, stream))
    ws = ws or Workspace(dev)
    buf = ws.get(L.opattr_workspace_bytes(C.byref(m.k), C.byref(m.p), C.byref(m.r), C.byref(m.d)))
    k_keep, kp = _kinds(agg_kind)
    rc = L.opattr_aggregate(C.byref(m.k), C.byref(m.p), _p(match), _p(range_id), C.byref(m.r),
                            C.byref(m.d), kp, _p(out["table"]), _p(out["summary"]),
                            _p(out["diag"]), _p(buf), C.c_size_t(buf.numel()),
                            _stream_handle(stream))
    del k_keep
    _check(rc, "opattr_aggregate")
    return out
