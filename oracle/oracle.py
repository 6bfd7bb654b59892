"""Python wrapper of the C oracle (test infrastructure only).

Only the test-suite, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this module. It loads ``oracle/_build/liboracle.so``,
built from ``opattr_oracle.c`` by :func:`build` (plain gcc, one thread), and
shares nothing with the GPU library.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "opattr_oracle.c")
HDR = os.path.join(HERE, "opattr_oracle.h")
OUT_DIR = os.path.join(HERE, "_build")
LIB = os.path.join(OUT_DIR, "liboracle.so")

NC = 20
PREFIX, SKIP_NAME, STRICT = 0, 1, 2
SUM, DWMEAN, MAX = 0, 1, 2
# counter appendix table (rows 1..20): SUM for additive counts, duration-weighted
# mean for rates and utilisations, MAX for per-kernel constants
DEFAULT_KIND = np.array([SUM, SUM, SUM, DWMEAN, DWMEAN, DWMEAN, DWMEAN, DWMEAN, DWMEAN,
                         DWMEAN, SUM, DWMEAN, DWMEAN, DWMEAN, SUM, DWMEAN, DWMEAN, MAX,
                         SUM, MAX], dtype=np.uint8)

F_DATA, F_ORDER, F_LIMIT, F_NOT_NESTED, F_PARTITION, F_DEDUP, F_COUNT = (
    1, 2, 4, 8, 16, 32, 64)


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (single-threaded, no fast-math, no FMA
    contraction, so every product is rounded once)."""
    os.makedirs(OUT_DIR, exist_ok=True)
    if not force and os.path.exists(LIB) and \
            os.path.getmtime(LIB) >= max(os.path.getmtime(SRC), os.path.getmtime(HDR)):
        return LIB
    tmp = LIB + ".tmp"
    cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-ffp-contract=off",
           "-fno-fast-math", "-Wall", "-Wextra", "-o", tmp, SRC, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    return LIB


class Kernels(C.Structure):
    _fields_ = [("n", C.c_int64), ("seq", C.c_void_p), ("start_ns", C.c_void_p),
                ("dur_ns", C.c_void_p), ("stream_id", C.c_void_p),
                ("name_id", C.c_void_p), ("part_id", C.c_void_p),
                ("query_ns", C.c_void_p)]


class Profiled(C.Structure):
    _fields_ = [("n", C.c_int64), ("name_id", C.c_void_p), ("counters", C.c_void_p),
                ("row_stride", C.c_int64), ("col_stride", C.c_int64),
                ("absent_mask", C.c_uint32)]


class Ranges(C.Structure):
    _fields_ = [("n", C.c_int64), ("start_ns", C.c_void_p), ("end_ns", C.c_void_p),
                ("stream_id", C.c_void_p), ("op_id", C.c_void_p), ("kind", C.c_void_p)]


# range kinds of the enclosure walk (Alg. 2)
KIND_OP, KIND_BOUNDARY, KIND_SKIP = 0, 1, 2


class Dims(C.Structure):
    _fields_ = [("n_names", C.c_uint32), ("n_streams", C.c_uint32),
                ("n_ops", C.c_uint32), ("n_parts", C.c_uint32), ("part_rep", C.c_void_p)]


class Diag(C.Structure):
    _fields_ = [("status", C.c_int32), ("flags", C.c_uint32),
                ("names_mismatched", C.c_uint32), ("nesting_errors", C.c_uint32),
                ("tl_unmatched", C.c_uint64), ("pf_unmatched", C.c_uint64),
                ("dedup_errors", C.c_uint64), ("bad_records", C.c_uint64)]


class Summary(C.Structure):
    _fields_ = [("total_ns", C.c_uint64), ("attributed_ns", C.c_uint64),
                ("unattributed_ns", C.c_uint64), ("matched_ns", C.c_uint64),
                ("attributed_fraction", C.c_double)]


class Corr(C.Structure):
    _fields_ = [("n", C.c_int64), ("name_id", C.c_void_p), ("op_id", C.c_void_p)]


class Fusion(C.Structure):
    _fields_ = [("off", C.c_void_p), ("op_id", C.c_void_p)]


class Coverage(C.Structure):
    _fields_ = [("count", C.c_uint64 * 4), ("ns", C.c_uint64 * 4), ("frac", C.c_double * 4)]


# attribution tiers (Table "tiers")
TIER_UNATTRIBUTED, TIER_HIGH, TIER_NVTX, TIER_FUSION = 0, 1, 2, 3

ROW_DTYPE = np.dtype([("kernel_count", "<u8"), ("total_ns", "<u8"),
                      ("matched_count", "<u8"), ("matched_ns", "<u8"),
                      ("value", "<f8", (NC,))])

_lib = None


def load(path: str):
    """Load an oracle library built from opattr_oracle.c and declare its
    entry points."""
    L = C.CDLL(path)
    P = C.POINTER
    L.oref_match.argtypes = [P(Kernels), P(Profiled), P(Dims), C.c_int, C.c_void_p,
                             C.c_void_p, P(Diag)]
    L.oref_dedup.argtypes = [P(Kernels), P(Dims), C.c_void_p, P(Diag)]
    L.oref_counters_out.argtypes = [P(Profiled), C.c_void_p, C.c_int64, C.c_void_p]
    L.oref_enclose.argtypes = [P(Kernels), P(Ranges), P(Dims), C.c_void_p, C.c_void_p,
                               P(Diag)]
    L.oref_aggregate.argtypes = [P(Kernels), P(Profiled), C.c_void_p, C.c_void_p,
                                 P(Ranges), P(Dims), C.c_void_p, C.c_void_p,
                                 P(Summary), P(Diag)]
    L.oref_enclose_walk.argtypes = [P(Kernels), P(Ranges), P(Dims), C.c_void_p, C.c_void_p,
                                    C.c_void_p, C.c_void_p, C.c_void_p, P(Diag)]
    L.oref_dedup_classes.argtypes = [P(Kernels), P(Dims), C.c_void_p, P(Diag)]
    L.oref_aggregate_ops.argtypes = [P(Kernels), P(Profiled), C.c_void_p, C.c_void_p, P(Dims),
                                     C.c_void_p, C.c_void_p, P(Summary), P(Diag)]
    L.oref_enclose_all.argtypes = [P(Kernels), P(Ranges), P(Dims), C.c_void_p, C.c_void_p,
                                   C.c_int64, P(Diag)]
    L.oref_aggregate_dispatch.argtypes = [P(Kernels), P(Profiled), C.c_void_p, C.c_void_p,
                                          C.c_void_p, P(Ranges), P(Dims), C.c_void_p,
                                          C.c_void_p, P(Summary), P(Diag)]
    L.oref_tiers.argtypes = [P(Kernels), P(Corr), P(Fusion), P(Ranges), P(Dims), C.c_int,
                             C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p,
                             P(Coverage), P(Diag)]
    L.oref_diag_finish.argtypes = [P(Diag), C.c_int]
    for f in ("oref_match", "oref_dedup", "oref_counters_out", "oref_enclose", "oref_enclose_walk", "oref_aggregate",
              "oref_dedup_classes", "oref_aggregate_ops", "oref_tiers",
              "oref_aggregate_dispatch", "oref_enclose_all"):
        getattr(L, f).restype = C.c_int
    return L


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB):
            build()
        _lib = load(LIB)
    return _lib


def _ptr(a):
    return None if a is None else a.ctypes.data


def _c(a, dt):
    return None if a is None else np.ascontiguousarray(a, dtype=dt)


class _Inputs:
    """Contiguous, correctly typed views of a trace dict, kept alive with the
    ctypes structs that point into them."""

    def __init__(self, tr, absent_mask=0):
        self.seq = _c(tr["seq"], np.uint32)
        self.start = _c(tr["start_ns"], np.uint64)
        self.dur = _c(tr["dur_ns"], np.uint32)
        self.stream = _c(tr["stream_id"], np.uint16)
        self.name = _c(tr["name_id"], np.uint32)
        self.part = _c(tr.get("part_id"), np.int32)
        self.query = _c(tr.get("query_ns"), np.uint64)
        self.pf_name = _c(tr["pf_name"], np.uint32)
        cnt = tr["counters"]
        if cnt.dtype != np.float32:
            raise TypeError("counters must be float32")
        self.counters = cnt  # arbitrary strides honoured
        self.r_start = _c(tr["r_start"], np.uint64)
        self.r_end = _c(tr["r_end"], np.uint64)
        self.r_stream = _c(tr["r_stream"], np.uint16)
        self.r_op = _c(tr["r_op"], np.uint32)
        self.r_kind = _c(tr.get("r_kind"), np.uint8)
        self.part_rep = _c(tr.get("part_rep"), np.int32)
        T = self.seq.size
        self.k = Kernels(T, _ptr(self.seq), _ptr(self.start), _ptr(self.dur),
                         _ptr(self.stream), _ptr(self.name), _ptr(self.part),
                         _ptr(self.query))
        P = self.pf_name.size
        rs = cnt.strides[0] // 4 if cnt.ndim == 2 and P > 0 else NC
        cs = cnt.strides[1] // 4 if cnt.ndim == 2 and P > 0 else 1
        self.p = Profiled(P, _ptr(self.pf_name), cnt.ctypes.data if P > 0 else None,
                          rs, cs, absent_mask)
        self.r = Ranges(self.r_start.size, _ptr(self.r_start), _ptr(self.r_end),
                        _ptr(self.r_stream), _ptr(self.r_op), _ptr(self.r_kind))
        self.d = Dims(tr["n_names"], tr["n_streams"], tr["n_ops"],
                      tr.get("n_parts", 0) or 0, _ptr(self.part_rep))


def diag_dict(dg: Diag) -> dict:
    return {f: int(getattr(dg, f)) for f, _ in Diag._fields_}


def attribute(tr, policy=PREFIX, agg_kind=None, absent_mask=0, stages=None, library=None):
    """Run the oracle on a trace dict. ``stages`` (default all) is a subset of
    {"match", "dedup", "enclose", "aggregate"}; stages not run leave their
    outputs as provided in ``tr`` ("match", "range_id") or absent. ``library``
    replaces the default build (used to load deliberately broken copies)."""
    L = library if library is not None else lib()
    x = _Inputs(tr, absent_mask)
    stages = {"match", "dedup", "enclose", "aggregate"} if stages is None else set(stages)
    T = x.seq.size
    out = {}
    dg = Diag()
    if "match" in stages:
        match = np.empty(T, dtype=np.int32)
        nc = np.empty((tr["n_names"], 2), dtype=np.uint32)
        rc = L.oref_match(C.byref(x.k), C.byref(x.p), C.byref(x.d), policy,
                          _ptr(match), _ptr(nc), C.byref(dg))
        if rc:
            raise ValueError(f"oref_match: {rc}")
        out["match_iom"] = match.copy()
        out["name_counts"] = nc
    else:
        match = np.array(tr["match"], dtype=np.int32, copy=True)
    if "dedup" in stages:
        rc = L.oref_dedup(C.byref(x.k), C.byref(x.d), _ptr(match), C.byref(dg))
        if rc:
            raise ValueError(f"oref_dedup: {rc}")
    out["match"] = match
    if "enclose" in stages:
        rid = np.empty(T, dtype=np.int32)
        depth = np.empty(x.r_start.size, dtype=np.uint8)
        rc = L.oref_enclose(C.byref(x.k), C.byref(x.r), C.byref(x.d), _ptr(rid),
                            _ptr(depth), C.byref(dg))
        if rc:
            raise ValueError(f"oref_enclose: {rc}")
        out["range_id"] = rid
        out["range_depth"] = depth
    else:
        rid = np.array(tr["range_id"], dtype=np.int32, copy=True) if "range_id" in tr else None
    if "aggregate" in stages:
        rid_in = out.get("range_id", rid)
        table = np.zeros(tr["n_ops"] + 1, dtype=ROW_DTYPE)
        sm = Summary()
        kind = None if agg_kind is None else np.ascontiguousarray(agg_kind, dtype=np.uint8)
        rc = L.oref_aggregate(C.byref(x.k), C.byref(x.p), _ptr(match), _ptr(rid_in),
                              C.byref(x.r), C.byref(x.d), _ptr(kind), _ptr(table),
                              C.byref(sm), C.byref(dg))
        if rc:
            raise ValueError(f"oref_aggregate: {rc}")
        out["table"] = table
        out["summary"] = {f: getattr(sm, f) for f, _ in Summary._fields_}
    L.oref_diag_finish(C.byref(dg), policy)
    out["diag"] = diag_dict(dg)
    return out


def counters_out(tr, match, absent_mask=0, library=None):
    """Each launch's inherited counter row (Sec. 3.7): ``out[i, c]`` = counter c
    of profiled row ``match[i]``, NaN when unmatched or absent. ``tr`` gives
    the profiled rows (``counters``, ``pf_name``)."""
    L = library if library is not None else lib()
    x = _Inputs(tr, absent_mask)
    m = np.ascontiguousarray(match, dtype=np.int32)
    out = np.empty((m.size, NC), dtype=np.float32)
    rc = L.oref_counters_out(C.byref(x.p), _ptr(m), m.size, _ptr(out))
    if rc:
        raise ValueError(f"oref_counters_out: {rc}")
    return out


def enclose_walk(tr, library=None):
    """The full enclosure walk of Alg. 2 (range kinds from ``tr["r_kind"]``,
    absent = every range an attributed op): per kernel ``range_id`` (innermost
    attributed op before a structural boundary), ``fused`` and ``range_any``
    (innermost enclosing range of any kind); per range ``range_parent`` and
    ``range_depth``."""
    L = library if library is not None else lib()
    x = _Inputs(tr)
    T, R = x.seq.size, x.r_start.size
    dg = Diag()
    rid = np.empty(T, dtype=np.int32)
    fused = np.empty(T, dtype=np.uint8)
    rany = np.empty(T, dtype=np.int32)
    par = np.empty(R, dtype=np.int32)
    depth = np.empty(R, dtype=np.uint8)
    rc = L.oref_enclose_walk(C.byref(x.k), C.byref(x.r), C.byref(x.d), _ptr(rid), _ptr(fused),
                             _ptr(rany), _ptr(par), _ptr(depth), C.byref(dg))
    if rc:
        raise ValueError(f"oref_enclose_walk: {rc}")
    L.oref_diag_finish(C.byref(dg), PREFIX)
    return {"range_id": rid, "fused": fused, "range_any": rany, "range_parent": par,
            "range_depth": depth, "diag": diag_dict(dg)}


def dedup_classes(tr, library=None):
    """Dedup class discovery (Sec. 3.7): the class representative of every
    partition (``tr["part_id"]``, ``tr["n_parts"]``; ``tr["part_rep"]`` is not
    read) from the partitions' (name, stream) sequences in launch order."""
    L = library if library is not None else lib()
    tr = dict(tr)
    tr["part_rep"] = None
    x = _Inputs(tr)
    NP = int(tr.get("n_parts", 0) or 0)
    x.d.n_parts = NP
    dg = Diag()
    rep = np.empty(NP, dtype=np.int32)
    rc = L.oref_dedup_classes(C.byref(x.k), C.byref(x.d), _ptr(rep), C.byref(dg))
    if rc:
        raise ValueError(f"oref_dedup_classes: {rc}")
    L.oref_diag_finish(C.byref(dg), PREFIX)
    return {"part_rep": rep, "diag": diag_dict(dg)}


def _maps(tr):
    """ctypes views of the correlation map (corr_name, corr_op) and the
    fusion map (fmap_off, fmap_op) of a trace dict; absent maps give NULL."""
    keep = []
    corr = None
    if tr.get("corr_name") is not None:
        cn, co = _c(tr["corr_name"], np.uint32), _c(tr["corr_op"], np.int32)
        keep += [cn, co]
        corr = Corr(cn.size, _ptr(cn), _ptr(co))
    fm = None
    if tr.get("fmap_off") is not None:
        fo, fop = _c(tr["fmap_off"], np.uint32), _c(tr["fmap_op"], np.int32)
        if fop.size == 0:
            fop = np.zeros(1, np.int32)  # a valid pointer for an empty list
        keep += [fo, fop]
        fm = Fusion(_ptr(fo), _ptr(fop))
    return corr, fm, keep


def _coverage_dict(cv: Coverage) -> dict:
    return {"count": np.array(cv.count[:], dtype=np.uint64),
            "ns": np.array(cv.ns[:], dtype=np.uint64),
            "frac": np.array(cv.frac[:], dtype=np.float64)}


def tiers(tr, corr_policy=SKIP_NAME, library=None):
    """Tiered attribution (Table "tiers", decision-tree figure): the
    enclosure walk of Alg. 2, then per kernel the tier (HIGH from the
    correlation map, NVTX from the walk, FUSION from the fusion map,
    UNATTRIBUTED), its operator, the fused flag, and per-tier coverage."""
    L = library if library is not None else lib()
    walk = enclose_walk(tr, library=L)
    x = _Inputs(tr)
    T = x.seq.size
    corr, fm, keep = _maps(tr)
    tier = np.empty(T, dtype=np.uint8)
    op = np.empty(T, dtype=np.int32)
    fused = np.empty(T, dtype=np.uint8)
    cv = Coverage()
    dg = Diag()
    rc = L.oref_tiers(C.byref(x.k), C.byref(corr) if corr is not None else None,
                      C.byref(fm) if fm is not None else None, C.byref(x.r), C.byref(x.d),
                      corr_policy, _ptr(walk["range_id"]), _ptr(walk["fused"]), _ptr(tier),
                      _ptr(op), _ptr(fused), C.byref(cv), C.byref(dg))
    del keep
    if rc:
        raise ValueError(f"oref_tiers: {rc}")
    L.oref_diag_finish(C.byref(dg), corr_policy)
    return {"range_id": walk["range_id"], "walk_fused": walk["fused"], "tier": tier, "op": op,
            "fused": fused, "coverage": _coverage_dict(cv), "diag": diag_dict(dg)}


def aggregate_ops(tr, match, op, agg_kind=None, absent_mask=0, library=None):
    """Eq. 1 with the operator of every kernel given (``op``, -1 =
    UNATTRIBUTED)."""
    L = library if library is not None else lib()
    x = _Inputs(tr, absent_mask)
    match = np.ascontiguousarray(match, dtype=np.int32)
    op = np.ascontiguousarray(op, dtype=np.int32)
    table = np.zeros(tr["n_ops"] + 1, dtype=ROW_DTYPE)
    sm = Summary()
    dg = Diag()
    kind = None if agg_kind is None else np.ascontiguousarray(agg_kind, dtype=np.uint8)
    rc = L.oref_aggregate_ops(C.byref(x.k), C.byref(x.p), _ptr(match), _ptr(op), C.byref(x.d),
                              _ptr(kind), _ptr(table), C.byref(sm), C.byref(dg))
    if rc:
        raise ValueError(f"oref_aggregate_ops: {rc}")
    L.oref_diag_finish(C.byref(dg), PREFIX)
    return {"table": table, "summary": {f: getattr(sm, f) for f, _ in Summary._fields_},
            "diag": diag_dict(dg)}


def aggregate_dispatch(tr, match, range_id, op=None, agg_kind=None, absent_mask=0,
                       library=None):
    """Eq. 1 per operator dispatch: rows 0..R-1 the ranges, R + o the kernels
    of operator o outside a range of o, R + n_ops the unattributed ones."""
    L = library if library is not None else lib()
    x = _Inputs(tr, absent_mask)
    match = np.ascontiguousarray(match, dtype=np.int32)
    rid = np.ascontiguousarray(range_id, dtype=np.int32)
    opa = None if op is None else np.ascontiguousarray(op, dtype=np.int32)
    G = x.r_start.size + tr["n_ops"] + 1
    table = np.zeros(G, dtype=ROW_DTYPE)
    sm = Summary()
    dg = Diag()
    kind = None if agg_kind is None else np.ascontiguousarray(agg_kind, dtype=np.uint8)
    rc = L.oref_aggregate_dispatch(C.byref(x.k), C.byref(x.p), _ptr(match), _ptr(rid), _ptr(opa),
                                   C.byref(x.r), C.byref(x.d), _ptr(kind), _ptr(table),
                                   C.byref(sm), C.byref(dg))
    if rc:
        raise ValueError(f"oref_aggregate_dispatch: {rc}")
    L.oref_diag_finish(C.byref(dg), PREFIX)
    return {"table": table, "summary": {f: getattr(sm, f) for f, _ in Summary._fields_},
            "diag": diag_dict(dg)}


def enclose_all(tr, library=None):
    """All enclosing ranges of every kernel (Alg. 2's all_enclosing) as CSR:
    ``off`` (T + 1) and ``ids``, innermost first."""
    L = library if library is not None else lib()
    x = _Inputs(tr)
    T = x.seq.size
    off = np.empty(T + 1, dtype=np.int64)
    dg = Diag()
    rc = L.oref_enclose_all(C.byref(x.k), C.byref(x.r), C.byref(x.d), _ptr(off), None, 0,
                            C.byref(dg))
    if rc:
        raise ValueError(f"oref_enclose_all: {rc}")
    ids = np.empty(max(int(off[-1]), 1), dtype=np.int32)
    dg = Diag()
    rc = L.oref_enclose_all(C.byref(x.k), C.byref(x.r), C.byref(x.d), _ptr(off), _ptr(ids),
                            int(off[-1]), C.byref(dg))
    if rc:
        raise ValueError(f"oref_enclose_all: {rc}")
    L.oref_diag_finish(C.byref(dg), PREFIX)
    return {"off": off, "ids": ids[:int(off[-1])], "diag": diag_dict(dg)}
