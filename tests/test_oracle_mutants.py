"""Plant one plausible mistake at a time in a copy of the oracle (on the CPU)
and check that the pins catch it: an off-by-one, a reversed order, a dropped
term, a wrong comparison. Every mutant must fail the pin battery; the
unmodified source must pass it."""
import math
import os
import subprocess

import numpy as np
import pytest

import brute
import cases
from oracle import oracle as O

SRC = open(O.SRC).read()

MUTANTS = {
    "iom_descending_seq": ("ord[ne].a = k->seq[i];", "ord[ne].a = UINT32_MAX - k->seq[i];"),
    "iom_rank_not_advanced": ("const int64_t r = tl_cnt[n]++;", "const int64_t r = 0 * tl_cnt[n]++;"),
    "iom_rank_off_by_one": ("if (r < pf_cnt[n]) match[i] = (int32_t)rows[pf_off[n] + r];",
                            "if (r + 1 < pf_cnt[n]) match[i] = (int32_t)rows[pf_off[n] + r + 1];"),
    "iom_skip_name_ignored": ("if (tl_cnt[n] != pf_cnt[n]) match[i] = -1;",
                              "if (0) match[i] = -1;"),
    "dedup_reversed_position": ("int64_t src = mem[off[r] + pos].idx;",
                                "int64_t src = mem[off[r] + cnt[r] - 1 - pos].idx;"),
    "dedup_contiguity_on_seq_values": ("e->a = (uint64_t)q;\n    e->b = (uint64_t)rank[i];",
                                       "e->a = (uint64_t)q;\n    e->b = k->seq[i];"),
    "classes_contiguity_on_seq_values": ("e->a = (uint64_t)p;\n    e->b = (uint64_t)rank[i];",
                                         "e->a = (uint64_t)p;\n    e->b = k->seq[i];"),
    "dedup_no_name_check": ("ok = k->name_id[src] == k->name_id[i];", "ok = 1;"),
    "enclose_end_ascending": ("rs[nr].c = UINT64_MAX - r->end_ns[x];",
                              "rs[nr].c = r->end_ns[x];"),
    "enclose_open_at_start_excluded": ("while (*x < a_end && rs[*x].b <= t)",
                                       "while (*x < a_end && rs[*x].b < t)"),
    "enclose_closed_at_end_excluded": ("while (*top > 0 && r->end_ns[stack[*top - 1]] < t) (*top)--;",
                                       "while (*top > 0 && r->end_ns[stack[*top - 1]] <= t) (*top)--;"),
    "depth_root_zero": ("depth[id] = top > 0 ? depth[stack[top - 1]] + 1 : 1;",
                        "depth[id] = top > 0 ? depth[stack[top - 1]] + 1 : 0;"),
    "nesting_touch_is_cross": ("while (top > 0 && r->end_ns[stack[top - 1]] <= r->start_ns[id]) top--;",
                               "while (top > 0 && r->end_ns[stack[top - 1]] < r->start_ns[id]) top--;"),
    "dw_without_duration": ("nadd(&acc[x], v * (double)dur); /* m_i * d_i */",
                            "nadd(&acc[x], v);"),
    "max_is_min": ("else if (isnan(v) || v > mx[x]) mx[x] = v;",
                   "else if (isnan(v) || v < mx[x] || isinf(mx[x])) mx[x] = v;"),
    "absent_mask_ignored": ("if (((p->absent_mask >> c) & 1u) || row->matched_count == 0)",
                            "if (row->matched_count == 0)"),
    "unmatched_in_dw_denominator": ("if (m < 0) continue; /* unmatched kernels carry no counters */",
                                    "if (m < 0) { row->matched_ns += dur; continue; }"),
    "unattributed_dropped": ("row->kernel_count++;", "if (g < d->n_ops) row->kernel_count++;"),
    "walk_skip_ends_walk": ("if (kd == OREF_KIND_SKIP) continue;",
                            "if (kd == OREF_KIND_SKIP) break;"),
    "walk_boundary_passed": ("if (kd == OREF_KIND_BOUNDARY) break;",
                             "if (kd == OREF_KIND_BOUNDARY) continue;"),
    "walk_outermost_op_kept": ("if (first < 0) first = (int32_t)id;", "first = (int32_t)id;"),
    "fused_counts_every_range": ("if (fused) fused[i] = nops > 1 ? 1 : 0;",
                                 "if (fused) fused[i] = top > 1 ? 1 : 0;"),
    "classes_names_only": ("eq = k->name_id[a] == k->name_id[b] && k->stream_id[a] == k->stream_id[b];",
                           "eq = k->name_id[a] == k->name_id[b];"),
    "classes_contiguity_ignored": ("contig[q] = (hi - lo + 1 == (uint64_t)cnt[q]);\n    if (!contig[q]) diag->flags |= OREF_F_PARTITION;\n  }\n\n  /* sort partitions",
                                   "contig[q] = 1;\n  }\n\n  /* sort partitions"),
    "ranks_order_unchecked": ("if (all[x].a == all[x - 1].a) { diag->flags |= OREF_F_ORDER; break; }",
                              "if (0) break;"),
    "classes_never_grouped": ("part_rep[q] = (int32_t)head;", "part_rep[q] = (int32_t)q;"),
    "tiers_nvtx_before_high": ("if (e >= 0 && corr->op_id[e] >= 0 && (uint32_t)corr->op_id[e] < NOPS) {",
                               "if (rid < 0 && e >= 0 && corr->op_id[e] >= 0 && (uint32_t)corr->op_id[e] < NOPS) {"),
    "tiers_fusion_overrides_nvtx": ("} else if (rid >= 0 && rid < r->n) {",
                                    "} else if (rid >= 0 && rid < r->n && nf == 0) {"),
    "tiers_fused_not_augmented": ("fused[i] = (uint8_t)(((walk_fused && walk_fused[i]) || nf > 1) ? 1 : 0);",
                                  "fused[i] = (uint8_t)((walk_fused && walk_fused[i]) ? 1 : 0);"),
    "tiers_index_with_dedup": ("kk.part_id = NULL;\n    oref_dims dd = *d;\n    dd.part_rep = NULL;\n    dd.n_parts = 0;",
                               "oref_dims dd = *d;"),
    "tiers_fusion_last_op": ("o = fm->op_id[fm->off[nm]];", "o = fm->op_id[fm->off[nm + 1] - 1];"),
    "coverage_counts_kernels": ("cov->ns[t] += k->dur_ns[i];", "cov->ns[t] += 1;"),
    "dispatch_ignores_operator": ("if (rid >= 0 && rid < R && o >= 0 && (uint32_t)o == r->op_id[rid] && (uint32_t)o < NOPS)",
                                  "if (rid >= 0 && rid < R && o >= 0 && (uint32_t)o < NOPS)"),
    "dispatch_op_row_shifted": ("row_of[i] = (uint32_t)(R + o);", "row_of[i] = (uint32_t)(R + o - (o > 0));"),
    "all_outermost_first": ("for (int64_t u = top - 1; u >= 0; --u) {\n          const int64_t id = stack[u];\n          if (r->end_ns[id] < t) continue; /* ended before the point */",
                            "for (int64_t u = 0; u < top; ++u) {\n          const int64_t id = stack[u];\n          if (r->end_ns[id] < t) continue; /* ended before the point */"),
    "all_touching_excluded": ("if (r->end_ns[id] < t) continue; /* ended before the point */",
                              "if (r->end_ns[id] <= t) continue; /* ended before the point */"),
    "counters_out_absent_ignored": ("if (m >= 0 && m < p->n && !((p->absent_mask >> c) & 1u))",
                                    "if (m >= 0 && m < p->n)"),
    "counters_out_strides_swapped": (
        "v = p->counters[(int64_t)m * p->row_stride + (int64_t)c * p->col_stride];",
        "v = p->counters[(int64_t)m * p->col_stride + (int64_t)c * p->row_stride];"),
    "counters_out_no_upper_bound": ("if (m >= 0 && m < p->n && !((p->absent_mask >> c) & 1u))",
                                    "if (m >= 0 && !((p->absent_mask >> c) & 1u))"),
    "parent_is_root": ("if (range_parent) range_parent[id] = top > 0 ? (int32_t)stack[top - 1] : -1;",
                       "if (range_parent) range_parent[id] = top > 0 ? (int32_t)stack[0] : -1;"),
}


def _build(tmp_path, name, src):
    c = tmp_path / f"{name}.c"
    so = tmp_path / f"{name}.so"
    c.write_text(src)
    subprocess.run(["gcc", "-O1", "-std=c11", "-fPIC", "-shared", "-ffp-contract=off",
                    "-I", os.path.dirname(O.SRC), "-o", str(so), str(c), "-lm"], check=True)
    return O.load(str(so))


def _edge_trace():
    q = np.array([5, 10, 20, 25, 30, 35, 60], np.uint64)
    T = q.size
    return dict(seq=np.arange(T, dtype=np.uint32), start_ns=q, dur_ns=np.arange(1, T + 1, dtype=np.uint32),
                stream_id=np.zeros(T, np.uint16), name_id=np.zeros(T, np.uint32), part_id=None,
                pf_name=np.zeros(T, np.uint32),
                counters=np.random.default_rng(0).random((T, 20), dtype=np.float32),
                r_start=np.array([10, 10, 20, 25, 40], np.uint64),
                r_end=np.array([20, 20, 30, 25, 50], np.uint64),
                r_stream=np.zeros(5, np.uint16), r_op=np.arange(5, dtype=np.uint32),
                part_rep=None, n_names=1, n_streams=1, n_ops=5)


def _rows_close(out, want, rtol=1e-12):
    for a, b in zip(out["table"], want):
        for f in ("kernel_count", "total_ns", "matched_count", "matched_ns"):
            if int(a[f]) != b[f]:
                return False
        for x, y in zip(a["value"], b["value"]):
            if math.isnan(y) != math.isnan(float(x)):
                return False
            if not math.isnan(y) and abs(float(x) - y) > rtol * max(abs(float(x)), abs(y)):
                return False
    return True


def battery(L) -> bool:
    """True when every pin holds for library L."""
    for seed in range(8):
        tr = cases.random_trace(seed, T=40, drop=0.2 if seed % 2 else 0.0,
                                dedup=seed % 3 == 0)
        for pol in (O.PREFIX, O.SKIP_NAME):
            got = O.attribute(tr, policy=pol, stages=["match"], library=L)["match_iom"]
            if not np.array_equal(got, brute.iom(tr, policy=1 if pol == O.SKIP_NAME else 0)):
                return False
    for seed in range(8):
        tr = cases.random_trace(100 + seed, T=60, dedup=True, seq_gaps=seed % 2 == 0)
        tr["name_id"] = tr["name_id"].copy()
        if seed % 2:
            tr["name_id"][int(np.argmax(tr["part_id"]))] ^= 1  # one foreign name
        out = O.attribute(tr, stages=["match", "dedup"], library=L)
        want, errs = brute.dedup(tr, brute.iom(tr))
        if not np.array_equal(out["match"], want) or out["diag"]["dedup_errors"] != errs:
            return False
    for seed in range(12):
        tr = cases.random_trace(200 + seed, T=60, R=25, S=2, t_max=30,
                                nested=seed % 4 != 3)
        out = O.attribute(tr, stages=["match", "enclose"], library=L)
        if not np.array_equal(out["range_id"], brute.enclose(tr)):
            return False
        if not np.array_equal(out["range_depth"], np.minimum(brute.depth(tr), 255)):
            return False
        if out["diag"]["nesting_errors"] != len(brute.crossing_streams(tr)):
            return False
    for seed in range(6):
        tr = cases.random_trace(700 + seed, T=60, R=30, S=2, t_max=40, max_depth=5)
        rng = np.random.default_rng(seed)
        u = rng.random(tr["r_start"].size)
        tr["r_kind"] = np.where(u < 0.2, 1, np.where(u < 0.45, 2, 0)).astype(np.uint8)
        out = O.enclose_walk(tr, library=L)
        rid, fused, rany, par = brute.enclose_walk(tr)
        for got, want in ((out["range_id"], rid), (out["fused"], fused),
                          (out["range_any"], rany), (out["range_parent"], par)):
            if not np.array_equal(got, want):
                return False
    import test_oracle
    for seed in range(8):
        tr = test_oracle._class_trace(seed, noncontig=seed % 3 == 1, bad=seed % 4 == 3)
        if seed % 4 == 2:  # two launches share a seq value
            tr["seq"] = tr["seq"].copy()
            tr["seq"][7] = tr["seq"][3]
        out = O.dedup_classes(tr, library=L)
        rep, has_nc = brute.dedup_classes(tr)
        if not np.array_equal(out["part_rep"], rep) or bool(out["diag"]["flags"] & 16) != has_nc:
            return False
        if bool(out["diag"]["flags"] & 2) != (np.unique(tr["seq"]).size < tr["seq"].size):
            return False
    for seed in range(6):
        tr = test_oracle._tier_trace(seed, T=80, dedup=seed % 2 == 0, shuffle=seed % 3 == 1)
        for pol in (0, 1):
            out = O.tiers(tr, corr_policy=pol, library=L)
            tier, op, fused, cnt, ns = brute.tiers(tr, pol)
            if not (np.array_equal(out["tier"], tier) and np.array_equal(out["op"], op)
                    and np.array_equal(out["fused"], fused)
                    and list(out["coverage"]["count"]) == cnt
                    and list(out["coverage"]["ns"]) == ns):
                return False
    for seed in range(4):
        tr, match, t = test_oracle._dispatch_case(seed)
        out = O.aggregate_dispatch(tr, match, t["range_id"], t["op"], library=L)
        keys = brute.dispatch_keys(tr, t["range_id"], t["op"])
        want = brute.aggregate_groups(tr, match, keys, tr["r_start"].size + tr["n_ops"] + 1)
        if not _rows_close(out, want):
            return False
    for seed in range(4):
        tr = cases.random_trace(960 + seed, T=60, R=30, S=2, t_max=40, max_depth=4)
        out = O.enclose_all(tr, library=L)
        want = brute.enclosing_lists(tr)
        if int(out["off"][-1]) != sum(len(w) for w in want):
            return False
        for i, w in enumerate(want):
            if list(out["ids"][out["off"][i]:out["off"][i + 1]]) != w:
                return False
    tr = _edge_trace()
    out = O.attribute(tr, library=L)
    if not np.array_equal(out["range_id"], brute.enclose(tr)):
        return False
    if not _rows_close(out, brute.aggregate(tr, out["match"], out["range_id"])):
        return False
    import test_oracle
    tr = test_oracle._dedup_case()
    # three rows of a larger block, so that a mistaken stride stays in bounds
    big = (1000 * np.arange(20)[:, None] + np.arange(20)[None, :]).astype(np.float32)
    rows = big[:3]
    tr["counters"] = rows
    m = O.attribute(tr, stages=["match", "dedup"], library=L)["match"]
    got = O.counters_out(tr, m, absent_mask=1 << 7, library=L)
    want = rows[[0, 1, 2] * 3].copy()
    want[:, 7] = np.nan
    if not np.array_equal(got, want, equal_nan=True):
        return False
    got = O.counters_out(dict(tr, counters=np.asfortranarray(rows)),
                         np.array([2, -1, 3], np.int32), library=L)
    if not (np.array_equal(got[0], rows[2]) and np.isnan(got[1:]).all()):
        return False
    for seed in range(6):
        tr = cases.random_trace(400 + seed, T=80, R=20, drop=0.3)
        absent = (1 << 4) if seed % 2 else 0
        out = O.attribute(tr, absent_mask=absent, library=L)
        if not _rows_close(out, brute.aggregate(tr, out["match"], out["range_id"], None, absent)):
            return False
    return True


def test_unmodified_oracle_passes_battery(tmp_path):
    assert battery(_build(tmp_path, "orig", SRC))


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(tmp_path, name):
    old, new = MUTANTS[name]
    assert SRC.count(old) == 1, f"mutation site for {name} not found exactly once"
    L = _build(tmp_path, name, SRC.replace(old, new))
    assert not battery(L), f"mutant {name} survived the pins"
