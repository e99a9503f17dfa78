"""Pins of the oracle's memory plan: the Figure 3 example of Section 3.1
(golden fixture; hand result of the reverse slot pass), hazard freedom and
descriptor consistency on all configurations.  CPU only."""
import json
import os

import numpy as np
import pytest

from oracle import plan as P
from oracle import schedule as S
from paper_2302_03851_amd import workloads as WL


@pytest.fixture(scope="module")
def fig3(golden_dir):
    with open(os.path.join(golden_dir, "fig3_memory.json")) as f:
        g = json.load(f)
    names = [n["name"] for n in g["nodes"]]
    nid = {n: i for i, n in enumerate(names)}
    op = np.array([g["types"][n["type"]] for n in g["nodes"]], dtype=np.int32)
    children = [[nid[c] for c in n["children"]] for n in g["nodes"]]
    ptr = np.zeros(len(children) + 1, dtype=np.int64)
    for v, ch in enumerate(children):
        ptr[v + 1] = ptr[v] + len(ch)
    idx = np.array([c for ch in children for c in ch], dtype=np.int32)
    return g, names, op, ptr, idx


def test_fig3_label_layout_needs_two_gathers_one_scatter(fig3):
    g, names, op, ptr, idx = fig3
    batches, _ = S.schedule(op, ptr, idx, 3)
    shapes = [(0, 0, 0), (2, 0, 0), (1, 0, 0)]
    # the label layout: slot = label order; operands as listed in the figure
    pl = P.plan_memory(op, ptr, idx, batches, shapes, P.PLAN_IDENTITY)
    alpha, sigma = 1, 2
    gathers = sum(1 for k, ss in pl.segments[alpha] if k != P.SEG_NONE and
                  not all(ss[i + 1] == ss[i] + 1 for i in range(len(ss) - 1)))
    assert gathers == g["printed"]["label_layout_gathers"]
    # sigma's results [x8, x6, x7] in the figure's row order are not aligned in label order
    fig_rows = [names.index(x) for x in ("x8", "x6", "x7")]
    slots = [int(pl.slot[v]) for v in fig_rows]
    assert not all(slots[i + 1] == slots[i] + 1 for i in range(2))


def test_fig3_reverse_pass_hand_result(fig3):
    g, names, op, ptr, idx = fig3
    batches, bt = S.schedule(op, ptr, idx, 3)
    assert bt == [0, 1, 2]
    shapes = [(0, 0, 0), (2, 0, 0), (1, 0, 0)]
    pl = P.plan_memory(op, ptr, idx, batches, shapes, P.PLAN_RC)
    exp = g["reverse_pass_plan"]
    for n, s in exp["slot"].items():
        assert pl.slot[names.index(n)] == s
    assert pl.results[2] == (P.SEG_CONTIG, exp["sigma_results"])
    assert pl.segments[2][0] == (P.SEG_CONTIG, exp["sigma_source"])
    assert pl.results[1] == (P.SEG_CONTIG, exp["alpha_results"])
    assert pl.segments[1][0] == (P.SEG_GATHER, exp["alpha_source_0"])
    assert pl.segments[1][1] == (P.SEG_GATHER, exp["alpha_source_1"])
    assert pl.results[0] == (P.SEG_CONTIG, exp["input_results"])
    P.hazard_check(op, ptr, idx, batches, pl)


def test_fig3_ideal_order_satisfies_constraints(fig3):
    """The printed ideal order makes every operand of both batches
    contiguous and aligned (Section 3.1's two constraints)."""
    g, names, op, ptr, idx = fig3
    pos = {n: i for i, n in enumerate(g["printed"]["ideal_order"])}
    def aligned(lst):
        return all(pos[lst[i + 1]] == pos[lst[i]] + 1 for i in range(len(lst) - 1))
    rows_b1 = sorted(["x4", "x5"], key=pos.get)
    srcs_b1 = [[g["nodes"][names.index(r)]["children"][p] for r in rows_b1] for p in range(2)]
    assert aligned(rows_b1) and all(aligned(s) for s in srcs_b1)
    rows_b2 = sorted(["x6", "x7", "x8"], key=pos.get)
    src_b2 = [g["nodes"][names.index(r)]["children"][0] for r in rows_b2]
    assert aligned(rows_b2) and aligned(src_b2)
    for s in g["printed"]["adjacency_sets"]:
        p = sorted(pos[x] for x in s)
        assert p == list(range(p[0], p[0] + len(p)))


def _shapes(w):
    return [(nf, rg, int(WL.KIND_SHAPE[k][2])) for (nf, rg), k in zip(w.shapes(), w.kinds)]


def _table(k):
    return {(0,): 0, (1,): 1, (0, 1): 0, (1, 0): 1} if k == 3 else None


@pytest.mark.parametrize("k", [1, 2, 3, 4, 5])
@pytest.mark.parametrize("mode", [P.PLAN_RC, P.PLAN_IDENTITY])
def test_plan_hazard_free(k, mode):
    w = WL.make_config(k, instances={1: 8, 2: 16, 3: 8, 4: 4, 5: 8}[k])
    batches, _ = S.schedule(w.op_type, w.child_ptr, w.child_idx, w.n_types, table=_table(k))
    pl = P.plan_memory(w.op_type, w.child_ptr, w.child_idx, batches, _shapes(w), mode)
    P.hazard_check(w.op_type, w.child_ptr, w.child_idx, batches, pl)
    # descriptor consistency
    for b, batch in enumerate(batches):
        assert sorted(pl.order[b]) == sorted(batch)
        for kind, ss in pl.segments[b]:
            if kind == P.SEG_CONTIG:
                assert ss == list(range(ss[0], ss[0] + len(ss)))
        if pl.ragged_ptr[b] is not None:
            assert pl.ragged_ptr[b][-1] == len(pl.segments[b][-1][1])
    # x rows numbered in batch order: every x operand is a contiguous run
    nx = 0
    for b in range(len(batches)):
        for v in pl.order[b]:
            if pl.x_slot[v] >= 0:
                assert pl.x_slot[v] == nx
                nx += 1
    assert nx == int((w.x_row >= 0).sum())


def test_plan_contiguity_expectations():
    # chain: every source operand and result contiguous
    w = WL.make_config(1)
    batches, _ = S.schedule(w.op_type, w.child_ptr, w.child_idx, 1)
    pl = P.plan_memory(w.op_type, w.child_ptr, w.child_idx, batches, _shapes(w))
    cs, ns, cr, nb = P.contig_fraction(pl)
    assert cs == ns and cr == nb
    # binary trees: both child operands contiguous in every internal batch
    w = WL.make_config(2)
    batches, bt = S.schedule(w.op_type, w.child_ptr, w.child_idx, 2)
    pl = P.plan_memory(w.op_type, w.child_ptr, w.child_idx, batches, _shapes(w))
    for b, t in enumerate(bt):
        if t == 1:
            assert all(k == P.SEG_CONTIG for k, _ in pl.segments[b])
    # child-sum trees: the ragged child list contiguous in every internal batch
    w = WL.make_config(5, instances=32)
    batches, bt = S.schedule(w.op_type, w.child_ptr, w.child_idx, 2)
    pl = P.plan_memory(w.op_type, w.child_ptr, w.child_idx, batches, _shapes(w))
    for b, t in enumerate(bt):
        if t == 1:
            assert pl.segments[b][-1][0] == P.SEG_CONTIG


def test_identity_plan_is_labels():
    w = WL.make_config(2, instances=2)
    batches, _ = S.schedule(w.op_type, w.child_ptr, w.child_idx, 2)
    pl = P.plan_memory(w.op_type, w.child_ptr, w.child_idx, batches, _shapes(w), P.PLAN_IDENTITY)
    assert list(pl.slot) == list(range(1, w.n_nodes + 1))
    assert pl.n_slots == w.n_nodes + 1
    assert all(k == P.SEG_SCATTER for k, _ in pl.results)
