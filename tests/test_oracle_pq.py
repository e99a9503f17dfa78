"""Pins of the oracle's PQ tree and PQ-tree memory layout (Section 3.2,
Appendix B): the tree represents exactly the permutations that keep every
applied set consecutive (brute force over all permutations of up to 7
leaves) and rejects exactly the sets no such permutation allows; the layout
of Figure 3 is ideal; every batch whose relations all merged is contiguous
and aligned in the final layout; the grid's ideal layout is found; plans are
hazard free.  CPU only."""
import itertools
import json
import os

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

from oracle import plan as P
from oracle import pqplan as Q
from oracle import schedule as S
from oracle.pqtree import LEAF, PNODE, QNODE, PQTree
from paper_2302_03851_amd import workloads as WL


def _consecutive(perm, A):
    pos = sorted(perm.index(x) for x in A)
    return pos[-1] - pos[0] == len(A) - 1


def _tree_ok(t):
    for x in range(len(t.kind)):
        if not t.alive[x] or t.kind[x] == LEAF or (x != t.root and t.parent[x] < 0):
            continue
        k = len(t.children[x])
        assert (t.kind[x] == PNODE and k >= 2) or (t.kind[x] == QNODE and k >= 3)
        assert all(t.parent[c] == x for c in t.children[x])


@settings(max_examples=300, deadline=None)
@given(st.integers(1, 7).flatmap(
    lambda n: st.tuples(st.just(n), st.lists(st.lists(st.integers(0, n - 1), min_size=1, max_size=n, unique=True),
                                             max_size=6))))
def test_pq_tree_represents_exactly_the_consecutive_permutations(case):
    n, sets = case
    t = PQTree(n)
    applied = []
    for A in sets:
        allowed = [p for p in itertools.permutations(range(n)) if all(_consecutive(p, B) for B in applied)]
        ok, _ = t.reduce(A)
        assert ok == any(_consecutive(p, A) for p in allowed)
        if ok:
            applied.append(A)
        _tree_ok(t)
        fr = t.frontier()
        assert sorted(fr) == list(range(n))
        assert all(_consecutive(fr, B) for B in applied)
        assert t.count_frontiers() == sum(
            1 for p in itertools.permutations(range(n)) if all(_consecutive(p, B) for B in applied))


def test_pq_tree_templates_by_hand():
    # {0,1} then {1,2} on 4 leaves: 0-1-2 must be a path, read in either
    # direction, with leaf 3 before or after it: 4 permutations.
    t = PQTree(4)
    assert t.reduce([0, 1]) == (True, True)
    assert t.reduce([1, 2]) == (True, True)
    assert t.count_frontiers() == 4     # (0 1 2 | 2 1 0) x (3 first | 3 last)
    assert t.reduce([0, 2]) == (False, False)
    assert t.reduce([2, 1]) == (True, False)   # implied
    assert t.reduce([0, 1, 2]) == (True, False)


def _fig3(golden_dir):
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


def test_fig3_pq_layout_is_ideal(golden_dir):
    # Section 3.1: the ideal layout makes every source and result operand of
    # both batches contiguous and aligned; the PQ-tree algorithm finds one.
    g, names, op, ptr, idx = _fig3(golden_dir)
    batches, _ = S.schedule(op, ptr, idx, 3)
    pl = P.plan_memory(op, ptr, idx, batches, [(0, 0, 0), (2, 0, 0), (1, 0, 0)], P.PLAN_PQ)
    P.hazard_check(op, ptr, idx, batches, pl)
    assert all(k == P.SEG_CONTIG for k, _ in pl.results)
    assert all(k == P.SEG_CONTIG for segs in pl.segments for k, _ in segs if k != P.SEG_NONE)
    order = sorted(range(8), key=lambda v: pl.slot[v])
    pos = {names[v]: i for i, v in enumerate(order)}
    for A in g["printed"]["adjacency_sets"]:
        p = sorted(pos[x] for x in A)
        assert p == list(range(p[0], p[0] + len(p)))
    assert pl.pq_stats["decided"] == 2


def _aligned_in_layout(op, ptr, idx, rows, b, nf, slot_of, pad_of):
    """Every positional operand of batch b contiguous and aligned with the
    rows in the layout (rows ordered by their slots)."""
    rows = sorted(rows, key=lambda v: slot_of[v])
    rs = [slot_of[v] for v in rows]
    if rs != list(range(rs[0], rs[0] + len(rs))):
        return False
    for p in range(nf):
        L = [int(idx[ptr[v] + p]) for v in rows]
        real = [c for c in L if c >= 0]
        if not real or len(set(real)) < len(real):
            continue     # no operand, or a repeated child: not an aligned operand
        ss = [slot_of[c] if c >= 0 else slot_of[pad_of[(b, p, v)]] for c, v in zip(L, rows)]
        if ss != list(range(ss[0], ss[0] + len(ss))):
            return False
    return True


@st.composite
def tiny_batched(draw):
    """Random typed DAGs of up to 10 nodes with 0-2 positional children."""
    n = draw(st.integers(2, 10))
    T = draw(st.integers(1, 3))
    nf = [draw(st.integers(0, 2)) for _ in range(T)]
    op, children = [], []
    for v in range(n):
        t = draw(st.integers(0, T - 1))
        op.append(t)
        children.append([draw(st.integers(-1, v - 1)) if v else -1 for _ in range(nf[t])])
    return np.array(op, dtype=np.int32), children, T, [(nf[t], 0, 0) for t in range(T)]


@settings(max_examples=150, deadline=None)
@given(tiny_batched())
def test_decided_batches_are_contiguous_and_aligned(g):
    op, children, T, shapes = g
    ptr = np.zeros(len(children) + 1, dtype=np.int64)
    for v, ch in enumerate(children):
        ptr[v + 1] = ptr[v] + len(ch)
    idx = np.array([c for ch in children for c in ch], dtype=np.int32)
    batches, _ = S.schedule(op, ptr, idx, T)
    pl = P.plan_memory(op, ptr, idx, batches, shapes, P.PLAN_PQ)
    P.hazard_check(op, ptr, idx, batches, pl)
    slot_of, pad_of, lead, stats = Q.pq_layout(op, ptr, idx, batches, shapes)
    assert sorted(slot_of) == list(range(1, len(slot_of) + 1))       # a permutation of the variables
    # every batch whose group kept all of its operands and whose relations
    # all merged must come out contiguous and aligned
    for b in stats["fully_decided"]:
        nf = shapes[int(op[batches[b][0]])][0]
        assert _aligned_in_layout(op, ptr, idx, batches[b], b, nf, slot_of, pad_of), b


def test_grid_layout_is_ideal():
    # 2D grids: diagonal d's results, left and top operands can all be made
    # contiguous and aligned (one zero pad per absent neighbour).
    w = WL.make_config(4, instances=2)
    batches, _ = S.schedule(w.op_type, w.child_ptr, w.child_idx, w.n_types)
    shapes = [(nf, rg, int(WL.KIND_SHAPE[k][2])) for (nf, rg), k in zip(w.shapes(), w.kinds)]
    pl = P.plan_memory(w.op_type, w.child_ptr, w.child_idx, batches, shapes, P.PLAN_PQ)
    P.hazard_check(w.op_type, w.child_ptr, w.child_idx, batches, pl)
    cs, ns, cr, nb = P.contig_fraction(pl)
    assert (cs, cr) == (ns, nb)


@pytest.mark.parametrize("k", [1, 2, 3, 4, 5])
def test_pq_plan_hazard_free_and_consistent(k):
    w = WL.make_config(k, instances={1: 8, 2: 8, 3: 4, 4: 2, 5: 4}[k])
    table = {(0,): 0, (1,): 1, (0, 1): 0, (1, 0): 1} if k == 3 else None
    batches, _ = S.schedule(w.op_type, w.child_ptr, w.child_idx, w.n_types, table=table)
    shapes = [(nf, rg, int(WL.KIND_SHAPE[kk][2])) for (nf, rg), kk in zip(w.shapes(), w.kinds)]
    pl = P.plan_memory(w.op_type, w.child_ptr, w.child_idx, batches, shapes, P.PLAN_PQ)
    P.hazard_check(w.op_type, w.child_ptr, w.child_idx, batches, pl)
    for b, batch in enumerate(batches):
        assert sorted(pl.order[b]) == sorted(batch)
        for kind, ss in pl.segments[b]:
            if kind == P.SEG_CONTIG:
                assert ss == list(range(ss[0], ss[0] + len(ss)))
    rc = P.plan_memory(w.op_type, w.child_ptr, w.child_idx, batches, shapes, P.PLAN_RC)
    cs, ns, cr, nb = P.contig_fraction(pl)
    cs0, ns0, cr0, nb0 = P.contig_fraction(rc)
    if k in (1, 2):
        # chains and binary trees keep every operand contiguous, as the
        # reverse pass does, with at least as many contiguous results
        assert cs == ns == cs0 and cr >= cr0
    if k == 4:
        assert cs == ns > cs0 and cr == cr0 == nb     # both grid neighbours contiguous
    if k == 3:
        assert cr > cr0


# A batch whose rows cannot be made consecutive and whose first child list is
# absent in every row (so not an operand): its rows follow its second child
# list, and that list must come out contiguous.
SKIPPED_LIST_CASE = ([0, 0, 0, 1, 1, 1, 1], [[], [], [], [-1, 2], [-1, 3], [-1, 0], [3, 0]])


def test_rows_follow_the_leading_operand_after_a_skipped_list():
    op, children = SKIPPED_LIST_CASE
    op = np.array(op, dtype=np.int32)
    ptr = np.zeros(len(children) + 1, dtype=np.int64)
    for v, ch in enumerate(children):
        ptr[v + 1] = ptr[v] + len(ch)
    idx = np.array([c for ch in children for c in ch], dtype=np.int32)
    batches, _ = S.schedule(op, ptr, idx, 2, S.POLICY_DEPTH)
    shapes = [(0, 0, 0), (2, 0, 0)]
    _slot, _pads, lead, _st = Q.pq_layout(op, ptr, idx, batches, shapes)
    b = next(i for i, bt in enumerate(batches) if bt == [3, 5])
    assert lead[b] == 2                       # positional child 1
    pl = P.plan_memory(op, ptr, idx, batches, shapes, P.PLAN_PQ)
    P.hazard_check(op, ptr, idx, batches, pl)
    assert pl.segments[b][0][0] == P.SEG_NONE
    assert pl.segments[b][1][0] == P.SEG_CONTIG
