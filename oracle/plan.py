"""Batching-aware memory plan for the node-state arena (Section 3).

Section 3.1: a batched operator wants each batch's source and result operands
contiguous and aligned in memory (the adjacency and alignment constraints);
otherwise a gather runs before the batch and a scatter after it.  The paper
solves the full constraint system with a PQ tree (Section 3.2) and notes that
its cost is too high for the runtime path of dynamic graphs.  The plan here is
the runtime reading: one reverse pass over the batch schedule in which each
consumer claims fresh, consecutive slots for its operand lists before their
producers are placed, so that the producers' results and most operands
become contiguous.

Rule (reverse pass, b = B-1 .. 0; slot 0 is the ZERO row):
  1. order_b = batch b stably sorted by slot, unset slots last; every unset
     node of order_b, in that order, takes the next slot.
  2. Operand lists of batch b: one per positional child p,
     L_p = [child_p(v) for v in order_b], then, for types with ragged
     children, L_r = [the present ragged children of v, CSR order, for v in order_b].
  3. Per list: no present entry -> NONE.  All present entries unset and
     distinct -> fresh: in list order an absent entry takes a new pad slot
     (zero, never written) and a node takes the next slot, so the list is
     contiguous.  Otherwise every unset present entry takes the next slot in
     list order and absent entries read slot 0.
A list is CONTIG(base) when its slots are consecutive, else GATHER; results
are CONTIG when slot[order_b] is consecutive, else SCATTER.  x rows are
numbered in (batch, order_b) order so every x operand is contiguous.

The IDENTITY layout (slot[v] = v + 1, every operand indexed) is the
unplanned baseline of the ablation.  The PQ layout (Section 3.2) takes its
slots from the PQ-tree algorithm in `pqplan`; each batch's rows then follow
their slots, and an absent positional child reads its own zero pad.
"""
from __future__ import annotations

import numpy as np

SEG_NONE = 0
SEG_CONTIG = 1
SEG_GATHER = 2
SEG_SCATTER = 3

PLAN_RC = 0
PLAN_IDENTITY = 1
PLAN_PQ = 2

UNSET = -1


class Plan:
    def __init__(self):
        self.slot = None          # int32 [V]
        self.n_slots = 0
        self.order = []           # per batch: list of node ids (row order)
        self.x_slot = None        # int32 [V], -1 for nodes without x
        self.results = []         # per batch: (kind, [slots])
        self.segments = []        # per batch: [(kind, [slots]) per list]
        self.ragged_ptr = []      # per batch: row offsets into the ragged list, or None
        self.pads = []            # pad slots


def _lists(v_order, child_ptr, child_idx, n_fixed, ragged):
    lists = []
    for p in range(n_fixed):
        lists.append([int(child_idx[child_ptr[v] + p]) for v in v_order])
    rptr = None
    if ragged:
        rl, rptr = [], [0]
        for v in v_order:
            for c in child_idx[child_ptr[v] + n_fixed:child_ptr[v + 1]]:
                if c >= 0:
                    rl.append(int(c))
            rptr.append(len(rl))
        lists.append(rl)
    return lists, rptr


def _kind_of(slots, indexed_kind):
    if all(slots[i + 1] == slots[i] + 1 for i in range(len(slots) - 1)):
        return SEG_CONTIG
    return indexed_kind


def plan_memory(op_type, child_ptr, child_idx, batches, shapes, mode=PLAN_RC):
    """shapes[t] = (n_fixed, ragged, has_x).  Returns a Plan."""
    V = int(len(op_type))
    pl = Plan()
    slot = np.full(V, UNSET, dtype=np.int64)
    B = len(batches)
    orders = [None] * B
    seg_lists = [None] * B
    rptrs = [None] * B
    pad_of = {}   # (batch, list index, entry index) -> pad slot

    if mode == PLAN_IDENTITY:
        for v in range(V):
            slot[v] = v + 1
        nxt = V + 1
        for b in range(B):
            orders[b] = list(batches[b])
            t = int(op_type[orders[b][0]])
            nf, rg = shapes[t][0], shapes[t][1]
            seg_lists[b], rptrs[b] = _lists(orders[b], child_ptr, child_idx, nf, rg)
    elif mode == PLAN_RC:
        nxt = 1
        for b in range(B - 1, -1, -1):
            nodes = list(batches[b])
            # stable sort by slot, unset last
            order_b = sorted(nodes, key=lambda v: (slot[v] == UNSET, slot[v] if slot[v] != UNSET else 0))
            for v in order_b:
                if slot[v] == UNSET:
                    slot[v] = nxt
                    nxt += 1
            orders[b] = order_b
            t = int(op_type[order_b[0]])
            nf, rg = shapes[t][0], shapes[t][1]
            lists, rptr = _lists(order_b, child_ptr, child_idx, nf, rg)
            seg_lists[b], rptrs[b] = lists, rptr
            for li, L in enumerate(lists):
                real = [c for c in L if c >= 0]
                if not real:
                    continue
                fresh = all(slot[c] == UNSET for c in real) and len(set(real)) == len(real)
                if fresh:
                    for ei, c in enumerate(L):
                        if c < 0:
                            pad_of[(b, li, ei)] = nxt
                            pl.pads.append(nxt)
                        else:
                            slot[c] = nxt
                        nxt += 1
                else:
                    for c in L:
                        if c >= 0 and slot[c] == UNSET:
                            slot[c] = nxt
                            nxt += 1
    elif mode == PLAN_PQ:
        from .pqplan import pq_layout
        slot_of, pad_var, lead, pl.pq_stats = pq_layout(op_type, child_ptr, child_idx, batches, shapes)
        for v in range(V):
            slot[v] = slot_of[v]
        nxt = len(slot_of) + 1
        pl.pads = sorted(slot_of[x] for x in pad_var.values())
        for b in range(B):
            if lead[b] == 0:
                order_b = sorted(batches[b], key=lambda v: slot[v])
            else:
                p = lead[b] - 1

                def key(v, b=b, p=p):
                    c = int(child_idx[child_ptr[v] + p])
                    return slot_of[c] if c >= 0 else slot_of[pad_var[(b, p, v)]]
                order_b = sorted(batches[b], key=key)
            orders[b] = order_b
            t = int(op_type[order_b[0]])
            nf, rg = shapes[t][0], shapes[t][1]
            seg_lists[b], rptrs[b] = _lists(order_b, child_ptr, child_idx, nf, rg)
            for p in range(nf):
                for ei, v in enumerate(order_b):
                    if (b, p, v) in pad_var:
                        pad_of[(b, p, ei)] = slot_of[pad_var[(b, p, v)]]
    else:
        raise ValueError("unknown plan mode")

    if (slot == UNSET).any():
        raise ValueError("node left without a slot (not scheduled?)")
    pl.slot = slot.astype(np.int32)
    pl.n_slots = int(nxt)
    pl.order = orders

    xs = np.full(V, -1, dtype=np.int32)
    nx = 0
    for b in range(B):
        t = int(op_type[orders[b][0]])
        if shapes[t][2]:
            for v in orders[b]:
                xs[v] = nx
                nx += 1
    pl.x_slot = xs

    indexed = mode == PLAN_IDENTITY
    for b in range(B):
        rs = [int(slot[v]) for v in orders[b]]
        pl.results.append((SEG_SCATTER if indexed else _kind_of(rs, SEG_SCATTER), rs))
        segs = []
        for li, L in enumerate(seg_lists[b]):
            if not any(c >= 0 for c in L):
                segs.append((SEG_NONE, []))
                continue
            ss = []
            for ei, c in enumerate(L):
                if c >= 0:
                    ss.append(int(slot[c]))
                else:
                    ss.append(int(pad_of.get((b, li, ei), 0)))
            segs.append((SEG_GATHER if indexed else _kind_of(ss, SEG_GATHER), ss))
        pl.segments.append(segs)
        pl.ragged_ptr.append(rptrs[b])
    return pl


def hazard_check(op_type, child_ptr, child_idx, batches, plan):
    """Each node's slot is written exactly once (slots injective, never the
    ZERO row or a pad); every slot a batch reads is the ZERO row, a pad, or
    the slot of a node finished in an earlier batch."""
    V = int(len(op_type))
    slot = plan.slot
    when = np.full(V, -1)
    for b, batch in enumerate(batches):
        for v in batch:
            when[v] = b
    if len(set(int(s) for s in slot)) != V:
        raise AssertionError("slots not injective")
    if (slot <= 0).any() or (slot >= plan.n_slots).any():
        raise AssertionError("node slot out of range or ZERO")
    pads = set(plan.pads)
    if pads & set(int(s) for s in slot):
        raise AssertionError("pad slot written")
    owner = {int(slot[v]): v for v in range(V)}
    for b in range(len(batches)):
        kind, rs = plan.results[b]
        if rs != [int(slot[v]) for v in plan.order[b]]:
            raise AssertionError("result slots inconsistent")
        for kind, ss in plan.segments[b]:
            for s in ss:
                if s == 0 or s in pads:
                    continue
                v = owner.get(s)
                if v is None or when[v] >= b:
                    raise AssertionError(f"batch {b} reads slot {s} before it is written")
    return True


def contig_fraction(plan):
    """(contiguous source operands, present source operands, contiguous results, batches)."""
    cs = ns = 0
    for segs in plan.segments:
        for kind, _ in segs:
            if kind != SEG_NONE:
                ns += 1
                cs += kind == SEG_CONTIG
    cr = sum(1 for kind, _ in plan.results if kind == SEG_CONTIG)
    return cs, ns, cr, len(plan.results)
