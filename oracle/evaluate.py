"""Node-at-a-time evaluation of a typed dataflow graph (the unbatched semantics).

Section 2.1: a mini-batch is the union of per-instance dataflow graphs whose
operations carry a type; batching only groups independent ready operations of
one type, so it must leave every node's result unchanged.  This module
therefore ignores batching and memory planning altogether: it evaluates every
node once, in a topological order given by Kahn's algorithm (smallest ready
node id first), with the float64 cell equations of `oracle.cells`.

bf16 storage (the large child-sum configuration): weights and x arrive holding
bf16 values; each node's h is rounded to bf16 and its c to fp32 at the node
output, because that is what is stored and read by the consumers.
"""
from __future__ import annotations

import heapq

import numpy as np

from . import cells as C


def round_to_bf16(a):
    """Round to the nearest bf16 value, ties to even (via fp32, as stored).

    bf16 keeps the top 16 bits of an IEEE fp32 number; rounding adds half an
    ulp of the kept part (0x7FFF plus the kept part's lowest bit, which makes
    ties go to even) before truncating the low 16 bits.
    """
    f = np.asarray(a, dtype=np.float64).astype(np.float32)
    bits = f.view(np.uint32).astype(np.uint64)
    keep_lsb = (bits >> np.uint64(16)) & np.uint64(1)
    rounded = ((bits + np.uint64(0x7FFF) + keep_lsb) >> np.uint64(16)) << np.uint64(16)
    out = (rounded & np.uint64(0xFFFFFFFF)).astype(np.uint32).view(np.float32)
    out = np.where(np.isnan(f), np.float32(np.nan), out)
    return out.astype(np.float64)


def topo_order(n_nodes, child_ptr, child_idx):
    """Kahn's algorithm over the present (non -1) children, smallest ready id first."""
    pending = np.zeros(n_nodes, dtype=np.int64)
    consumers = [[] for _ in range(n_nodes)]
    for v in range(n_nodes):
        for c in child_idx[child_ptr[v]:child_ptr[v + 1]]:
            if c >= 0:
                pending[v] += 1
                consumers[int(c)].append(v)
    ready = [v for v in range(n_nodes) if pending[v] == 0]
    heapq.heapify(ready)
    order = []
    while ready:
        v = heapq.heappop(ready)
        order.append(v)
        for p in consumers[v]:
            pending[p] -= 1
            if pending[p] == 0:
                heapq.heappush(ready, p)
    if len(order) != n_nodes:
        raise ValueError("graph has a cycle")
    return order


def evaluate(kinds, op_type, child_ptr, child_idx, x_row, x, weights, hidden,
             n_fixed=None, dtype="f32", order=None):
    """Evaluate every node once; return (h, c) as float64 arrays [V, hidden].

    kinds[t]   cell kind of type t (ids in oracle.cells)
    weights[t] dict of logical matrices of type t (names as in the cell functions)
    n_fixed[t] number of positional children of NARY_INTERNAL types (default 2)
    order      optional evaluation order (any topological order gives the same
               result); default Kahn smallest-id-first
    """
    V = int(len(op_type))
    H = int(hidden)
    hs = np.zeros((V, H))
    cs = np.zeros((V, H))
    done = np.zeros(V, dtype=bool)
    bf16 = dtype == "bf16"
    zero = np.zeros(H)
    if order is None:
        order = topo_order(V, child_ptr, child_idx)

    def state(c):
        if c < 0:
            return zero, zero
        if not done[c]:
            raise ValueError(f"child {c} read before it was evaluated")
        return hs[c], cs[c]

    for v in order:
        v = int(v)
        t = int(op_type[v])
        k = int(kinds[t])
        w = weights[t]
        ch = [int(c) for c in child_idx[child_ptr[v]:child_ptr[v + 1]]]
        xv = x[x_row[v]] if x_row[v] >= 0 else None
        if k == C.LSTM_CHAIN:
            hp, cp = state(ch[0])
            h, c = C.lstm_chain(xv, hp, cp, w["W"], w["b"])
        elif k in (C.NARY_LEAF, C.CS_LEAF):
            h, c = C.tree_leaf(xv, w["W"], w["b"])
        elif k == C.NARY_INTERNAL:
            N = len(ch) if n_fixed is None else n_fixed[t]
            st = [state(c) for c in ch[:N]]
            h, c = C.nary_internal([s[0] for s in st], [s[1] for s in st], w["W"], w["b"])
        elif k == C.GRID:
            (hl, cl), (ht, ct) = state(ch[0]), state(ch[1])
            h, c = C.grid(xv, hl, cl, ht, ct, w["W"], w["b"])
        elif k == C.CS_INTERNAL:
            st = [state(c) for c in ch if c >= 0]
            h, c = C.childsum_internal([s[0] for s in st], [s[1] for s in st],
                                       w["U_iou"], w["U_f"], w["b_iou"], w["b_f"])
        elif k == C.LAT_WORD:
            hb, cb = state(ch[0])
            h, c = C.lattice_word(xv, hb, cb, w["W"], w["b"])
        elif k == C.GRU_LEAF:
            h, c = C.gru_leaf(xv, w["W"], w["b"])
        elif k == C.GRU_INTERNAL:
            # a GRU node's state is its cell-state row (h before any rounding)
            st = [state(c)[1] for c in ch[:2]]
            h, c = C.gru_internal(st, w["W"], w["b"])
        elif k == C.LGRU_EDGE:
            # the source position's state is read from its cell-state row
            h, c = C.lgru_edge(xv, state(ch[0])[1], w["W"], w["b"])
        elif k == C.POOL_MEAN:
            h, c = C.pool_mean([state(c)[0] for c in ch if c >= 0], w["W"], w["b"])
        elif k == C.LAT_CHAR:
            hp, cp = state(ch[0])
            words = [state(c)[1] for c in ch[1:] if c >= 0]
            h, c = C.lattice_char(xv, hp, cp, words, w["W"], w["W_lx"], w["W_lc"],
                                  w["b"], w["b_l"])
        else:
            raise ValueError(f"unknown cell kind {k}")
        if bf16:
            h = round_to_bf16(h)
            c = np.asarray(c, dtype=np.float64).astype(np.float32).astype(np.float64)
        hs[v] = h
        cs[v] = c
        done[v] = True
    return hs, cs


def evaluate_workload(w, order=None):
    """Convenience wrapper reading the arrays of a workload object."""
    n_fixed = None
    if getattr(w, "n_children", None) is not None:
        n_fixed = list(w.n_children)
    return evaluate(w.kinds, w.op_type, w.child_ptr, w.child_idx, w.x_row, w.x,
                    w.weights, w.hidden, n_fixed=n_fixed, dtype=w.dtype, order=order)
