"""Oracle evaluation of a whole workload, instance by instance.

Instances (trees, chains, lattices, grids) are independent graphs, so the
oracle evaluates each connected component on its own (`oracle.evaluate`
unchanged, node at a time) and the results are put back in node order; a
selection of instances costs only their own nodes.  Optional worker threads
spread independent oracle calls; nothing of the oracle's arithmetic changes.
Test infrastructure: the GPU tests call it for full-size workloads (the
largest, 52k child-sum nodes, takes about half a minute on one core).
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

from oracle.evaluate import evaluate


def components(w):
    """Instance id (a representative node) of every node: connected
    components over the present child edges."""
    parent = np.arange(w.n_nodes)

    def find(a):
        while parent[a] != a:
            parent[a] = parent[parent[a]]
            a = parent[a]
        return a
    for v in range(w.n_nodes):
        for c in w.children(v):
            if c >= 0:
                ra, rb = find(v), find(int(c))
                if ra != rb:
                    parent[ra] = rb
    return np.array([find(v) for v in range(w.n_nodes)])


def subgraph(w, nodes):
    """The graph arrays restricted to `nodes` (closed under children), ids
    remapped in ascending node order."""
    nodes = np.sort(nodes)
    remap = {int(v): i for i, v in enumerate(nodes)}
    ptr = [0]
    idx = []
    for v in nodes:
        for c in w.children(int(v)):
            idx.append(remap[int(c)] if c >= 0 else -1)
        ptr.append(len(idx))
    return dict(op_type=w.op_type[nodes], child_ptr=np.array(ptr, dtype=np.int64),
                child_idx=np.array(idx, dtype=np.int32), x_row=w.x_row[nodes])


def evaluate_by_instance(w, workers=None, nodes_of=None):
    """(h, c) of every node, float64 [V, H], node order.  `nodes_of`
    restricts the evaluation to the listed instance ids (the others stay 0)."""
    from threadpoolctl import threadpool_limits
    comp = components(w)
    roots = np.unique(comp) if nodes_of is None else np.asarray(sorted(nodes_of))
    groups = [np.nonzero(comp == r)[0] for r in roots]
    hs = np.zeros((w.n_nodes, w.hidden))
    cs = np.zeros((w.n_nodes, w.hidden))

    # the weights as float64 once (exact: every float32 value is a float64
    # value), instead of a conversion of each matrix at every node
    w64 = [{k: np.asarray(v, dtype=np.float64) for k, v in d.items()} for d in w.weights]

    def one(nodes):
        sg = subgraph(w, nodes)
        return nodes, evaluate(w.kinds, sg["op_type"], sg["child_ptr"], sg["child_idx"], sg["x_row"], w.x,
                               w64, w.hidden, n_fixed=w.n_children, dtype=w.dtype)

    if workers is None:
        # the per-node work is mostly interpreter time, which threads do not
        # overlap: one worker unless asked
        workers = 1
    # largest instances first, so that the pool does not end on a long one
    groups.sort(key=len, reverse=True)
    with threadpool_limits(limits=1), ThreadPoolExecutor(max_workers=workers) as ex:
        for nodes, (h, c) in ex.map(one, groups):
            hs[nodes] = h
            cs[nodes] = c
    return hs, cs
