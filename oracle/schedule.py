"""Batching schedules of a typed dataflow graph (Section 2 and Appendix A).

Algorithm 1 (FSM-based dynamic batching): while nodes remain, encode the
graph state S = E(G), pick the next type t = pi(S), and execute as one batch
*every* frontier node of type t; then update the frontier.  The frontier is
the set of unexecuted nodes whose present children have all executed.

Policies
  table   pi is a lookup table keyed by the state encoding (the learned FSM's
          inference form, Section 2.3: argmax_a Q(S, a) stored per state)
  agenda  the type with minimal average topological depth (DyNet's heuristic,
          Section 2.1), the average taken over all unexecuted nodes of the type
  depth   batches are the groups of equal (topological depth, type)
          (TensorFlow Fold's heuristic, Section 2.1)
  sufficient  the type maximizing the second term of Eq. 1, the frontier
          ratio of Lemma 1 (the sufficient-condition-guided heuristic of the
          batch-count study, Section 5); ties to the lowest type id

State encodings (Section 2.3): E_base = the set of frontier types, E_max =
E_base plus the most common frontier type, E_sort = the frontier types sorted
by their frontier count.  Ties everywhere go to the lowest type id; nodes of a
batch are listed in ascending node id; a table miss, or a table action that is
not on the frontier, falls back to the most common frontier type.
"""
from __future__ import annotations

from collections import deque

import numpy as np

POLICY_TABLE = 0
POLICY_AGENDA = 1
POLICY_DEPTH = 2
POLICY_SUFFICIENT = 3

ENC_SORT = 0
ENC_BASE = 1
ENC_MAX = 2


def _consumers(n, child_ptr, child_idx):
    pending = np.zeros(n, dtype=np.int64)
    cons = [[] for _ in range(n)]
    for v in range(n):
        for c in child_idx[child_ptr[v]:child_ptr[v + 1]]:
            if c >= 0:
                pending[v] += 1
                cons[int(c)].append(v)
    return pending, cons


def topo_depth(n, child_ptr, child_idx):
    """depth(v) = 0 without present children, else 1 + max depth(child)
    (the input operation has depth 0, Section 2.1).  Node ids need not be
    topologically sorted."""
    pending, cons = _consumers(n, child_ptr, child_idx)
    depth = np.zeros(n, dtype=np.int64)
    q = deque(v for v in range(n) if pending[v] == 0)
    seen = 0
    while q:
        v = q.popleft()
        seen += 1
        for p in cons[v]:
            depth[p] = max(depth[p], depth[v] + 1)
            pending[p] -= 1
            if pending[p] == 0:
                q.append(p)
    if seen != n:
        raise ValueError("graph has a cycle")
    return depth


def encode_state(counts, encoding=ENC_SORT):
    """State key of a frontier given per-type frontier counts (Section 2.3)."""
    present = [t for t in range(len(counts)) if counts[t] > 0]
    if encoding == ENC_SORT:
        return tuple(sorted(present, key=lambda t: (-counts[t], t)))
    if encoding == ENC_BASE:
        return tuple(present)
    if encoding == ENC_MAX:
        return tuple(present) + (majority_type(counts),)
    raise ValueError("unknown encoding")


def majority_type(counts):
    best = -1
    for t in range(len(counts)):
        if counts[t] > 0 and (best < 0 or counts[t] > counts[best]):
            best = t
    return best


def parse_table(flat):
    """Flat int32 table: [n_entries, {key_len, key[0..key_len), action} x n_entries]."""
    flat = [int(v) for v in flat]
    if not flat:
        return {}
    n = flat[0]
    pos = 1
    table = {}
    for _ in range(n):
        if pos >= len(flat):
            raise ValueError("malformed table")
        kl = flat[pos]
        if kl < 0 or pos + 1 + kl >= len(flat):
            raise ValueError("malformed table")
        key = tuple(flat[pos + 1:pos + 1 + kl])
        table[key] = flat[pos + 1 + kl]
        pos += 2 + kl
    if pos != len(flat):
        raise ValueError("malformed table")
    return table


def flatten_table(table):
    out = [len(table)]
    for key, action in table.items():
        out += [len(key)] + list(key) + [action]
    return out


def schedule(op_type, child_ptr, child_idx, n_types, policy=POLICY_TABLE,
             table=None, encoding=ENC_SORT):
    """Run Algorithm 1 (or the depth grouping); return (batches, batch_types),
    batches being lists of node ids in ascending order."""
    n = int(len(op_type))
    op_type = [int(t) for t in op_type]
    if policy == POLICY_DEPTH:
        depth = topo_depth(n, child_ptr, child_idx)
        groups = {}
        for v in range(n):
            groups.setdefault((int(depth[v]), op_type[v]), []).append(v)
        keys = sorted(groups)
        return [groups[k] for k in keys], [k[1] for k in keys]

    table = table or {}
    pending, cons = _consumers(n, child_ptr, child_idx)
    ready = [set() for _ in range(n_types)]
    for v in range(n):
        if pending[v] == 0:
            ready[op_type[v]].add(v)
    if policy == POLICY_AGENDA:
        depth = topo_depth(n, child_ptr, child_idx)
        dsum = [0] * n_types
        dcnt = [0] * n_types
        for v in range(n):
            dsum[op_type[v]] += int(depth[v])
            dcnt[op_type[v]] += 1

    batches, btypes = [], []
    remaining = n
    while remaining:
        counts = [len(r) for r in ready]
        if policy == POLICY_TABLE:
            key = encode_state(counts, encoding)
            t = table.get(key, -1)
            if t < 0 or t >= n_types or counts[t] == 0:
                t = majority_type(counts)
        elif policy == POLICY_SUFFICIENT:
            executed = [False] * n
            for b in batches:
                for v in b:
                    executed[v] = True
            t, best = -1, None
            for a in range(n_types):
                if counts[a] == 0:
                    continue
                num, den = frontier_ratio(op_type, child_ptr, child_idx, executed, a)
                # ratios compared exactly: num_a / den_a > num_t / den_t
                if t < 0 or num * best[1] > best[0] * den:
                    t, best = a, (num, den)
        elif policy == POLICY_AGENDA:
            t = -1
            for a in range(n_types):
                if counts[a] == 0:
                    continue
                # mean depth S_a / n_a compared exactly: S_a n_t < S_t n_a
                if t < 0 or dsum[a] * dcnt[t] < dsum[t] * dcnt[a]:
                    t = a
        else:
            raise ValueError("unknown policy")
        batch = sorted(ready[t])
        ready[t] = set()
        for v in batch:
            if policy == POLICY_AGENDA:
                dsum[t] -= int(depth[v])
                dcnt[t] -= 1
            for p in cons[v]:
                pending[p] -= 1
                if pending[p] == 0:
                    ready[op_type[p]].add(p)
        remaining -= len(batch)
        batches.append(batch)
        btypes.append(t)
    return batches, btypes


def lower_bound(op_type, child_ptr, child_idx, n_types):
    """Appendix A.3: |Batching*(G)| >= sum_t Depth(G_t), Depth(G_t) being the
    longest path, counted in nodes, of the subgraph induced on type-t nodes
    (direct edges between type-t nodes only)."""
    n = int(len(op_type))
    total = 0
    for t in range(n_types):
        nodes = [v for v in range(n) if int(op_type[v]) == t]
        if not nodes:
            continue
        ptr = [0]
        idx = []
        pos = {v: i for i, v in enumerate(nodes)}
        for v in nodes:
            kids = [pos[int(c)] for c in child_idx[child_ptr[v]:child_ptr[v + 1]]
                    if c >= 0 and int(op_type[int(c)]) == t]
            idx += kids
            ptr.append(len(idx))
        d = topo_depth(len(nodes), np.array(ptr), np.array(idx, dtype=np.int64))
        total += int(d.max()) + 1
    return total


def frontier_ratio(op_type, child_ptr, child_idx, executed, a):
    """Second term of Eq. 1 for type a, read as |Frontier_a(G_t)| / |Frontier(G^a_t)|
    (a value in (0, 1]; Lemma 1's sufficient condition is ratio == 1).

    Frontier_a(G_t): unexecuted type-a nodes whose present children have all
    executed.  Frontier(G^a_t): unexecuted type-a nodes none of whose present
    children is an unexecuted type-a node (the frontier of the subgraph
    induced on type a).  Returns (numerator, denominator)."""
    n = int(len(op_type))
    num = den = 0
    for v in range(n):
        if executed[v] or int(op_type[v]) != a:
            continue
        kids = [int(c) for c in child_idx[child_ptr[v]:child_ptr[v + 1]] if c >= 0]
        if all(executed[c] for c in kids):
            num += 1
        if all(executed[c] or int(op_type[c]) != a for c in kids):
            den += 1
    return num, den


def optimal_batch_count(op_type, child_ptr, child_idx, n_types):
    """Brute-force minimum number of batches (Appendix A.1's Batching problem):
    breadth-first search over executed sets, each step executing all frontier
    nodes of one type.  Exponential; for graphs of at most ~16 nodes."""
    n = int(len(op_type))
    kids = [[int(c) for c in child_idx[child_ptr[v]:child_ptr[v + 1]] if c >= 0]
            for v in range(n)]
    kid_mask = [sum(1 << c for c in kids[v]) for v in range(n)]
    full = (1 << n) - 1
    dist = {0: 0}
    q = deque([0])
    while q:
        s = q.popleft()
        if s == full:
            return dist[s]
        for t in range(n_types):
            add = 0
            for v in range(n):
                if not (s >> v) & 1 and int(op_type[v]) == t and (kid_mask[v] & s) == kid_mask[v]:
                    add |= 1 << v
            if add:
                ns = s | add
                if ns not in dist:
                    dist[ns] = dist[s] + 1
                    q.append(ns)
    raise ValueError("unreachable")


def check_schedule(op_type, child_ptr, child_idx, batches, btypes, maximal=True):
    """Invariants: every node exactly once; all present children in earlier
    batches; each batch homogeneous in type; and (Algorithm 1's line that
    takes every frontier node of the chosen type) each batch maximal."""
    n = int(len(op_type))
    when = np.full(n, -1, dtype=np.int64)
    for b, batch in enumerate(batches):
        for v in batch:
            if when[v] >= 0:
                raise AssertionError(f"node {v} scheduled twice")
            when[v] = b
    if (when < 0).any():
        raise AssertionError("node never scheduled")
    for b, batch in enumerate(batches):
        if list(batch) != sorted(batch):
            raise AssertionError("batch not in ascending node order")
        for v in batch:
            if int(op_type[v]) != btypes[b]:
                raise AssertionError("inhomogeneous batch")
            for c in child_idx[child_ptr[v]:child_ptr[v + 1]]:
                if c >= 0 and when[int(c)] >= b:
                    raise AssertionError(f"node {v} runs before its child {int(c)}")
    if maximal:
        for b, batch in enumerate(batches):
            t = btypes[b]
            members = set(batch)
            for v in range(n):
                if when[v] > b and int(op_type[v]) == t and v not in members:
                    kids = [int(c) for c in child_idx[child_ptr[v]:child_ptr[v + 1]] if c >= 0]
                    if all(when[c] < b for c in kids):
                        raise AssertionError(f"batch {b} misses ready node {v}")
    return True
