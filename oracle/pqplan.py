"""PQ-tree memory layout (Section 3.2, Algorithm 2, Appendix B), plain and slow.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Variables are the node states plus one zero pad per absent entry of a
positional operand list that has a present entry (a pad keeps the list's rows
aligned).  A batch b with rows R_b (its nodes in ascending id) has the aligned
operands O_0 = R_b and O_{1+p} = [child p of each row, or its pad] for every
positional child p whose list has a present entry and no repeated variable;
a ragged child list adds an adjacency-only set.  Position i of every aligned
operand belongs to row i.

Main (Algorithm 2):
  ConstructPQTree: every operand's variable set is reduced into a PQ tree,
    batches from last to first (consumers before producers), and in a batch
    the positional child lists, then the ragged set, then the results.  A set
    that cannot be made consecutive is skipped and its operand leaves the
    batch's aligned group: the rows of a batch may take any order, so they
    follow the group's first operand (the results when they are in it), and
    results outside the group are scattered.
  BroadcastConstraint: the structure of each operand of the group (its
    covering subtree: every P-node's leaf set and every pair of neighbouring
    Q-node children, in depth-first order) is read in positions, the union
    over the group's operands is mapped back onto every operand and reduced.
    Sweeps over the batches repeat until a sweep changes nothing.  A batch
    whose constraint fails keeps only its first operand.
  DecideNodesOrder: the operands' structures are matched by position set.
    Matching Q-nodes must read in the same or in reversed order (an equal /
    opposite relation between their directions), matching P-nodes give a
    bijection of their children; a batch whose structures do not match
    leaves the pass.  Relations are merged with a union-find that carries
    the relative order (a parity for Q-nodes, a child bijection for P-nodes,
    Appendix B); a relation that contradicts the merged ones is dropped.
  GetLeafOrder: a depth-first traversal in which each class root keeps its
    stored order and every other node takes the order its relation gives.
The frontier position of a variable is its slot minus one (slot 0 = zero row).
"""
from __future__ import annotations

from .pqtree import LEAF, PNODE, QNODE, PQTree


def variables(op_type, child_ptr, child_idx, batches, shapes):
    """Returns (n_vars, pad_of, operands, slot_ids, ragged_sets): pad_of[(b, p, v)] is
    the pad variable of row v's absent child p in batch b; operands[b] the
    aligned operand lists and slot_ids[b] their ids (0 the rows, 1 + p child
    p); ragged_sets[b] the ragged list's variables or None."""
    V = len(op_type)
    nxt = V
    pad_of = {}
    operands, ids, ragged_sets = [], [], []
    for b, rows in enumerate(batches):
        t = int(op_type[rows[0]])
        nf, rg = shapes[t][0], shapes[t][1]
        ops = [list(rows)]
        oid = [0]
        for p in range(nf):
            L = [int(child_idx[child_ptr[v] + p]) for v in rows]
            if all(c < 0 for c in L):
                continue
            vars_ = []
            for v, c in zip(rows, L):
                if c < 0:
                    pad_of[(b, p, v)] = nxt
                    c = nxt
                    nxt += 1
                vars_.append(c)
            if len(set(vars_)) == len(vars_):
                ops.append(vars_)
                oid.append(1 + p)
        operands.append(ops)
        ids.append(oid)
        rs = None
        if rg:
            rl = [int(c) for v in rows for c in child_idx[child_ptr[v] + nf:child_ptr[v + 1]] if c >= 0]
            if len(rl) >= 2 and len(set(rl)) == len(rl):
                rs = rl
        ragged_sets.append(rs)
    return nxt, pad_of, operands, ids, ragged_sets


def order_kind(tree, x):
    """A node's order is a direction (QNODE) when it is a Q-node or has two
    children (both of its orders are then each other's reversal), else a
    permutation of its children (PNODE)."""
    if tree.kind[x] == QNODE or len(tree.children[x]) == 2:
        return QNODE
    return PNODE


def _structure(tree, o):
    """Covering structure of operand o: a list of (kind, node, children) in
    depth-first pre-order, kind PNODE or QNODE, node the tree node whose order
    it reads (for a run of a Q-node's children, that Q-node), children the
    child nodes in tree order."""
    A = set(o)
    r = tree.pertinent_root(list(o))
    out = []

    def visit(x):
        if tree.kind[x] == LEAF:
            return
        out.append((order_kind(tree, x), x, list(tree.children[x])))
        for c in tree.children[x]:
            visit(c)
    if set(tree.leaves(r)) == A:
        visit(r)
    else:
        kids = [c for c in tree.children[r] if set(tree.leaves(c)) <= A]
        out.append((QNODE, r, kids))
        for c in kids:
            visit(c)
    return out


def _position_constraints(tree, o):
    pos = {x: i for i, x in enumerate(o)}
    cons = []
    for kind, _x, kids in _structure(tree, o):
        sets = [sorted(pos[l] for l in tree.leaves(c)) for c in kids]
        if kind == PNODE:
            cons.append(tuple(sorted(i for s in sets for i in s)))
        else:
            for a, b in zip(sets, sets[1:]):
                cons.append(tuple(sorted(a + b)))
    return cons


def parse_constraints(tree, ops):
    uniform, seen = [], set()
    for o in ops:
        for c in _position_constraints(tree, o):
            if c not in seen:
                seen.add(c)
                uniform.append(c)
    return [[o[i] for i in c] for o in ops for c in uniform]


class _UnionFind:
    """Union-find over tree nodes with the order relative to the parent:
    Q-nodes a direction parity, P-nodes a map from the parent's children to
    the node's children (order(x) = [sigma[c] for c in order(parent)])."""

    def __init__(self, tree):
        self.tree = tree
        self.up = {}
        self.rel = {}

    def find(self, x):
        if order_kind(self.tree, x) == QNODE:
            par = 0
            while self.up.get(x, x) != x:
                par ^= self.rel[x]
                x = self.up[x]
            return x, par
        total = {c: c for c in self.tree.children[x]}
        while self.up.get(x, x) != x:
            s = self.rel[x]
            total = {c: total[s[c]] for c in s}
            x = self.up[x]
        return x, total

    def union_q(self, a, b, rel):
        """dir(b) = dir(a) xor rel."""
        ra, pa = self.find(a)
        rb, pb = self.find(b)
        if ra == rb:
            return (pa ^ pb) == rel
        self.up[ra] = rb
        self.rel[ra] = pa ^ pb ^ rel
        return True

    def union_p(self, a, b, f):
        """order(b) = [f[c] for c in order(a)]."""
        ra, Ta = self.find(a)
        rb, Tb = self.find(b)
        if ra == rb:
            return all(f[Ta[c]] == Tb[c] for c in Ta)
        finv = {v: k for k, v in f.items()}
        Tainv = {v: k for k, v in Ta.items()}
        self.up[ra] = rb
        self.rel[ra] = {c: Tainv[finv[Tb[c]]] for c in Tb}
        return True


def _relations(tree, ops):
    """Order relations between the structures of O_0 and every other operand,
    or None when some structure does not match."""
    rels = []
    s0 = _structure(tree, ops[0])
    p0 = {x: i for i, x in enumerate(ops[0])}
    key0 = [[frozenset(p0[l] for l in tree.leaves(c)) for c in kids] for _k, _x, kids in s0]
    for o in ops[1:]:
        sj = _structure(tree, o)
        pj = {x: i for i, x in enumerate(o)}
        byset = {}
        for (kind, x, kids) in sj:
            ks = [frozenset(pj[l] for l in tree.leaves(c)) for c in kids]
            byset[frozenset().union(*ks)] = (kind, x, kids, ks)
        for (kind, x, kids), ks in zip(s0, key0):
            m = byset.get(frozenset().union(*ks))
            if m is None or m[0] != kind or set(m[3]) != set(ks):
                return None
            _k, y, ykids, yks = m
            if kind == QNODE:
                if yks == ks:
                    rels.append((QNODE, x, y, 0))
                elif yks == ks[::-1]:
                    rels.append((QNODE, x, y, 1))
                else:
                    return None
            else:
                at = {s: c for s, c in zip(yks, ykids)}
                rels.append((PNODE, x, y, {c: at[s] for c, s in zip(kids, ks)}))
    return rels


def leaf_order(tree, uf):
    out = []

    def walk(x):
        if tree.kind[x] == LEAF:
            out.append(x)
            return
        if order_kind(tree, x) == QNODE:
            _r, par = uf.find(x)
            kids = tree.children[x][::-1] if par else tree.children[x]
        else:
            r, T = uf.find(x)
            kids = [T[c] for c in tree.children[r]]
        for c in kids:
            walk(c)
    if tree.root >= 0:
        walk(tree.root)
    return out


def pq_layout(op_type, child_ptr, child_idx, batches, shapes):
    """Returns (slot_of_var, pad_of, lead, stats): slot_of_var[x] for every
    variable (nodes first, then pads), pad_of as in `variables`, lead[b] the
    operand whose memory order the rows of batch b follow (0 = the results,
    1 + p = positional child p), stats the consecutive operands after
    ConstructPQTree, the batches still aligned after BroadcastConstraint, the
    batches whose every operand stayed aligned and whose relations all merged
    (`fully_decided`), and the sweeps of BroadcastConstraint."""
    n, pad_of, operands, ids, ragged_sets = variables(op_type, child_ptr, child_idx, batches, shapes)
    tree = PQTree(n)
    B = len(batches)
    # group[b]: the operands of b taking part in alignment, as (operand index, variables)
    group = [None] * B
    for b in range(B - 1, -1, -1):
        g = []
        ops = list(enumerate(operands[b]))
        for i, o in ops[1:]:
            ok, _ = tree.reduce(o)
            if ok:
                g.append((i, o))
        if ragged_sets[b]:
            tree.reduce(ragged_sets[b])
        ok, _ = tree.reduce(operands[b][0])
        if ok:
            g.insert(0, (0, operands[b][0]))
        group[b] = g
    built = sum(len(g) for g in group)
    lead = [ids[b][group[b][0][0]] if group[b] else 0 for b in range(B)]

    def active(b):
        return len(group[b]) >= 2 and len(group[b][0][1]) >= 2
    sweeps = 0
    while True:
        sweeps += 1
        changed = False
        for b in range(B):
            if not active(b):
                continue
            for c in parse_constraints(tree, [o for _i, o in group[b]]):
                ok, ch = tree.reduce(c)
                if not ok:
                    group[b] = group[b][:1]
                    break
                changed |= ch
        if not changed:
            break
    broadcast = sum(1 for b in range(B) if active(b))
    uf = _UnionFind(tree)
    decided = []
    for b in range(B):
        if not active(b):
            continue
        rels = _relations(tree, [o for _i, o in group[b]])
        if rels is None:
            continue
        ok_all = True
        for kind, x, y, r in rels:
            ok = uf.union_q(x, y, r) if kind == QNODE else uf.union_p(x, y, r)
            ok_all &= ok
        if ok_all and len(group[b]) == len(operands[b]):
            decided.append(b)
    order = leaf_order(tree, uf)
    slot = [0] * n
    for i, x in enumerate(order):
        slot[x] = i + 1
    stats = {"batches": B, "operands_consecutive": built, "broadcast": broadcast, "decided": len(decided),
             "fully_decided": decided, "sweeps": sweeps, "variables": n}
    return slot, pad_of, lead, stats
