"""PQ tree (Booth and Lueker 1976), plain and slow: the structure ED-Batch
uses for its batching-aware memory layout (Section 3.2, Appendix B).

TEST INFRASTRUCTURE ONLY (see the package docstring).

A PQ tree over a set of leaves represents the permutations of the leaves in
which every set applied with `reduce` is consecutive.  P-nodes (at least two
children) may order their children arbitrarily; Q-nodes (at least three) keep
their children's order up to reversal.  The frontier (leaves read left to
right) is one represented permutation.

`reduce(S)` makes S consecutive.  It first classifies the pertinent subtree
(the smallest subtree holding S) bottom-up, each node EMPTY (no leaf of S),
FULL (only leaves of S) or PARTIAL, and checks that the templates apply;
only then does it restructure, so a set that cannot be made consecutive
leaves the tree as it was.  The templates, for a PARTIAL node X with empty
children E, full children F and partial children (already Q-nodes ordered
empty end first):
  P-node, not the pertinent root: no partial child -> X becomes the Q-node
    [E*, F*]; one partial child Y -> X becomes the Q-node [E*, Y's children, F*];
    more -> fail.  (E* and F* stand for the single child or a new P-node of
    the group, and are left out when the group is empty.)
  P-node, pertinent root: no partial child -> the full children move into a
    new P-node, appended after the empty ones; one partial Y -> F* is appended
    to Y's full end and X keeps [E..., Y]; two partials Y1, Y2 -> Y1 takes
    [Y1's children, F*, Y2's children reversed]; X keeps [E..., Y1]; when no
    empty child remains, the merged node replaces X.  More -> fail.
  Q-node, not the pertinent root: the children must read E... [partial] F...
    in one of the two directions (X is reversed if needed); the partial
    child's children replace it.
  Q-node, pertinent root: the children must read E... [partial] F...
    [partial] E...; the left partial child's children replace it in order,
    the right one's reversed.
A Q-node left with two children (the merged node, or the pertinent root)
becomes a P-node.  New nodes take
the next node id in creation order.
"""
from __future__ import annotations

LEAF, PNODE, QNODE = 0, 1, 2
EMPTY, FULL, PARTIAL = 0, 1, 2


class PQTree:
    def __init__(self, n):
        self.n = n
        self.kind = [LEAF] * n
        self.children = [[] for _ in range(n)]
        self.parent = [-1] * n
        self.alive = [True] * n
        if n >= 2:
            self.root = self._new(PNODE, list(range(n)))
        else:
            self.root = 0 if n == 1 else -1

    def _new(self, kind, kids):
        i = len(self.kind)
        self.kind.append(kind)
        self.children.append(list(kids))
        self.parent.append(-1)
        self.alive.append(True)
        for c in kids:
            self.parent[c] = i
        return i

    def _set_children(self, x, kids):
        self.children[x] = list(kids)
        for c in kids:
            self.parent[c] = x

    def _replace(self, old, new):
        """Puts `new` where `old` is (in old's parent, or as the root)."""
        p = self.parent[old]
        self.parent[new] = p
        if p < 0:
            self.root = new
        else:
            self.children[p] = [new if c == old else c for c in self.children[p]]
        self.alive[old] = False

    def frontier(self):
        out = []

        def walk(x):
            if self.kind[x] == LEAF:
                out.append(x)
            for c in self.children[x]:
                walk(c)
        if self.root >= 0:
            walk(self.root)
        return out

    def leaves(self, x):
        if self.kind[x] == LEAF:
            return [x]
        out = []
        for c in self.children[x]:
            out += self.leaves(c)
        return out

    def count_frontiers(self):
        """Number of permutations the tree represents: k! per P-node with k
        children, 2 per Q-node."""
        total = 1

        def walk(x):
            nonlocal total
            if self.kind[x] == PNODE:
                for i in range(2, len(self.children[x]) + 1):
                    total *= i
            elif self.kind[x] == QNODE:
                total *= 2
            for c in self.children[x]:
                walk(c)
        if self.root >= 0:
            walk(self.root)
        return total

    # -- reduce ---------------------------------------------------------------

    def pertinent_root(self, S):
        """Deepest node whose subtree holds every leaf of S."""
        target = set(S)
        x = S[0]
        while not target <= set(self.leaves(x)):
            x = self.parent[x]
        return x

    def _status(self, x, S):
        """Status of every node in x's subtree, bottom-up (dict)."""
        st = {}

        def walk(y):
            if self.kind[y] == LEAF:
                st[y] = FULL if y in S else EMPTY
                return st[y]
            ss = [walk(c) for c in self.children[y]]
            if all(s == FULL for s in ss):
                st[y] = FULL
            elif all(s == EMPTY for s in ss):
                st[y] = EMPTY
            else:
                st[y] = PARTIAL
            return st[y]
        walk(x)
        return st

    @staticmethod
    def _q_pattern_ok(seq, root):
        """Q-node child statuses read left to right."""
        i, n = 0, len(seq)
        if root:
            while i < n and seq[i] == EMPTY:
                i += 1
            if i < n and seq[i] == PARTIAL:
                i += 1
            while i < n and seq[i] == FULL:
                i += 1
            if i < n and seq[i] == PARTIAL:
                i += 1
            while i < n and seq[i] == EMPTY:
                i += 1
            return i == n
        while i < n and seq[i] == EMPTY:
            i += 1
        if i < n and seq[i] == PARTIAL:
            i += 1
        while i < n and seq[i] == FULL:
            i += 1
        return i == n

    def _check(self, x, st, is_root):
        if st[x] != PARTIAL:
            return True
        kids = self.children[x]
        if not all(self._check(c, st, False) for c in kids if st[c] == PARTIAL):
            return False
        seq = [st[c] for c in kids]
        npart = seq.count(PARTIAL)
        if self.kind[x] == PNODE:
            return npart <= (2 if is_root else 1)
        if is_root:
            return self._q_pattern_ok(seq, True)
        return self._q_pattern_ok(seq, False) or self._q_pattern_ok(seq[::-1], False)

    def implied(self, S):
        """True when S is consecutive in every permutation the tree represents."""
        if len(S) < 2:
            return True
        x = self.pertinent_root(S)
        st = self._status(x, set(S))
        if st[x] == FULL:
            return True
        if self.kind[x] != QNODE:
            return False
        seq = [st[c] for c in self.children[x]]
        if PARTIAL in seq:
            return False
        idx = [i for i, s in enumerate(seq) if s == FULL]
        return idx == list(range(idx[0], idx[-1] + 1))

    def _group(self, kids):
        if not kids:
            return []
        if len(kids) == 1:
            return [kids[0]]
        return [self._new(PNODE, kids)]

    def _apply(self, x, st, is_root):
        """Restructures x's subtree; returns the node standing where x was."""
        if st[x] != PARTIAL:
            return x
        for c in list(self.children[x]):
            if st[c] == PARTIAL:
                self._apply(c, st, False)
        kids = self.children[x]
        E = [c for c in kids if st[c] == EMPTY]
        F = [c for c in kids if st[c] == FULL]
        Pa = [c for c in kids if st[c] == PARTIAL]
        if self.kind[x] == PNODE and not is_root:
            gE = self._group(E)
            gF = self._group(F)
            mid = []
            if Pa:
                y = Pa[0]
                mid = list(self.children[y])
                self.alive[y] = False
            self.kind[x] = QNODE
            self._set_children(x, gE + mid + gF)
            return x
        if self.kind[x] == PNODE:
            if not Pa:
                if len(F) >= 2:
                    self._set_children(x, E + self._group(F))
                return x
            y = Pa[0]
            if len(Pa) == 2:
                y2 = Pa[1]
                gF = self._group(F)
                self._set_children(y, self.children[y] + gF + self.children[y2][::-1])
                self.alive[y2] = False
            else:
                self._set_children(y, self.children[y] + self._group(F))
                if len(self.children[y]) == 2:
                    self.kind[y] = PNODE
            if E:
                self._set_children(x, E + [y])
                return x
            self._replace(x, y)
            return y
        # Q-node
        if not is_root:
            seq = [st[c] for c in kids]
            if not self._q_pattern_ok(seq, False):
                kids = kids[::-1]
            out = []
            for c in kids:
                if st[c] == PARTIAL:
                    out += self.children[c]
                    self.alive[c] = False
                else:
                    out.append(c)
            self._set_children(x, out)
            return x
        out = []
        seen_full = False
        for c in kids:
            if st[c] == PARTIAL:
                # before the full block: empty end first; after it: reversed
                out += self.children[c] if not seen_full else self.children[c][::-1]
                self.alive[c] = False
                seen_full = True
            else:
                if st[c] == FULL:
                    seen_full = True
                out.append(c)
        self._set_children(x, out)
        return x

    def reduce(self, S):
        """Makes the leaves of S consecutive.  Returns (ok, changed): ok False
        (tree unchanged) when no represented permutation has S consecutive;
        changed False when S already was consecutive in all of them."""
        S = list(S)
        if len(S) < 2:
            return True, False
        if self.implied(S):
            return True, False
        x = self.pertinent_root(S)
        st = self._status(x, set(S))
        if not self._check(x, st, True):
            return False, False
        top = self._apply(x, st, True)
        if self.kind[top] == QNODE and len(self.children[top]) == 2:
            self.kind[top] = PNODE
        return True, True
