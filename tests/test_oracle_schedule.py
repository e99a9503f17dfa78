"""Pins of the oracle's schedules: the worked example of Section 2.1 / 2.3
(Figure 1, reconstructed; golden fixture), schedule invariants, the lower
bound of Appendix A.3, brute-force optima on tiny graphs and the reduction
from shortest common supersequence (Appendix A.1).  CPU only."""
import itertools
import json
import os
from collections import deque

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

from oracle import schedule as S
from paper_2302_03851_amd import workloads as WL


def csr(children):
    ptr = np.zeros(len(children) + 1, dtype=np.int64)
    for v, ch in enumerate(children):
        ptr[v + 1] = ptr[v] + len(ch)
    idx = np.array([c for ch in children for c in ch], dtype=np.int32)
    return ptr, idx


@pytest.fixture(scope="module")
def fig1(golden_dir):
    with open(os.path.join(golden_dir, "fig1_tree.json")) as f:
        g = json.load(f)
    types = g["types"]
    op = np.array([types[n["type"]] for n in g["nodes"]], dtype=np.int32)
    ptr, idx = csr([n["children"] for n in g["nodes"]])
    return g, op, ptr, idx, len(types)


def test_fig1_depth_policy(fig1):
    g, op, ptr, idx, T = fig1
    batches, bt = S.schedule(op, ptr, idx, T, S.POLICY_DEPTH)
    S.check_schedule(op, ptr, idx, batches, bt, maximal=False)
    O = g["types"]["O"]
    assert sum(1 for t in bt if t == O) == g["printed"]["depth_policy_O_batches"]
    assert len(batches) == g["derived"]["depth_batches"]


def test_fig1_agenda_average_depths_and_choice(fig1):
    g, op, ptr, idx, T = fig1
    depth = S.topo_depth(len(op), ptr, idx)
    for name, key in (("O", "agenda_mean_depth_O"), ("I", "agenda_mean_depth_I")):
        t = g["types"][name]
        d = [int(depth[v]) for v in range(len(op)) if op[v] == t]
        num, den = g["printed"][key]
        assert sum(d) * den == num * len(d)
    batches, bt = S.schedule(op, ptr, idx, T, S.POLICY_AGENDA)
    S.check_schedule(op, ptr, idx, batches, bt)
    # after the inputs, agenda picks O (13/7 < 2): the extra batch of Section 2.1
    assert bt[1] == g["types"]["O"]
    assert len(batches) == g["derived"]["agenda_batches"]


def test_fig1_fsm_table_policy(fig1):
    g, op, ptr, idx, T = fig1
    I, O = g["types"]["I"], g["types"]["O"]
    table = {(O, I): I, (I, O): I}
    batches, bt = S.schedule(op, ptr, idx, T, S.POLICY_TABLE, table=table)
    S.check_schedule(op, ptr, idx, batches, bt)
    assert sum(1 for t in bt if t == O) == 1            # all O nodes in one batch
    assert len(batches) == g["derived"]["table_batches"]
    assert S.lower_bound(op, ptr, idx, T) == g["derived"]["lower_bound"]
    assert S.optimal_batch_count(op, ptr, idx, T) == g["derived"]["optimal"]


def test_fig1_reward_ratio_at_iteration_2(fig1):
    g, op, ptr, idx, T = fig1
    executed = np.zeros(len(op), dtype=bool)
    executed[[0, 1, 2, 3, 4]] = True       # the inputs and I1
    for name in ("O", "I"):
        assert list(S.frontier_ratio(op, ptr, idx, executed, g["types"][name])) == \
            g["printed"]["ratio_after_In_and_I1"][name]


def test_encodings():
    counts = [3, 0, 5, 5]
    assert S.encode_state(counts, S.ENC_SORT) == (2, 3, 0)
    assert S.encode_state(counts, S.ENC_BASE) == (0, 2, 3)
    assert S.encode_state(counts, S.ENC_MAX) == (0, 2, 3, 2)
    t = {(2, 3, 0): 0, (1,): 1}
    assert S.parse_table(S.flatten_table(t)) == t
    with pytest.raises(ValueError):
        S.parse_table([2, 1, 0, 0])


@pytest.mark.parametrize("L", [1, 2, 7, 20])
def test_chain_batch_count_is_length(L):
    op = np.zeros(L, dtype=np.int32)
    ptr, idx = csr([[]] + [[i] for i in range(L - 1)])
    for pol in (S.POLICY_TABLE, S.POLICY_AGENDA, S.POLICY_DEPTH):
        batches, bt = S.schedule(op, ptr, idx, 1, pol)
        assert len(batches) == L


def _small(k):
    return WL.make_config(k, instances={1: 8, 2: 6, 3: 4, 4: 2, 5: 3}[k])


@pytest.mark.parametrize("k", [1, 2, 3, 4, 5])
@pytest.mark.parametrize("pol", [S.POLICY_TABLE, S.POLICY_AGENDA, S.POLICY_DEPTH])
def test_invariants_on_configs(k, pol):
    w = _small(k)
    batches, bt = S.schedule(w.op_type, w.child_ptr, w.child_idx, w.n_types, pol)
    S.check_schedule(w.op_type, w.child_ptr, w.child_idx, batches, bt, maximal=pol != S.POLICY_DEPTH)
    assert len(batches) >= S.lower_bound(w.op_type, w.child_ptr, w.child_idx, w.n_types)


@pytest.mark.parametrize("k", [2, 5])
def test_tree_batch_count_is_height_and_bound(k):
    w = _small(k)
    batches, _ = S.schedule(w.op_type, w.child_ptr, w.child_idx, w.n_types)
    depth = S.topo_depth(w.n_nodes, w.child_ptr, w.child_idx)
    assert len(batches) == int(depth.max()) + 1
    assert len(batches) == S.lower_bound(w.op_type, w.child_ptr, w.child_idx, w.n_types)


def test_grid_batch_count_is_antidiagonals():
    w = _small(4)
    batches, _ = S.schedule(w.op_type, w.child_ptr, w.child_idx, w.n_types)
    assert len(batches) == 31
    assert max(len(b) for b in batches) == 16 * w.instances


def test_lattice_table_beats_heuristics():
    w = WL.make_config(3)
    table = {(0,): 0, (1,): 1, (0, 1): 0, (1, 0): 1}
    n_tab = len(S.schedule(w.op_type, w.child_ptr, w.child_idx, 2, S.POLICY_TABLE, table)[0])
    n_ag = len(S.schedule(w.op_type, w.child_ptr, w.child_idx, 2, S.POLICY_AGENDA)[0])
    n_dp = len(S.schedule(w.op_type, w.child_ptr, w.child_idx, 2, S.POLICY_DEPTH)[0])
    lb = S.lower_bound(w.op_type, w.child_ptr, w.child_idx, 2)
    assert lb <= n_tab < n_ag < n_dp
    # the 4 tables of the two-type E_sort state space
    counts = []
    for a, b in itertools.product([0, 1], repeat=2):
        t = {(0,): 0, (1,): 1, (0, 1): a, (1, 0): b}
        counts.append(len(S.schedule(w.op_type, w.child_ptr, w.child_idx, 2, S.POLICY_TABLE, t)[0]))
    assert n_tab == min(counts)


@st.composite
def small_dags(draw):
    n = draw(st.integers(1, 11))
    T = draw(st.integers(1, 3))
    op = [draw(st.integers(0, T - 1)) for _ in range(n)]
    children = []
    for v in range(n):
        kids = draw(st.lists(st.integers(0, v - 1), max_size=3, unique=True)) if v else []
        children.append(kids)
    return np.array(op, dtype=np.int32), children, T


@settings(max_examples=60, deadline=None)
@given(small_dags())
def test_bruteforce_optimum_bounds_policies(g):
    op, children, T = g
    ptr, idx = csr(children)
    opt = S.optimal_batch_count(op, ptr, idx, T)
    assert S.lower_bound(op, ptr, idx, T) <= opt
    for pol in (S.POLICY_TABLE, S.POLICY_AGENDA, S.POLICY_DEPTH):
        batches, bt = S.schedule(op, ptr, idx, T, pol)
        S.check_schedule(op, ptr, idx, batches, bt, maximal=pol != S.POLICY_DEPTH)
        assert len(batches) >= opt


def _scs_length(strings):
    """Shortest common supersequence by BFS over position tuples."""
    start = tuple(0 for _ in strings)
    goal = tuple(len(s) for s in strings)
    dist = {start: 0}
    q = deque([start])
    alphabet = sorted(set(c for s in strings for c in s))
    while q:
        pos = q.popleft()
        if pos == goal:
            return dist[pos]
        for a in alphabet:
            nxt = tuple(p + (p < len(s) and s[p] == a) for p, s in zip(pos, strings))
            if nxt != pos and nxt not in dist:
                dist[nxt] = dist[pos] + 1
                q.append(nxt)


@settings(max_examples=40, deadline=None)
@given(st.lists(st.lists(st.integers(0, 2), min_size=1, max_size=4), min_size=1, max_size=3))
def test_independent_chains_optimum_is_scs(strings):
    """Appendix A.1: on independent chains the optimal batch sequence is a
    shortest common supersequence of the chains' type strings."""
    op, children = [], []
    for s in strings:
        prev = -1
        for c in s:
            op.append(c)
            children.append([prev] if prev >= 0 else [])
            prev = len(op) - 1
    ptr, idx = csr(children)
    assert S.optimal_batch_count(np.array(op), ptr, idx, 3) == _scs_length(strings)


def test_absent_children_are_ignored():
    op = np.array([0, 0, 1], dtype=np.int32)
    ptr, idx = csr([[-1], [0], [-1, 1]])
    batches, bt = S.schedule(op, ptr, idx, 2)
    assert batches == [[0], [1], [2]]
