"""Pins of the oracle's policy learner and sufficient-condition policy
(Section 2.3, Lemma 1, Appendix A): the published SplitMix64 outputs, Q values
derived by hand for one episode, the reward of the worked example, Lemma 1 by
brute force on tiny graphs, and learned schedules against brute-force optima
and against every possible E_sort table.  CPU only."""
import itertools
import json
import os

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

from oracle import learn as OL
from oracle import schedule as S
from paper_2302_03851_amd import workloads as WL


def csr(children):
    ptr = np.zeros(len(children) + 1, dtype=np.int64)
    for v, ch in enumerate(children):
        ptr[v + 1] = ptr[v] + len(ch)
    return ptr, np.array([c for ch in children for c in ch], dtype=np.int32)


@pytest.fixture(scope="module")
def fig1(golden_dir):
    with open(os.path.join(golden_dir, "fig1_tree.json")) as f:
        g = json.load(f)
    op = np.array([g["types"][n["type"]] for n in g["nodes"]], dtype=np.int32)
    ptr, idx = csr([n["children"] for n in g["nodes"]])
    return g, op, ptr, idx, len(g["types"])


def test_splitmix64_published_outputs():
    # Outputs of the reference SplitMix64 (Vigna's splitmix64.c, the generator
    # of Steele, Lea and Flood 2014) for seeds 0 and 1234567.
    assert [OL.splitmix64(0, k) for k in range(3)] == [
        0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4, 0x06C45D188009454F]
    assert [OL.splitmix64(1234567, k) for k in range(5)] == [
        6457827717110365317, 3203168211198807973, 9817491932198370423,
        4593380528125082431, 16408922859458223821]


def _chain(L):
    return np.zeros(L, dtype=np.int32), *csr([[]] + [[v - 1] for v in range(1, L)])


def test_one_episode_q_values_by_hand():
    # A chain of 3 nodes of one type: one state (0,), one action, and every
    # step has ratio 1/1, so r = -1 + alpha = -0.5 (alpha = 0.5).
    op, ptr, idx = _chain(3)
    # N = 2, lr = 0.5, gamma = 1:
    #   after step 1: tau 0, target r0 + r1 + max Q(S2) = -1    -> Q = -0.5
    #   episode end:  tau 1, target r1 + r2 = -1 (no bootstrap) -> Q = -0.75
    #                 tau 2, target r2 = -0.5                   -> Q = -0.625
    _, _, Q = OL.learn(op, ptr, idx, 1, trials=1, check_every=1, n_step=2, alpha=0.5,
                       epsilon=0.0, lr=0.5, gamma=1.0)
    assert Q == {((0,), 0): -0.625}
    # N = 1, lr = 0.5, gamma = 0.5:
    #   tau 0: target -0.5 + 0.5 * 0       = -0.5    -> Q = -0.25
    #   tau 1: target -0.5 + 0.5 * (-0.25) = -0.625  -> Q = -0.4375
    #   tau 2: target -0.5 (episode end)             -> Q = -0.46875
    _, _, Q = OL.learn(op, ptr, idx, 1, trials=1, check_every=1, n_step=1, alpha=0.5,
                       epsilon=0.0, lr=0.5, gamma=0.5)
    assert Q == {((0,), 0): -0.46875}


def test_reward_of_the_worked_example(fig1):
    # Section 2.3: after the inputs and the first I node the ratio term is
    # 5/7 for O and 1/1 for I, so I earns the larger reward.
    g, op, ptr, idx, T = fig1
    ep = OL._Episode(op, ptr, idx, T)
    ep.execute(g["types"]["In"])
    ep.execute(g["types"]["I"])
    assert OL.reward(ep, g["types"]["O"], 0.5) == -1.0 + 0.5 * (5 / 7)
    assert OL.reward(ep, g["types"]["I"], 0.5) == -0.5


def test_learned_policy_on_the_worked_example(fig1):
    g, op, ptr, idx, T = fig1
    table, stats, _ = OL.learn(op, ptr, idx, T)
    batches, bt = S.schedule(op, ptr, idx, T, S.POLICY_TABLE, table=table)
    S.check_schedule(op, ptr, idx, batches, bt)
    assert len(batches) == stats["batches"] == S.optimal_batch_count(op, ptr, idx, T) == 6
    assert sum(1 for t in bt if t == g["types"]["O"]) == 1     # Figure 2's FSM
    assert stats["trials"] == 50                               # stops at the first check


def test_sufficient_policy_on_the_worked_example(fig1):
    g, op, ptr, idx, T = fig1
    batches, bt = S.schedule(op, ptr, idx, T, S.POLICY_SUFFICIENT)
    S.check_schedule(op, ptr, idx, batches, bt)
    assert len(batches) == 6
    assert bt[1] == g["types"]["I"]


def test_single_type_chain_learns_its_length():
    op, ptr, idx = _chain(7)
    table, stats, _ = OL.learn(op, ptr, idx, 1)
    assert table == {(0,): 0}
    assert stats == {"trials": 50, "batches": 7, "lower_bound": 7, "states": 1}


@st.composite
def tiny_graphs(draw):
    n = draw(st.integers(1, 11))
    T = draw(st.integers(1, 3))
    op, children = [], []
    for v in range(n):
        op.append(draw(st.integers(0, T - 1)))
        k = draw(st.integers(0, min(2, v)))
        children.append(sorted(set(draw(st.lists(st.integers(0, v - 1), min_size=k, max_size=k)))) if v else [])
    return np.array(op, dtype=np.int32), children, T


def _opt_from(op, kids, T, executed):
    """Fewest batches to finish from an executed set (breadth-first search)."""
    n = len(op)
    full = (1 << n) - 1
    start = sum(1 << v for v in range(n) if executed[v])
    dist, frontier = {start: 0}, [start]
    while frontier:
        nxt = []
        for s in frontier:
            if s == full:
                return dist[s]
            for t in range(T):
                add = sum(1 << v for v in range(n) if not (s >> v) & 1 and op[v] == t
                          and all((s >> c) & 1 for c in kids[v]))
                if add and (s | add) not in dist:
                    dist[s | add] = dist[s] + 1
                    nxt.append(s | add)
        frontier = nxt
    raise AssertionError("unreachable")


@settings(max_examples=120, deadline=None)
@given(tiny_graphs(), st.integers(0, 3))
def test_lemma1_by_brute_force(g, prefix):
    # Lemma 1: if |Frontier_a(G_t)| / |Frontier(G^a_t)| = 1 for a frontier type a,
    # some shortest batching sequence from G_t starts with a.  Checked at the
    # state reached after up to `prefix` majority-type batches.
    op, children, T = g
    ptr, idx = csr(children)
    ep = OL._Episode(op, ptr, idx, T)
    for _ in range(prefix):
        if ep.left == 0:
            break
        ep.execute(S.majority_type(ep.counts()))
    if ep.left == 0:
        return
    best = _opt_from(op, children, T, ep.executed)
    for a in range(T):
        if ep.counts()[a] == 0:
            continue
        num, den = S.frontier_ratio(op, ptr, idx, ep.executed, a)
        assert 1 <= num <= den
        if num == den:
            trial = OL._Episode(op, ptr, idx, T)
            for _ in range(prefix):
                if trial.left == 0:
                    break
                trial.execute(S.majority_type(trial.counts()))
            trial.execute(a)
            assert 1 + _opt_from(op, children, T, trial.executed) == best


@settings(max_examples=40, deadline=None)
@given(tiny_graphs(), st.sampled_from([S.ENC_SORT, S.ENC_BASE, S.ENC_MAX]))
def test_learned_schedule_valid_and_bounded(g, enc):
    op, children, T = g
    ptr, idx = csr(children)
    table, stats, _ = OL.learn(op, ptr, idx, T, encoding=enc, trials=100, check_every=25)
    batches, bt = S.schedule(op, ptr, idx, T, S.POLICY_TABLE, table=table, encoding=enc)
    S.check_schedule(op, ptr, idx, batches, bt)
    assert len(batches) == stats["batches"]
    assert S.lower_bound(op, ptr, idx, T) <= S.optimal_batch_count(op, ptr, idx, T) <= len(batches)


def _all_sort_tables(T):
    keys = [p for r in range(2, T + 1) for sub in itertools.combinations(range(T), r)
            for p in itertools.permutations(sub)]
    for choice in itertools.product(*keys):
        yield dict(zip(keys, choice))


def test_learned_equals_best_sort_table_on_small_workloads():
    # The lattice has two types, so four E_sort tables (keys (0, 1) and (1, 0),
    # two choices each): the learned table reaches the best of them.  On a
    # small Figure 1-shaped workload it reaches the lower bound.
    w = WL.make_config(3, instances=3)
    T = w.n_types
    best = min(len(S.schedule(w.op_type, w.child_ptr, w.child_idx, T, S.POLICY_TABLE, table=tab)[0])
               for tab in _all_sort_tables(T))
    table, stats, _ = OL.learn(w.op_type, w.child_ptr, w.child_idx, T, trials=200)
    assert stats["batches"] == best
    op, ptr, idx, T = WL.make_typed_trees("outputs", 3, leaves=(4, 9), seed=5)
    table, stats, _ = OL.learn(op, ptr, idx, T, trials=200)
    assert stats["batches"] == stats["lower_bound"]
