"""The host library's policy learner (edb_learn_policy) against the oracle's:
the learned table, the statistics and every Q value are bit-exact on the
worked example, on lattices, on typed trees and on random graphs, for all
three state encodings and several parameter sets; plus the batch-count study
figures and the C-ABI error conventions.  CPU only."""
import ctypes as C
import json
import os

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

from oracle import learn as OLN
from oracle import schedule as OS
from paper_2302_03851_amd import _lib as L
from paper_2302_03851_amd import edb
from paper_2302_03851_amd import workloads as WL


def csr(children):
    ptr = np.zeros(len(children) + 1, dtype=np.int64)
    for v, ch in enumerate(children):
        ptr[v + 1] = ptr[v] + len(ch)
    return ptr, np.array([c for ch in children for c in ch], dtype=np.int32)


def _compare(op, ptr, idx, T, encoding=OS.ENC_SORT, **kw):
    table, stats, Q = OLN.learn(op, ptr, idx, T, encoding=encoding, **kw)
    g = edb.Graph(op, ptr, idx, np.full(len(op), -1, dtype=np.int32), T)
    ctable, cstats, cQ = edb.learn_policy(g, encoding, **kw)
    assert ctable == OS.flatten_table(table)
    assert cstats == stats
    assert set(cQ) == {k for (k, _a) in Q}
    for k, vals in cQ.items():
        for a in range(T):
            assert vals[a] == Q.get((k, a), 0.0), (k, a)
    return cstats


PARAMS = [
    {},
    dict(n_step=1, epsilon=0.3, lr=0.5),
    dict(n_step=8, alpha=0.9, gamma=0.9, seed=7),
    dict(epsilon=1.0, lr=1.0, seed=123456789),
]


@pytest.mark.parametrize("enc", [OS.ENC_SORT, OS.ENC_BASE, OS.ENC_MAX])
@pytest.mark.parametrize("params", range(len(PARAMS)))
def test_lattice_bit_exact(enc, params):
    w = WL.make_config(3, instances=3)
    _compare(w.op_type, w.child_ptr, w.child_idx, w.n_types, enc, trials=60, check_every=20,
             **PARAMS[params])


@pytest.mark.parametrize("shape", ["outputs", "two_type"])
@pytest.mark.parametrize("enc", [OS.ENC_SORT, OS.ENC_MAX])
def test_typed_trees_bit_exact(shape, enc):
    op, ptr, idx, T = WL.make_typed_trees(shape, 3, leaves=(4, 10), seed=11)
    _compare(op, ptr, idx, T, enc, trials=80, check_every=40, epsilon=0.2)


def test_worked_example_bit_exact(golden_dir):
    with open(os.path.join(golden_dir, "fig1_tree.json")) as f:
        g = json.load(f)
    op = np.array([g["types"][n["type"]] for n in g["nodes"]], dtype=np.int32)
    ptr, idx = csr([n["children"] for n in g["nodes"]])
    st_ = _compare(op, ptr, idx, len(g["types"]))
    assert st_["batches"] == st_["lower_bound"] == 6


@st.composite
def random_graphs(draw):
    n = draw(st.integers(0, 30))
    T = draw(st.integers(1, 4))
    op, children = [], []
    for v in range(n):
        op.append(draw(st.integers(0, T - 1)))
        children.append(draw(st.lists(st.integers(-1, v - 1), max_size=3)) if v else [])
    return np.array(op, dtype=np.int32), children, T


@settings(max_examples=60, deadline=None)
@given(random_graphs(), st.sampled_from([OS.ENC_SORT, OS.ENC_BASE, OS.ENC_MAX]),
       st.sampled_from(range(len(PARAMS))))
def test_random_graphs_bit_exact(g, enc, params):
    op, children, T = g
    ptr, idx = csr(children)
    _compare(op, ptr, idx, T, enc, trials=30, check_every=10, **PARAMS[params])


def _study(op, ptr, idx, T):
    g = edb.Graph(op, ptr, idx, np.full(len(op), -1, dtype=np.int32), T)
    out = {name: edb.Schedule(g, kind).n_batches for name, kind in
           (("depth", L.POLICY_DEPTH), ("agenda", L.POLICY_AGENDA), ("majority", L.POLICY_TABLE),
            ("sufficient", L.POLICY_SUFFICIENT))}
    out["lb"] = edb.lower_bound(g)
    for enc, name in ((L.ENC_SORT, "sort"), (L.ENC_BASE, "base"), (L.ENC_MAX, "max")):
        table, stats, _ = edb.learn_policy(g, enc)
        s = edb.Schedule(g, L.POLICY_TABLE, enc, table)
        assert s.n_batches == stats["batches"]
        OS.check_schedule(op, ptr, idx, s.batches(), s.batch_type.tolist())
        out[name] = stats["batches"]
    return out


def test_batch_count_study_lattice():
    # C3 (32 lattices): the learned E_sort table reaches the best of the four
    # E_sort tables (the configured one), ahead of agenda, depth and the
    # sufficient-condition heuristic; E_base is the weakest encoding.
    w = WL.make_config(3)
    r = _study(w.op_type, w.child_ptr, w.child_idx, w.n_types)
    assert r["sort"] == r["max"] == r["majority"] == 85
    assert r["sort"] < r["sufficient"] < r["agenda"] < r["depth"]
    assert r["base"] > r["sort"] and r["lb"] == 59


def test_batch_count_study_trees_with_outputs():
    # Figure 1's shape at scale (64 trees): every encoding learns a table that
    # meets the lower bound; agenda and depth batch the outputs level by level.
    op, ptr, idx, T = WL.make_typed_trees("outputs", 64, seed=1)
    r = _study(op, ptr, idx, T)
    assert r["sort"] == r["base"] == r["max"] == r["sufficient"] == r["lb"] == 15
    assert r["agenda"] == 24 and r["depth"] == 34


def test_learn_abi_errors():
    lib = L.load()
    op = np.array([0, 0], dtype=np.int32)
    ptr = np.array([0, 0, 1], dtype=np.int64)
    idx = np.array([0], dtype=np.int32)
    g = edb.Graph(op, ptr, idx, np.full(2, -1, dtype=np.int32), 1)
    for bad in (dict(trials=0), dict(check_every=0), dict(n_step=0), dict(alpha=0.0),
                dict(epsilon=1.5), dict(lr=0.0), dict(lr=1.5), dict(gamma=-0.1), dict(encoding=5)):
        enc = bad.pop("encoding", L.ENC_SORT)
        with pytest.raises(L.EdbError) as ei:
            edb.learn_policy(g, enc, **bad)
        assert ei.value.status == L.EDB_ERR_INVALID
    p = L.LearnParams()
    lib.edb_learn_defaults(C.byref(p))
    assert (p.trials, p.check_every, p.n_step, p.alpha, p.epsilon, p.lr, p.gamma, p.seed) == \
        (1000, 50, 4, 0.5, 0.1, 0.2, 1.0, 0)
    h = C.c_void_p()
    assert lib.edb_learn_policy(None, C.byref(p), C.byref(h)) == L.EDB_ERR_INVALID and not h.value
    assert lib.edb_learn_policy(g.handle, C.byref(p), None) == L.EDB_ERR_INVALID
    assert lib.edb_learned_view(None, None, None, None) == L.EDB_ERR_INVALID
    assert lib.edb_learned_q(None, None, None, None, None) == L.EDB_ERR_INVALID
    assert lib.edb_lower_bound(None, None) == L.EDB_ERR_INVALID
