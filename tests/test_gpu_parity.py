"""GPU parity: the HIP path through the C ABI against the oracle.

Bounds (normwise relative error per state vector, max over nodes and h/c):
1e-4 for the fp32 configurations, 2e-2 for the bf16 child-sum configuration.
Every test compares every node: small instances, and the full-size
configurations in the benchmark's launch configuration (HIP graph, planned
layout) and in its concurrent mode (host threads and streams), against the
oracle evaluated instance by instance (instances are independent graphs)."""
import numpy as np
import pytest

from oracle.compare import state_rel_err
from oracle.evaluate import evaluate
from oracle_instances import evaluate_by_instance
from paper_2302_03851_amd import _lib as L
from paper_2302_03851_amd import workloads as WL

pytestmark = pytest.mark.gpu

TOL = {"f32": 1e-4, "bf16": 2e-2}
SMALL = {1: 8, 2: 6, 3: 6, 4: 2, 5: 4, 6: 6, 7: 6}


def _torch():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


def _fwd(w, **kw):
    from paper_2302_03851_amd import edb
    return edb.Forward(w, **kw)


def _oracle(w):
    return evaluate(w.kinds, w.op_type, w.child_ptr, w.child_idx, w.x_row, w.x, w.weights, w.hidden,
                    n_fixed=w.n_children, dtype=w.dtype)


def _h_rows(w):
    """Nodes that have an h output (lattice word cells have none)."""
    return np.array([w.kinds[t] != WL.LAT_WORD for t in w.op_type])


def _check(w, h, c, hr, cr, label):
    err = state_rel_err(h, c, hr, cr, h_rows=_h_rows(w))
    print(f"{label}: {w.name} V={w.n_nodes} max normwise rel err {err:.3e}", flush=True)
    assert np.isfinite(h).all() and np.isfinite(c).all()
    assert err <= TOL[w.dtype], err
    return err


@pytest.mark.parametrize("k", [1, 2, 3, 4, 5, 6, 7])
def test_parity_small(k):
    _torch()
    w = WL.make_config(k, instances=SMALL[k])
    f = _fwd(w)
    f.run()
    h, c = f.states()
    hr, cr = _oracle(w)
    _check(w, h, c, hr, cr, f"small k={k}")
    # lattice words keep h == 0
    if k == 3:
        words = np.array([w.kinds[t] == WL.LAT_WORD for t in w.op_type])
        assert (h[words] == 0).all()


@pytest.mark.parametrize("k", [1, 2, 3, 4, 5, 6, 7])
def test_parity_full_size_every_node(k):
    """The full-size workload in the benchmark's launch configuration (HIP
    graph, planned layout, a replay of the captured graph), every node
    against the oracle (evaluated instance by instance)."""
    _torch()
    w = WL.make_config(k)
    f = _fwd(w)
    f.exec.validate()     # the uploaded descriptors, decoded and bounds-checked on the host
    f.run()
    f.run()               # a replay of the captured graph
    h, c = f.states()
    hr, cr = evaluate_by_instance(w)
    _check(w, h, c, hr, cr, f"full k={k}")


def test_bench_mode_threads_and_streams_every_node():
    """The benchmark's own mode: 16 host threads, each with its own stream and
    arena, call edb_forward (the whole path, eager launches) on the full binary
    TreeLSTM workload concurrently, three times each.  Every thread's arena
    holds the oracle's states at every node, bitwise equal across threads and
    to a single-stream graph replay."""
    import threading
    torch = _torch()
    from paper_2302_03851_amd import edb
    w = WL.make_config(2)
    base = _fwd(w)
    base.run()
    h0, c0 = base.states()
    hr, cr = evaluate_by_instance(w)
    _check(w, h0, c0, hr, cr, "single stream")
    S, steps = 16, 3
    streams = [torch.cuda.Stream() for _ in range(S)]
    arenas = [(torch.full_like(base.arena_h, 9.0), torch.full_like(base.arena_c, -9.0)) for _ in range(S)]
    fwd = edb.ForwardCall(w.op_type, w.child_ptr, w.child_idx, w.x_row, w.n_types, edb.operand_shapes(w),
                          base.cells)
    wptrs = [b.data_ptr() for b in base.weights]
    torch.cuda.synchronize()
    errors = []
    start = threading.Barrier(S)

    def worker(i):
        try:
            start.wait()
            ah, ac = arenas[i]
            for _ in range(steps):
                fwd.call(wptrs, base.x.data_ptr(), ah.data_ptr(), ac.data_ptr(), ah.shape[0],
                         streams[i].cuda_stream)
        except Exception as e:   # reported after the join
            errors.append((i, e))
    ths = [threading.Thread(target=worker, args=(i,)) for i in range(S)]
    for t in ths:
        t.start()
    for t in ths:
        t.join()
    torch.cuda.synchronize()
    assert not errors, errors
    s = base.plan.slot
    for i, (ah, ac) in enumerate(arenas):
        h = ah.float().cpu().numpy().astype(np.float64)[s]
        c = ac.cpu().numpy().astype(np.float64)[s]
        _check(w, h, c, hr, cr, f"thread {i}")
        np.testing.assert_array_equal(h, h0, err_msg=f"thread {i}")
        np.testing.assert_array_equal(c, c0, err_msg=f"thread {i}")


@pytest.mark.parametrize("k", [2, 3, 4, 5, 7])
def test_layout_and_launch_mode_bitwise(k):
    """The planned layout, the identity layout with every operand indexed,
    the PQ-tree layout (zero pads, rows in another order), forced gathers, x read in place and eager launches all give bitwise the
    same node states: only the addressing differs."""
    _torch()
    w = WL.make_config(k, instances=SMALL[k])
    ref = _fwd(w)
    ref.run()
    h0, c0 = ref.states()
    for kw in (dict(plan_mode=L.PLAN_IDENTITY), dict(plan_mode=L.PLAN_PQ), dict(flags=L.USE_GRAPH | L.FORCE_GATHER),
               dict(flags=L.USE_GRAPH | L.X_DIRECT), dict(flags=0),
               dict(flags=L.PROFILE)):
        f = _fwd(w, **kw)
        f.run()
        h, c = f.states()
        np.testing.assert_array_equal(h, h0, err_msg=str(kw))
        np.testing.assert_array_equal(c, c0, err_msg=str(kw))


def _grid_graph(n_grids, R, C, E, H, seed, dtype):
    """n_grids independent R x C grids of GRID cells (children: left, top)."""
    op, ch = [], []
    for gi in range(n_grids):
        base = gi * R * C
        for i in range(R):
            for j in range(C):
                op.append(0)
                ch.append([base + i * C + j - 1 if j > 0 else -1, base + (i - 1) * C + j if i > 0 else -1])
    return WL.make_graph([WL.GRID], E, H, op, ch, [True] * len(op), seed=seed, dtype=dtype, bias_scale=0.2)


def _gru_trees(n_trees, E, H, seed, dtype):
    """n_trees three-node TreeGRU trees (two leaves, one internal node) and a
    chain of internal nodes over them, with non-zero biases."""
    op, ch, hx = [], [], []
    for t in range(n_trees):
        op += [0, 0, 1]
        ch += [[], [], [3 * t, 3 * t + 1]]
        hx += [True, True, False]
    prev = 2
    for t in range(1, min(n_trees, 40)):     # a deeper spine: internal nodes over earlier roots
        op.append(1)
        ch.append([prev, 3 * t + 2])
        hx.append(False)
        prev = len(op) - 1
    return WL.make_graph([WL.GRU_LEAF, WL.GRU_INTERNAL], E, H, op, ch, hx, seed=seed, dtype=dtype,
                         bias_scale=0.2)


def _large_tile_workloads():
    """Workloads whose batches span several large tiles with a ragged row
    tail.  bf16: the child-sum configuration (its leaf batch), grids with a
    zero-padded x segment (E = 120 in a 128-wide segment) and padded units
    (H = 192 of 256), chains, binary trees.  fp32: the binary TreeLSTM
    configuration, the same grids, chains."""
    out = [WL.make_config(5, instances=12), _grid_graph(24, 12, 12, 120, 192, seed=11, dtype="bf16")]
    n = 300   # chains of length 3
    op = [0] * (3 * n)
    ch = [[-1] if i % 3 == 0 else [i - 1] for i in range(3 * n)]
    out.append(WL.make_graph([WL.LSTM_CHAIN], 64, 128, op, ch, [True] * (3 * n), seed=12, dtype="bf16",
                             bias_scale=0.2))
    # binary trees: 200 two-leaf trees
    op, ch, hx = [], [], []
    for t in range(200):
        op += [0, 0, 1]
        ch += [[], [], [3 * t, 3 * t + 1]]
        hx += [True, True, False]
    out.append(WL.make_graph([WL.NARY_LEAF, WL.NARY_INTERNAL], 128, 256, op, ch, hx, seed=13, dtype="bf16",
                             bias_scale=0.2))
    out.append(_gru_trees(200, 128, 256, seed=16, dtype="bf16"))
    out += [WL.make_config(2, instances=16), _grid_graph(24, 12, 12, 120, 192, seed=14, dtype="f32"),
            _gru_trees(200, 128, 192, seed=17, dtype="f32")]
    op = [0] * (3 * n)
    ch = [[-1] if i % 3 == 0 else [i - 1] for i in range(3 * n)]
    out.append(WL.make_graph([WL.LSTM_CHAIN], 64, 128, op, ch, [True] * (3 * n), seed=15, dtype="f32",
                             bias_scale=0.2))
    return out


@pytest.mark.parametrize("variant", [None, 8, 9, 10, 15, 16])
def test_large_tile_bitwise_and_parity(variant, monkeypatch):
    """The large tile, bf16 and fp32 (every supported batch forced onto it, or
    one size class for all), is bitwise equal to the small tile without
    split-K, and within the bound of the oracle."""
    _torch()
    for w in _large_tile_workloads():
        monkeypatch.delenv("EDB_VARIANT", raising=False)
        small = _fwd(w, flags=L.USE_GRAPH | L.NO_SPLIT_K | L.NO_LARGE)
        small.run()
        h0, c0 = small.states()
        if variant is not None:
            monkeypatch.setenv("EDB_VARIANT", str(variant))
        f = _fwd(w, flags=L.USE_GRAPH | L.NO_SPLIT_K | L.TILE_LARGE)
        used = {f.exec.launch_info(i)["variant"] for i in range(1, f.exec.launches())}
        assert used & set(L.LARGE_VARIANTS), used
        f.run()
        h, c = f.states()
        np.testing.assert_array_equal(h, h0, err_msg=f"{w.name} {w.kinds} variant {variant}")
        np.testing.assert_array_equal(c, c0, err_msg=f"{w.name} {w.kinds} variant {variant}")
        if variant is None:
            hr, cr = _oracle(w)
            _check(w, h, c, hr, cr, f"large tile {w.kinds}")


def test_large_tile_indexed_operands_bitwise():
    """On the large tile, indexed operand lists (forced gathers, x read in place
    through its row list, the identity layout with every list indexed) give
    bitwise the states of the planned layout's contiguous lists."""
    _torch()
    w = WL.make_config(5, instances=12)
    base = _fwd(w, flags=L.USE_GRAPH | L.TILE_LARGE)
    assert any(base.exec.launch_info(i)["part"] == L.PART_FORGET for i in range(1, base.exec.launches()))
    base.run()
    h0, c0 = base.states()
    for kw in (dict(flags=L.USE_GRAPH | L.TILE_LARGE | L.FORCE_GATHER),
               dict(flags=L.USE_GRAPH | L.TILE_LARGE | L.X_DIRECT),
               dict(flags=L.USE_GRAPH | L.TILE_LARGE, plan_mode=L.PLAN_IDENTITY)):
        f = _fwd(w, **kw)
        f.run()
        h, c = f.states()
        np.testing.assert_array_equal(h, h0, err_msg=str(kw))
        np.testing.assert_array_equal(c, c0, err_msg=str(kw))


def _two_leaf_trees(kinds, n_trees, E, H, seed):
    """n_trees trees of two x leaves under one internal node (bf16)."""
    op, ch, hx = [], [], []
    for t in range(n_trees):
        op += [0, 0, 1]
        ch += [[], [], [3 * t, 3 * t + 1]]
        hx += [True, True, False]
    return WL.make_graph(kinds, E, H, op, ch, hx, seed=seed, dtype="bf16", scale=0.05, bias_scale=0.2)


WS_CASES = {
    # the child-sum configuration's leaves: 16 k-groups, several row tiles, a ragged tail
    "child-sum": lambda: WL.make_config(5, instances=12),
    # N-ary leaves: a zero-padded x segment (E = 248 of 256: two groups of k-groups) and padded units (H = 200 of 256)
    "nary-padded": lambda: _two_leaf_trees([WL.NARY_LEAF, WL.NARY_INTERNAL], 400, 248, 200, seed=31),
    # TreeGRU leaves
    "gru": lambda: _gru_trees(300, 256, 256, seed=32, dtype="bf16"),
    # 10 leaves (one row block, most rows past the batch) of 64 units (two unit tiles)
    "tiny": lambda: _two_leaf_trees([WL.CS_LEAF, WL.CS_INTERNAL], 5, 256, 64, seed=34),
    # 70,000 leaves: more row tiles than the row table holds at one work-group per CU
    "row-table-bound": lambda: _two_leaf_trees([WL.CS_LEAF, WL.CS_INTERNAL], 35000, 256, 512, seed=33),
}


@pytest.mark.parametrize("case", list(WS_CASES))
def test_weight_stationary_tile_bitwise_and_parity(case, monkeypatch):
    """The weight-stationary tile (every leaf batch forced onto it) is bitwise
    equal to the small tile without split-K, and within the bound of the
    oracle."""
    _torch()
    w = WS_CASES[case]()
    monkeypatch.delenv("EDB_VARIANT", raising=False)
    small = _fwd(w, flags=L.USE_GRAPH | L.NO_SPLIT_K | L.NO_LARGE)
    small.run()
    h0, c0 = small.states()
    monkeypatch.setenv("EDB_VARIANT", str(L.WS_VARIANT))
    f = _fwd(w, flags=L.USE_GRAPH | L.NO_SPLIT_K)
    used = {f.exec.launch_info(i)["variant"] for i in range(1, f.exec.launches())}
    assert L.WS_VARIANT in used, used
    f.run()
    f.run()
    h, c = f.states()
    np.testing.assert_array_equal(h, h0, err_msg=case)
    np.testing.assert_array_equal(c, c0, err_msg=case)
    if case != "row-table-bound":
        hr, cr = _oracle(w)
        _check(w, h, c, hr, cr, f"weight-stationary tile {case}")


def test_weight_stationary_tile_indexed_operands_bitwise(monkeypatch):
    """On the weight-stationary tile, indexed lists (forced gathers, x read in
    place through its row list, the identity layout with every list indexed)
    give bitwise the states of the planned layout's contiguous lists."""
    _torch()
    w = WL.make_config(5, instances=12)
    monkeypatch.setenv("EDB_VARIANT", str(L.WS_VARIANT))
    base = _fwd(w, flags=L.USE_GRAPH | L.NO_SPLIT_K)
    assert base.exec.launch_info(1)["variant"] == L.WS_VARIANT
    base.run()
    h0, c0 = base.states()
    for kw in (dict(flags=L.USE_GRAPH | L.NO_SPLIT_K | L.FORCE_GATHER),
               dict(flags=L.USE_GRAPH | L.NO_SPLIT_K | L.X_DIRECT),
               dict(flags=L.USE_GRAPH | L.NO_SPLIT_K, plan_mode=L.PLAN_IDENTITY)):
        f = _fwd(w, **kw)
        assert f.exec.launch_info(1)["variant"] == L.WS_VARIANT, kw
        f.run()
        h, c = f.states()
        np.testing.assert_array_equal(h, h0, err_msg=str(kw))
        np.testing.assert_array_equal(c, c0, err_msg=str(kw))


def test_large_tile_child_sum_many_children():
    """Child-sum parents with up to 9 children on the large tile (the per-parent
    reduction's loop beyond 4 children) against the small tile and the oracle."""
    _torch()
    rng = np.random.default_rng(21)
    op, ch, hx = [], [], []
    for t in range(160):                 # 160 two-level trees, root arity 1..9
        k = int(rng.integers(1, 10))
        leaves = list(range(len(op), len(op) + k))
        op += [0] * k
        ch += [[]] * k
        hx += [True] * k
        op.append(1)
        ch.append(leaves)
        hx.append(False)
    w = WL.make_graph([WL.CS_LEAF, WL.CS_INTERNAL], 512, 512, op, ch, hx, seed=22, dtype="bf16",
                      scale=0.05, bias_scale=0.2)
    small = _fwd(w, flags=L.USE_GRAPH | L.NO_SPLIT_K | L.NO_LARGE)
    small.run()
    h0, c0 = small.states()
    f = _fwd(w, flags=L.USE_GRAPH | L.NO_SPLIT_K | L.TILE_LARGE)
    parts = [f.exec.launch_info(i)["part"] for i in range(1, f.exec.launches())]
    assert L.PART_CHILD_SUM in parts and L.PART_FORGET in parts
    f.run()
    h, c = f.states()
    np.testing.assert_array_equal(h, h0)
    np.testing.assert_array_equal(c, c0)
    hr, cr = _oracle(w)
    _check(w, h, c, hr, cr, "child-sum up to 9 children, large tile")


def _stream_workloads():
    """Workloads of every kind the streamed tile serves, with ragged row tails:
    chains (fp32), binary trees (fp32), lattices (the word cells; the
    character cells keep the staged tile), grids with a zero-padded x segment
    (E = 120 of 128) and padded units (H = 200 of 256), the child-sum
    configuration (its leaves, bf16) and bf16 chains of 900 rows."""
    out = [WL.make_config(1), WL.make_config(2, instances=SMALL[2]), WL.make_config(3, instances=SMALL[3]),
           _grid_graph(3, 6, 7, 120, 200, seed=21, dtype="f32"), WL.make_config(5, instances=SMALL[5])]
    n = 300
    op = [0] * (3 * n)
    ch = [[-1] if i % 3 == 0 else [i - 1] for i in range(3 * n)]
    out.append(WL.make_graph([WL.LSTM_CHAIN], 64, 128, op, ch, [True] * (3 * n), seed=22, dtype="bf16",
                             bias_scale=0.2))
    out += [_gru_trees(60, 64, 128, seed=23, dtype="f32"), _gru_trees(60, 64, 128, seed=24, dtype="bf16")]
    return out


@pytest.mark.parametrize("variant", [11, 12, 13, 14])
def test_streamed_tile_bitwise_and_parity(variant, monkeypatch):
    """Every batch the streamed tile serves, forced onto `variant`, is bitwise
    equal to the staged tile with the same rows and reduction split (eager
    against two graph replays, planned and indexed operand lists), and within
    the bound of the oracle."""
    _torch()
    staged = L.STREAM_STAGED[variant]
    for w in _stream_workloads():
        monkeypatch.setenv("EDB_VARIANT", str(staged))
        ref = _fwd(w, flags=0)
        ref.run()
        h0, c0 = ref.states()
        monkeypatch.setenv("EDB_VARIANT", str(variant))
        for flags in (L.USE_GRAPH, L.USE_GRAPH | L.FORCE_GATHER | L.X_DIRECT):
            f = _fwd(w, flags=flags)
            used = {f.exec.launch_info(i)["variant"] for i in range(1, f.exec.launches())}
            assert variant in used, (w.name, used)
            for _ in range(2):
                f.run()
                h, c = f.states()
                np.testing.assert_array_equal(h, h0, err_msg=f"{w.name} {w.kinds} variant {variant} flags {flags}")
                np.testing.assert_array_equal(c, c0, err_msg=f"{w.name} {w.kinds} variant {variant} flags {flags}")
        hr, cr = _oracle(w)
        _check(w, h, c, hr, cr, f"streamed variant {variant}")


DATAFLOW_OFF = ("dataflow launches are switched off: their first GPU runs did not drain "
                "(cause not yet shown); every batch runs as its own launch")


@pytest.mark.skip(reason=DATAFLOW_OFF)
@pytest.mark.parametrize("k", [1, 2, 3, 4, 5])
def test_dataflow_matches_per_batch_launches(k):
    """Dataflow launches (default) against one launch per batch: both within
    the bound of the oracle, and identical where the tile shapes agree."""
    _torch()
    w = WL.make_config(k, instances=SMALL[k])
    hr, cr = _oracle(w)
    flow = _fwd(w)
    n_flow = sum(1 for i in range(flow.exec.launches())
                 if flow.exec.launch_info(i)["variant"] == L.FLOW_VARIANT)
    assert n_flow >= 1
    flow.run()
    h1, c1 = flow.states()
    _check(w, h1, c1, hr, cr, f"dataflow k={k}")
    per = _fwd(w, flags=L.USE_GRAPH | L.NO_FLOW)
    per.run()
    h2, c2 = per.states()
    _check(w, h2, c2, hr, cr, f"per-batch k={k}")


@pytest.mark.skip(reason=DATAFLOW_OFF)
def test_dataflow_full_size_replays():
    """Full-size binary trees through the dataflow launch, replayed several
    times: every replay bitwise equal to the first (no timing dependence)."""
    _torch()
    w = WL.make_config(2)
    f = _fwd(w)
    f.run()
    h0, c0 = f.states()
    for i in range(5):
        f.run()
        h, c = f.states()
        np.testing.assert_array_equal(h, h0, err_msg=f"replay {i}")
        np.testing.assert_array_equal(c, c0, err_msg=f"replay {i}")


@pytest.mark.skip(reason=DATAFLOW_OFF)
def test_dataflow_wait_timeout_is_reported(monkeypatch):
    """A wait bound of one microsecond forces the bounded-wait path from the
    host: every kernel still exits normally and edb_exec_check reports it."""
    _torch()
    monkeypatch.setenv("EDB_SPIN_US", "1")
    w = WL.make_config(2, instances=16)
    f = _fwd(w, flags=0)
    f.run()
    try:
        f.exec.check(f.stream.cuda_stream)
        timed_out = False
    except L.EdbError as e:
        timed_out = True
        assert e.status == L.EDB_ERR_HIP and "timed out" in str(e)
    # with a 1 us bound a timeout is all but certain; either way the launch
    # drained and a fresh executor with the default bound is correct
    monkeypatch.delenv("EDB_SPIN_US")
    g = _fwd(w, flags=0)
    g.run()
    h, c = g.states()
    hr, cr = _oracle(w)
    _check(w, h, c, hr, cr, f"after forced timeout (timed_out={timed_out})")


def test_graph_replays_match_eager():
    """Replays of the captured graph, with eager work and synchronisations in
    between, all equal the eager result."""
    torch = _torch()
    w = WL.make_config(2, instances=8)
    eager = _fwd(w, flags=0)
    eager.run()
    he, ce = eager.states()
    f = _fwd(w)
    for i in range(4):
        f.arena_h.fill_(7.0)
        f.arena_c.fill_(-3.0)
        torch.cuda.synchronize()
        f.run()
        h, c = f.states()
        np.testing.assert_array_equal(h, he, err_msg=f"replay {i}")
        np.testing.assert_array_equal(c, ce, err_msg=f"replay {i}")


def _kernel_sequence(f):
    out = []
    for i in range(f.exec.launches()):
        inf = f.exec.launch_info(i)
        if inf["grid"] > 0:
            out.append((inf["kind"], inf["variant"], inf["part"], inf["block"]))
    return out


@pytest.mark.parametrize("k", [2, 5])
def test_graph_kept_per_stream_reused_by_new_inputs(k):
    """EDB_USE_GRAPH executions share the stream's kept graphs: a new input
    graph (the mini-batch relabelled) with the same kernel sequence updates
    the kept graph's nodes instead of instantiating one, so does the first
    input again, and another workload's sequence gets a graph of its own
    without displacing the first.  Every arena is bitwise the eager one."""
    _torch()
    from paper_2302_03851_amd import edb
    w = WL.make_config(k, instances=SMALL[k])
    w2, perm = WL.relabel(w, 11)
    eager = _fwd(w, flags=0)
    eager.run()
    he, ce = eager.states()
    f1 = _fwd(w)
    f1.run()
    h1, c1 = f1.states()
    np.testing.assert_array_equal(h1, he)
    np.testing.assert_array_equal(c1, ce)
    i0, u0 = edb.graph_stats()
    f2 = _fwd(w2)
    same = _kernel_sequence(f2) == _kernel_sequence(f1)
    f2.run()
    h2, c2 = f2.states()
    np.testing.assert_array_equal(h2[perm], he)
    np.testing.assert_array_equal(c2[perm], ce)
    i1, u1 = edb.graph_stats()
    assert same, "a relabelled mini-batch should select the same kernels"
    assert (i1, u1) == (i0, u0 + 1), (i0, u0, i1, u1)
    f1.arena_h.fill_(3.0)
    f1.run()
    h1b, c1b = f1.states()
    np.testing.assert_array_equal(h1b, he)
    np.testing.assert_array_equal(c1b, ce)
    i2, u2 = edb.graph_stats()
    assert (i2, u2) == (i1, u1 + 1), (i1, u1, i2, u2)
    # another workload: its own graph (one instantiation at most), then the first input reuses its graph
    w3 = WL.make_config(1, instances=SMALL[1])
    e3 = _fwd(w3, flags=0)
    e3.run()
    h3e, c3e = e3.states()
    f3 = _fwd(w3)
    f3.run()
    h3, c3 = f3.states()
    np.testing.assert_array_equal(h3, h3e)
    np.testing.assert_array_equal(c3, c3e)
    i3, _ = edb.graph_stats()
    assert i3 <= i2 + 1
    f2.run()
    h2b, _ = f2.states()
    np.testing.assert_array_equal(h2b[perm], he)
    i4, _ = edb.graph_stats()
    assert i4 == i3


def test_kept_graphs_replaced_least_recently_used_and_per_stream_threads():
    """More kernel sequences on one stream than it keeps: the least recently
    used graph is replaced (after its last launch) and built again when its
    sequence returns; four threads, each with a stream of its own, run their
    executors through their streams' kept graphs at once; and releasing a
    stream drops its graphs.  Every arena is bitwise the eager one."""
    torch = _torch()
    import threading
    from paper_2302_03851_amd import edb
    ks = [1, 2, 3, 4, 6, 7]   # six different kernel sequences
    ws = {k: WL.make_config(k, instances=SMALL[k]) for k in ks}
    ref = {}
    for k in ks:
        e = _fwd(ws[k], flags=0)
        e.run()
        ref[k] = e.states()
    st = torch.cuda.Stream()
    with torch.cuda.stream(st):
        fs = {k: _fwd(ws[k]) for k in ks}
    i0, _ = edb.graph_stats()
    for rnd in range(2):
        for k in ks:
            with torch.cuda.stream(st):
                fs[k].arena_h.fill_(9.0)   # on the stream, ordered before the run
                fs[k].run()
            h, c = fs[k].states()
            np.testing.assert_array_equal(h, ref[k][0], err_msg=f"round {rnd} workload {k}")
            np.testing.assert_array_equal(c, ref[k][1], err_msg=f"round {rnd} workload {k}")
    i1, _ = edb.graph_stats()
    assert i1 - i0 >= len(ks) + 2, (i0, i1)   # the second round rebuilds the replaced ones
    # threads, one stream each, the same workload
    w = ws[2]
    streams = [torch.cuda.Stream() for _ in range(4)]
    fwds = []
    for sx in streams:
        with torch.cuda.stream(sx):
            fwds.append(_fwd(w))
    torch.cuda.synchronize()
    errors = []

    def work(j):
        try:
            for _ in range(5):
                fwds[j].run()
        except Exception as ex:   # reported below
            errors.append(ex)

    th = [threading.Thread(target=work, args=(j,)) for j in range(4)]
    for t in th:
        t.start()
    for t in th:
        t.join()
    assert not errors, errors
    for j in range(4):
        h, c = fwds[j].states()
        np.testing.assert_array_equal(h, ref[2][0], err_msg=f"thread {j}")
        np.testing.assert_array_equal(c, ref[2][1], err_msg=f"thread {j}")
    # releasing a stream drops its kept graphs: the next execution there builds its graph again
    edb.ForwardCall.release_stream(streams[0].cuda_stream)
    i2, _ = edb.graph_stats()
    fwds[0].arena_h.fill_(2.0)
    torch.cuda.synchronize()
    fwds[0].run()
    h, c = fwds[0].states()
    np.testing.assert_array_equal(h, ref[2][0])
    np.testing.assert_array_equal(c, ref[2][1])
    i3, _ = edb.graph_stats()
    assert i3 == i2 + 1, (i2, i3)


def test_forward_call_graph_path_matches_eager():
    """edb_forward with EDB_USE_GRAPH (the plain path's launches through the
    stream's kept graph): two different mini-batches of the same kernel
    sequence in turn, each arena bitwise the eager one."""
    torch = _torch()
    from paper_2302_03851_amd import edb
    w = WL.make_config(2, instances=SMALL[2])
    w2, perm = WL.relabel(w, 3)
    ref = _fwd(w, flags=0)
    ref.run()
    h0, c0 = ref.states()
    st = torch.cuda.Stream()
    fcs = [edb.ForwardCall(v.op_type, v.child_ptr, v.child_idx, v.x_row, v.n_types, edb.operand_shapes(v),
                           ref.cells, flags=L.USE_GRAPH) for v in (w, w2)]
    g2 = edb.Graph(w2.op_type, w2.child_ptr, w2.child_idx, w2.x_row, w2.n_types)
    plans = [ref.plan, edb.Plan(g2, edb.Schedule(g2), edb.operand_shapes(w2))]
    for rep in range(3):
        for j, fc in enumerate(fcs):
            ah = torch.full((plans[j].n_slots, ref.arena_h.shape[1]), 5.0, dtype=ref.arena_h.dtype, device="cuda")
            ac = torch.full((plans[j].n_slots, ref.arena_c.shape[1]), 5.0, dtype=torch.float32, device="cuda")
            torch.cuda.synchronize()
            fc.call([b.data_ptr() for b in ref.weights], ref.x.data_ptr(), ah.data_ptr(), ac.data_ptr(),
                    ah.shape[0], st.cuda_stream)
            st.synchronize()
            s = plans[j].slot
            h = ah.float().cpu().numpy()[s]
            c = ac.cpu().numpy()[s]
            if j == 1:
                h, c = h[perm], c[perm]
            np.testing.assert_array_equal(h, h0, err_msg=f"rep {rep} batch {j}")
            np.testing.assert_array_equal(c, c0, err_msg=f"rep {rep} batch {j}")
    edb.ForwardCall.release_stream(st.cuda_stream)


@pytest.mark.parametrize("k", [2, 5])
def test_forward_call_matches_handles(k):
    """edb_forward (the whole path in one call) writes bitwise the same arena
    as the separate calls with eager launches."""
    torch = _torch()
    from paper_2302_03851_amd import edb
    w = WL.make_config(k, instances=SMALL[k])
    ref = _fwd(w, flags=0)
    ref.run()
    h0, c0 = ref.states()
    table = edb.LATTICE_TABLE if k == 3 else None
    fc = edb.ForwardCall(w.op_type, w.child_ptr, w.child_idx, w.x_row, w.n_types, edb.operand_shapes(w),
                         ref.cells, table=table)
    ah = torch.full_like(ref.arena_h, 5.0)
    ac = torch.full_like(ref.arena_c, 5.0)
    fc.call([b.data_ptr() for b in ref.weights], ref.x.data_ptr(), ah.data_ptr(), ac.data_ptr(),
            ah.shape[0], ref.stream.cuda_stream)
    torch.cuda.synchronize()
    s = ref.plan.slot
    np.testing.assert_array_equal(ah.float().cpu().numpy()[s], h0)
    np.testing.assert_array_equal(ac.cpu().numpy()[s], c0)


@pytest.mark.gpu
def test_forward_stream_block_growth_release_and_shared_stream():
    """edb_forward's device block per stream: a small mini-batch, then a
    larger one on the same stream (the block grows in stream order), the
    release, another call, and two threads enqueueing on one stream; every
    arena is bitwise the one of the separate calls with eager launches."""
    torch = _torch()
    import threading
    from paper_2302_03851_amd import edb

    def case(k, inst):
        w = WL.make_config(k, instances=inst)
        ref = _fwd(w, flags=0)
        ref.run()
        torch.cuda.synchronize()
        h0, c0 = ref.states()
        fc = edb.ForwardCall(w.op_type, w.child_ptr, w.child_idx, w.x_row, w.n_types, edb.operand_shapes(w),
                             ref.cells)
        return w, ref, fc, h0, c0

    def run(cs, stream, fill):
        w, ref, fc, h0, c0 = cs
        ah = torch.full_like(ref.arena_h, fill)
        ac = torch.full_like(ref.arena_c, fill)
        torch.cuda.synchronize()
        fc.call([b.data_ptr() for b in ref.weights], ref.x.data_ptr(), ah.data_ptr(), ac.data_ptr(),
                ah.shape[0], stream.cuda_stream)
        return ah, ac

    def check(cs, ah, ac, what):
        _, ref, _, h0, c0 = cs
        s = ref.plan.slot
        np.testing.assert_array_equal(ah.float().cpu().numpy()[s], h0, err_msg=what)
        np.testing.assert_array_equal(ac.cpu().numpy()[s], c0, err_msg=what)

    small, large = case(2, 4), case(5, 24)
    st = torch.cuda.Stream()
    outs = [(small, run(small, st, 5.0), "small"), (large, run(large, st, 7.0), "larger after smaller"),
            (small, run(small, st, 9.0), "small after larger")]
    torch.cuda.synchronize()
    for cs, (ah, ac), what in outs:
        check(cs, ah, ac, what)
    edb.ForwardCall.release_stream(st.cuda_stream)
    ah, ac = run(large, st, 3.0)
    torch.cuda.synchronize()
    check(large, ah, ac, "after release")
    edb.ForwardCall.release_stream(st.cuda_stream)
    edb.ForwardCall.release_stream(st.cuda_stream)   # no block: a no-op

    # two threads, one stream, eight calls each, every call with its own arena
    res, errs = {}, []

    def worker(t):
        try:
            for j in range(8):
                res[(t, j)] = run(small if (t + j) % 2 else large, st, float(t * 8 + j))
        except Exception as e:   # reported below
            errs.append(e)
    th = [threading.Thread(target=worker, args=(t,)) for t in range(2)]
    for t in th:
        t.start()
    for t in th:
        t.join()
    torch.cuda.synchronize()
    assert not errs, errs
    for (t, j), (ah, ac) in res.items():
        check(small if (t + j) % 2 else large, ah, ac, f"thread {t} call {j}")
    edb.ForwardCall.release_stream(st.cuda_stream)


def test_policies_give_same_states():
    """Agenda, depth, sufficient-condition and learned schedules change the
    batches, not the results."""
    _torch()
    from paper_2302_03851_amd import edb
    w = WL.make_config(3, instances=4)
    hr, cr = _oracle(w)
    g = edb.Graph(w.op_type, w.child_ptr, w.child_idx, w.x_row, w.n_types)
    learned = {}
    for enc in (L.ENC_SORT, L.ENC_BASE):
        learned[enc], _, _ = edb.learn_policy(g, enc, trials=200)
    cases = [dict(policy=L.POLICY_AGENDA), dict(policy=L.POLICY_DEPTH), dict(policy=L.POLICY_SUFFICIENT),
             dict(policy=L.POLICY_TABLE, table=learned[L.ENC_SORT]),
             dict(policy=L.POLICY_TABLE, table=learned[L.ENC_BASE], encoding=L.ENC_BASE)]
    for kw in cases:
        f = _fwd(w, **kw)
        f.run()
        h, c = f.states()
        _check(w, h, c, hr, cr, f"policy {kw}")


def test_two_type_treelstm_policies_give_same_states():
    """TreeLSTM with two internal cell types: the batching policy (learned
    table, sufficient condition, agenda, depth) changes the batches, not the
    results."""
    _torch()
    from paper_2302_03851_amd import edb
    w = WL.make_config(6, instances=8)
    hr, cr = _oracle(w)
    g = edb.Graph(w.op_type, w.child_ptr, w.child_idx, w.x_row, w.n_types)
    table, _, _ = edb.learn_policy(g, L.ENC_SORT, trials=200)
    for kw in (dict(policy=L.POLICY_TABLE, table=table), dict(policy=L.POLICY_SUFFICIENT),
               dict(policy=L.POLICY_AGENDA), dict(policy=L.POLICY_DEPTH)):
        f = _fwd(w, **kw)
        f.run()
        h, c = f.states()
        _check(w, h, c, hr, cr, f"two-type policy {kw}")


def test_edge_cases():
    _torch()
    # single leaf; single chain node; a batch of one row per kind
    w = WL.make_graph([WL.NARY_LEAF, WL.NARY_INTERNAL], 256, 256, [0], [[]], [True], seed=3)
    f = _fwd(w)
    f.run()
    h, c = f.states()
    hr, cr = _oracle(w)
    _check(w, h, c, hr, cr, "single leaf")
    # internal nodes with one or both children absent, non-zero biases
    w = WL.make_graph([WL.NARY_LEAF, WL.NARY_INTERNAL], 64, 64, [0, 0, 1, 1, 1],
                      [[], [], [0, -1], [-1, 1], [2, 3]], [True, True, False, False, False],
                      seed=4, bias_scale=0.5)
    f = _fwd(w)
    f.run()
    h, c = f.states()
    hr, cr = _oracle(w)
    _check(w, h, c, hr, cr, "absent children")
    # odd sizes: H = 200 with E = 100 (padded K and units), ragged row tail
    w = WL.make_config(3, instances=1)
    f = _fwd(w)
    f.run()
    h, c = f.states()
    hr, cr = _oracle(w)
    _check(w, h, c, hr, cr, "one lattice")
    # child-sum in fp32 and chain in bf16 (the other dtype of each kind)
    for kinds, E, H, dt in (([WL.CS_LEAF, WL.CS_INTERNAL], 64, 64, "f32"),):
        ch = [[], [], [], [0, 1, 2], [3], [3, 4]]
        w = WL.make_graph(kinds, E, H, [0, 0, 0, 1, 1, 1], ch, [True] * 3 + [False] * 3, seed=5,
                          dtype=dt, bias_scale=0.3)
        f = _fwd(w)
        f.run()
        h, c = f.states()
        hr, cr = _oracle(w)
        _check(w, h, c, hr, cr, "child-sum f32")
    op = [0] * 12
    ch = [[-1]] + [[i] for i in range(11)]
    w = WL.make_graph([WL.LSTM_CHAIN], 64, 64, op, ch, [True] * 12, seed=6, dtype="bf16", bias_scale=0.2)
    f = _fwd(w)
    f.run()
    h, c = f.states()
    hr, cr = _oracle(w)
    _check(w, h, c, hr, cr, "chain bf16")


def test_empty_graph():
    torch = _torch()
    from paper_2302_03851_amd import edb
    w = WL.make_graph([WL.NARY_LEAF, WL.NARY_INTERNAL], 64, 64, [], [], [], seed=1)
    f = _fwd(w)
    assert f.sched.n_batches == 0 and f.exec.launches() == 1
    f.run()
    h, c = f.states()
    assert h.shape == (0, 64)
    # the one-call path on a stream of its own: nothing to copy or launch
    fc = edb.ForwardCall(w.op_type, w.child_ptr, w.child_idx, w.x_row, w.n_types, edb.operand_shapes(w), f.cells)
    st = torch.cuda.Stream()
    for _ in range(2):
        fc.call([b.data_ptr() for b in f.weights], f.x.data_ptr(), f.arena_h.data_ptr(), f.arena_c.data_ptr(),
                f.arena_h.shape[0], st.cuda_stream)
    torch.cuda.synchronize()
    edb.ForwardCall.release_stream(st.cuda_stream)
