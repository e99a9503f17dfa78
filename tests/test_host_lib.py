"""The C-ABI host library on the CPU: every declared symbol is exported; the
C++ schedule and memory plan are bit-exact against the oracle's on all five
configurations and on random graphs; error conventions; dry-run launch
lists (no GPU call)."""
import ctypes as C
import os
import re

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

from oracle import plan as OP
from oracle import schedule as OS
from paper_2302_03851_amd import _lib as L
from paper_2302_03851_amd import edb
from paper_2302_03851_amd import workloads as WL

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def lib():
    return L.load()


def test_header_symbols_exported(lib):
    with open(os.path.join(ROOT, "include", "edb.h")) as f:
        text = f.read()
    declared = set(re.findall(r"\b(edb_[a-z_]+)\s*\(", text))
    assert declared == set(L.EXPORTS)
    for name in declared:
        assert hasattr(lib, name), name
    assert lib.edb_version() >= 10000


def _oracle_schedule(w, policy=OS.POLICY_TABLE, table=None, encoding=OS.ENC_SORT):
    return OS.schedule(w.op_type, w.child_ptr, w.child_idx, w.n_types, policy, table, encoding)


CFG_INSTANCES = {1: None, 2: None, 3: None, 4: None, 5: 48, 6: None, 7: None, 8: 3, 9: None}


@pytest.mark.parametrize("k", [1, 2, 3, 4, 5, 8, 9])
@pytest.mark.parametrize("policy", [OS.POLICY_TABLE, OS.POLICY_AGENDA, OS.POLICY_DEPTH, OS.POLICY_SUFFICIENT])
def test_schedule_bit_exact_configs(k, policy):
    w = WL.make_config(k, instances=CFG_INSTANCES[k])
    table = edb.LATTICE_TABLE if k == 3 else None
    g = edb.Graph(w.op_type, w.child_ptr, w.child_idx, w.x_row, w.n_types)
    s = edb.Schedule(g, policy, L.ENC_SORT, table)
    batches, bt = _oracle_schedule(w, policy, table)
    assert s.batches() == batches
    assert s.batch_type.tolist() == bt
    assert edb.lower_bound(g) == OS.lower_bound(w.op_type, w.child_ptr, w.child_idx, w.n_types)


def _compare_plan(pl, ref, batches):
    assert pl.n_slots == ref.n_slots
    np.testing.assert_array_equal(pl.slot, ref.slot)
    np.testing.assert_array_equal(pl.x_slot, ref.x_slot)
    assert pl.order.tolist() == [v for o in ref.order for v in o]
    assert sorted(pl.pads.tolist()) == sorted(ref.pads)
    for b in range(len(batches)):
        segs = pl.batch_segments(b)
        assert segs[0] == ref.results[b]
        assert segs[1:] == [(k, s) for k, s in ref.segments[b]]
        if ref.ragged_ptr[b] is not None:
            off = int(pl.ragged_off[b])
            assert pl.ragged_pool[off:off + len(ref.ragged_ptr[b])].tolist() == ref.ragged_ptr[b]
        else:
            assert pl.ragged_off[b] == -1


@pytest.mark.parametrize("k", [1, 2, 3, 4, 5, 8, 9])
@pytest.mark.parametrize("mode", [OP.PLAN_RC, OP.PLAN_IDENTITY])
def test_plan_bit_exact_configs(k, mode):
    w = WL.make_config(k, instances=CFG_INSTANCES[k])
    table = edb.LATTICE_TABLE if k == 3 else None
    g = edb.Graph(w.op_type, w.child_ptr, w.child_idx, w.x_row, w.n_types)
    s = edb.Schedule(g, L.POLICY_TABLE, L.ENC_SORT, table)
    shapes = edb.operand_shapes(w)
    pl = edb.Plan(g, s, shapes, mode)
    batches, _ = _oracle_schedule(w, OS.POLICY_TABLE, table)
    ref = OP.plan_memory(w.op_type, w.child_ptr, w.child_idx, batches, shapes, mode)
    _compare_plan(pl, ref, batches)


@st.composite
def random_graphs(draw):
    n = draw(st.integers(1, 40))
    T = draw(st.integers(1, 3))
    # per type: n_fixed in 0..2, ragged flag
    nfix = [draw(st.integers(0, 2)) for _ in range(T)]
    rag = [draw(st.booleans()) for _ in range(T)]
    op, children = [], []
    for v in range(n):
        t = draw(st.integers(0, T - 1))
        op.append(t)
        kids = []
        for _ in range(nfix[t]):
            kids.append(draw(st.integers(-1, v - 1)) if v else -1)
        if rag[t] and v:
            kids += draw(st.lists(st.integers(-1, v - 1), max_size=4))
        children.append(kids)
    return np.array(op, dtype=np.int32), children, T, [(nfix[t], int(rag[t]), 0) for t in range(T)]


@settings(max_examples=80, deadline=None)
@given(random_graphs(), st.sampled_from([OS.ENC_SORT, OS.ENC_BASE, OS.ENC_MAX]),
       st.sampled_from([OS.POLICY_TABLE, OS.POLICY_AGENDA, OS.POLICY_DEPTH, OS.POLICY_SUFFICIENT]),
       st.sampled_from([OP.PLAN_RC, OP.PLAN_IDENTITY]))
def test_random_graphs_bit_exact(g, enc, policy, mode):
    op, children, T, shapes = g
    ptr = np.zeros(len(children) + 1, dtype=np.int64)
    for v, ch in enumerate(children):
        ptr[v + 1] = ptr[v] + len(ch)
    idx = np.array([c for ch in children for c in ch], dtype=np.int32)
    x_row = np.full(len(op), -1, dtype=np.int32)
    table = {(0,): 0, (1, 0): 1, (0, 1): 1, (2, 1, 0): 2, (0, 1, 2): 1}
    gr = edb.Graph(op, ptr, idx, x_row, T)
    s = edb.Schedule(gr, policy, enc, table)
    batches, bt = OS.schedule(op, ptr, idx, T, policy, table, enc)
    assert s.batches() == batches
    assert s.batch_type.tolist() == bt
    assert edb.lower_bound(gr) == OS.lower_bound(op, ptr, idx, T)
    pl = edb.Plan(gr, s, shapes, mode)
    ref = OP.plan_memory(op, ptr, idx, batches, shapes, mode)
    _compare_plan(pl, ref, batches)
    OP.hazard_check(op, ptr, idx, batches, ref)


def _status(lib, fn, *args):
    st_ = fn(*args)
    msg = lib.edb_last_error().decode()
    return st_, msg


def test_abi_errors(lib):
    P = C.POINTER
    h = C.c_void_p()
    op = np.array([0, 0], dtype=np.int32)
    ptr = np.array([0, 1, 2], dtype=np.int64)
    xr = np.array([-1, -1], dtype=np.int32)
    cyc = np.array([1, 0], dtype=np.int32)
    p_ = lambda a, t: a.ctypes.data_as(P(t))
    st_, msg = _status(lib, lib.edb_build_graph, 2, 1, p_(op, C.c_int32), p_(ptr, C.c_int64),
                       p_(cyc, C.c_int32), p_(xr, C.c_int32), C.byref(h))
    assert st_ == L.EDB_ERR_CYCLE and "cycle" in msg and not h.value
    bad = np.array([5, -1], dtype=np.int32)
    st_, _ = _status(lib, lib.edb_build_graph, 2, 1, p_(op, C.c_int32), p_(ptr, C.c_int64),
                     p_(bad, C.c_int32), p_(xr, C.c_int32), C.byref(h))
    assert st_ == L.EDB_ERR_INVALID and not h.value
    selfe = np.array([0, -1], dtype=np.int32)
    st_, _ = _status(lib, lib.edb_build_graph, 2, 1, p_(op, C.c_int32), p_(ptr, C.c_int64),
                     p_(selfe, C.c_int32), p_(xr, C.c_int32), C.byref(h))
    assert st_ == L.EDB_ERR_INVALID
    badt = np.array([0, 3], dtype=np.int32)
    ok_idx = np.array([-1, 0], dtype=np.int32)
    st_, _ = _status(lib, lib.edb_build_graph, 2, 1, p_(badt, C.c_int32), p_(ptr, C.c_int64),
                     p_(ok_idx, C.c_int32), p_(xr, C.c_int32), C.byref(h))
    assert st_ == L.EDB_ERR_INVALID
    nonmono = np.array([0, 2, 1], dtype=np.int64)
    st_, _ = _status(lib, lib.edb_build_graph, 2, 1, p_(op, C.c_int32), p_(nonmono, C.c_int64),
                     p_(ok_idx, C.c_int32), p_(xr, C.c_int32), C.byref(h))
    assert st_ == L.EDB_ERR_INVALID
    st_, _ = _status(lib, lib.edb_build_graph, -1, 1, None, p_(ptr, C.c_int64), None, None, C.byref(h))
    assert st_ == L.EDB_ERR_INVALID
    st_, _ = _status(lib, lib.edb_build_graph, 2, 1, p_(op, C.c_int32), p_(ptr, C.c_int64),
                     p_(ok_idx, C.c_int32), p_(xr, C.c_int32), None)
    assert st_ == L.EDB_ERR_INVALID

    g = edb.Graph(op, ptr, ok_idx, xr, 1)
    # malformed tables
    for flat in ([2, 1, 0, 0], [1, 5, 0, 0], [1, -1, 0], [1, 1, 0, 0, 9], [-1]):
        with pytest.raises(L.EdbError) as ei:
            edb.Schedule(g, L.POLICY_TABLE, L.ENC_SORT, flat)
        assert ei.value.status == L.EDB_ERR_TABLE
    with pytest.raises(L.EdbError) as ei:
        edb.Schedule(g, 7)
    assert ei.value.status == L.EDB_ERR_INVALID
    s = edb.Schedule(g)
    # shape mismatch: the second node has 1 child but the type declares 2 fixed
    with pytest.raises(L.EdbError) as ei:
        edb.Plan(g, s, [(2, 0, 0)])
    assert ei.value.status == L.EDB_ERR_UNSUPPORTED
    # has_x without an x row
    with pytest.raises(L.EdbError) as ei:
        edb.Plan(g, s, [(1, 0, 1)])
    assert ei.value.status == L.EDB_ERR_INVALID
    pl = edb.Plan(g, s, [(1, 0, 0)])
    # cell kind vs operand shape mismatch, unsupported N, bad dtype
    cells = [edb.cell_struct(WL.GRID, 8, 8, 0, L.F32)]
    with pytest.raises(L.EdbError) as ei:
        edb.Exec(g, s, pl, cells, L.DRYRUN)
    assert ei.value.status == L.EDB_ERR_UNSUPPORTED
    with pytest.raises(L.EdbError) as ei:
        edb.packed_bytes(edb.cell_struct(WL.NARY_INTERNAL, 0, 8, 3, L.F32))
    assert ei.value.status == L.EDB_ERR_UNSUPPORTED
    with pytest.raises(L.EdbError) as ei:
        edb.packed_bytes(edb.cell_struct(WL.NARY_LEAF, 8, 8, 0, 5))
    assert ei.value.status == L.EDB_ERR_INVALID
    with pytest.raises(L.EdbError) as ei:
        edb.packed_bytes(edb.cell_struct(WL.NARY_LEAF, 8, 6, 0, L.F32))   # 24-byte rows
    assert ei.value.status == L.EDB_ERR_UNSUPPORTED
    n = C.c_int32()
    assert lib.edb_exec_launches(None, C.byref(n)) == L.EDB_ERR_INVALID
    assert lib.edb_execute(None, None, None, None, None, None) == L.EDB_ERR_INVALID


@pytest.mark.parametrize("k", [1, 2, 3, 4, 5, 6, 7, 8, 9])
@pytest.mark.parametrize("flow", [True, False])
def test_dryrun_launch_list(k, flow):
    w = WL.make_config(k, instances=CFG_INSTANCES[k])
    f = edb.Forward(w, flags=L.DRYRUN | L.USE_GRAPH | (0 if flow else L.NO_FLOW))
    n = f.exec.launches()
    B = f.sched.n_batches
    info0 = f.exec.launch_info(0)
    assert info0["batch"] == -1 and info0["n_batches"] == 0
    # x is staged unless every staged row would be the node's own row of x (then read in
    # place) or a single batch reads x (then through its row list)
    xs = f.plan.x_slot
    in_place = bool((xs >= 0).any()) and bool(np.all(xs[xs >= 0] == w.x_row[xs >= 0]))
    x_batches = sum(WL.KIND_SHAPE[w.kinds[int(t)]][2] for t in f.sched.batch_type)
    staged = 0 if (in_place or x_batches == 1) else int((w.x_row >= 0).sum())
    # with nothing to stage, a first batch without child lists (and no x padding)
    # clears the zero and pad rows itself and the staging launch is dropped
    info1 = f.exec.launch_info(1)
    t0 = int(f.sched.batch_type[0])
    nf0, rg0, hx0 = edb.operand_shapes(w)[t0]
    kg = 16 if w.dtype == "f32" else 32
    folded = (staged == 0 and nf0 == 0 and not rg0 and (not hx0 or w.in_dim % kg == 0)
              and info1["batch"] == 0 and info1["part"] == L.PART_CELL
              and (n < 3 or f.exec.launch_info(2)["batch"] != 0))
    assert info0["grid"] == (0 if folded else (staged + 1 + len(f.plan.pads) + 3) // 4)
    seen = []
    for i in range(1, n):
        info = f.exec.launch_info(i)
        b = info["batch"]
        if info["variant"] == L.FLOW_VARIANT:
            assert flow and info["n_batches"] >= 2 and info["kind"] == -1
            rows = [f.sched.batch_ptr[q + 1] - f.sched.batch_ptr[q] for q in range(b, b + info["n_batches"])]
            assert max(rows) <= 1024 and info["m"] == sum(rows)
            assert 1 <= info["grid"] and info["block"] == 256
            seen += list(range(b, b + info["n_batches"]))
            continue
        t = int(f.sched.batch_type[b])
        assert info["kind"] == w.kinds[t]
        if info["part"] != L.PART_CELL and w.kinds[t] == WL.MV_VEC:
            # MV-RNN vector batch: the matrix-vector products, then (below) its GEMM
            assert info["part"] == L.PART_CHILD_SUM and info["n_batches"] == 0
            assert info["grid"] == (2 * info["m"] + 3) // 4 and info["n"] == 2 * w.hidden
            nxt = f.exec.launch_info(i + 1)
            assert nxt["batch"] == b and nxt["part"] == L.PART_CELL and nxt["k"] >= 2 * w.hidden
            continue
        if info["part"] != L.PART_CELL:
            # child-sum batch on the large tile: the forget GEMM over the batch's
            # children, then the per-parent sums, then (below) the parents
            assert w.kinds[t] == WL.CS_INTERNAL and w.dtype == "bf16" and info["n_batches"] == 0
            nxt = f.exec.launch_info(i + 1)
            assert nxt["batch"] == b and nxt["part"] == info["part"] - 1
            if info["part"] == L.PART_FORGET:
                nodes = f.sched.batch_nodes[f.sched.batch_ptr[b]:f.sched.batch_ptr[b + 1]]
                assert info["m"] == sum(int((w.children(int(v)) >= 0).sum()) for v in nodes)
                assert info["variant"] in L.LARGE_VARIANTS
                assert f.exec.launch_info(i + 2)["variant"] in L.LARGE_VARIANTS
            continue
        assert info["n_batches"] == 1
        assert info["m"] == f.sched.batch_ptr[b + 1] - f.sched.batch_ptr[b]
        assert 0 <= info["variant"] <= L.WS_VARIANT and info["grid"] >= 1 and info["block"] in (256, 512, 1024)
        if info["variant"] == L.WS_VARIANT:
            # weight-stationary tile: bf16 x-only leaves, 512 threads, (units / 32) x (row groups, a multiple of 8)
            assert w.dtype == "bf16" and w.kinds[t] in (WL.NARY_LEAF, WL.CS_LEAF, WL.GRU_LEAF)
            assert info["block"] == 512 and info["grid"] % 8 == 0
        if info["variant"] in L.LARGE_VARIANTS:
            # large tile: every kind but the lattice character cell (child-sum parents run
            # as a forget GEMM, child sums and a parent GEMM), 256 threads, grid a multiple of 8
            assert w.kinds[t] != WL.LAT_CHAR
            assert info["block"] == 256 and info["grid"] % 8 == 0
        segs = f.plan.batch_segments(b)
        assert info["seg_kind"][0] == segs[0][0]
        seen.append(b)
    assert seen == list(range(B))          # every batch exactly once, in schedule order
    if not flow:
        parts = [f.exec.launch_info(i)["part"] for i in range(1, n)]
        assert n == 1 + B + sum(p != L.PART_CELL for p in parts)
    with pytest.raises(L.EdbError):
        f.exec.launch_info(n)


LARGE_TILE_ROWS = {8: 256, 9: 128, 10: 64, 15: 64, 16: 32}      # rows per work-group of the large variants at G = 3
LARGE_TILE_ROWS_G1 = {8: 256, 9: 128, 10: 64, 15: 64, 16: 32}   # the one-gate forget GEMM of child-sum cells
LARGE_TILE_UNITS = {8: 64, 9: 64, 10: 64, 15: 32, 16: 32}       # units per work-group


WS_ROWS, WS_UNITS, WS_MAX_TILES = 256, 32, 8    # rows per row tile, units per work-group, row tiles per work-group


def _ws_grid(m, H, n_cu=256):
    """The weight-stationary launch's grid: unit tiles x row groups, the row groups
    a multiple of 8, about one work-group per CU, at most 8 row tiles each."""
    nut = -(-H // 64) * 64 // WS_UNITS
    nrt = -(-m // WS_ROWS)
    need = -(-nrt // WS_MAX_TILES)
    ngr = max(8, min(n_cu // nut // 8 * 8, -(-nrt // 8) * 8), -(-need // 8) * 8)
    return nut * ngr


def test_weight_stationary_selection_and_grid(monkeypatch):
    """bf16 x-only leaf batches of at least 8192 rows take the weight-stationary
    tile (a forced variant or EDB_NO_LARGE keeps them off it; fp32 never takes
    it), with the grid its kernel assumes, including the row table's bound."""
    monkeypatch.delenv("EDB_VARIANT", raising=False)
    base = L.DRYRUN | L.NO_FLOW
    big = WL.make_config(5)
    f = edb.Forward(big, flags=base)
    info = f.exec.launch_info(1)
    assert info["kind"] == WL.CS_LEAF and info["m"] == 28629 and info["variant"] == L.WS_VARIANT
    assert info["block"] == 512 and info["grid"] == _ws_grid(28629, 512) == 256
    for i in range(2, f.exec.launches()):
        assert f.exec.launch_info(i)["variant"] != L.WS_VARIANT   # internal nodes and small leaf batches
    monkeypatch.setenv("EDB_VARIANT", "9")
    assert edb.Forward(big, flags=base).exec.launch_info(1)["variant"] == 9
    monkeypatch.delenv("EDB_VARIANT")
    # 70,000 leaves of 512 units: 274 row tiles need 40 row groups (8 tiles each at most)
    op, ch, hx = [], [], []
    for t in range(35000):
        op += [0, 0, 1]
        ch += [[], [], [3 * t, 3 * t + 1]]
        hx += [True, True, False]
    w = WL.make_graph([WL.CS_LEAF, WL.CS_INTERNAL], 256, 512, op, ch, hx, seed=3, dtype="bf16")
    info = edb.Forward(w, flags=base).exec.launch_info(1)
    assert info["variant"] == L.WS_VARIANT and info["m"] == 70000
    assert info["grid"] == _ws_grid(70000, 512) == 16 * 40
    # a reduction of one group of four k-groups (K = 128) keeps the other tiles
    k128 = WL.make_graph([WL.CS_LEAF, WL.CS_INTERNAL], 128, 512, op[:3000], ch[:3000], hx[:3000], seed=4,
                         dtype="bf16")
    monkeypatch.setenv("EDB_VARIANT", str(L.WS_VARIANT))
    assert edb.Forward(k128, flags=base).exec.launch_info(1)["variant"] != L.WS_VARIANT
    # a forced weight-stationary tile on a small batch; fp32 keeps the other tiles
    monkeypatch.setenv("EDB_VARIANT", str(L.WS_VARIANT))
    small = WL.make_config(5, instances=12)
    info = edb.Forward(small, flags=base).exec.launch_info(1)
    assert info["variant"] == L.WS_VARIANT and info["grid"] == _ws_grid(info["m"], 512)
    f32 = WL.make_config(2, instances=6)
    f = edb.Forward(f32, flags=base)
    assert all(f.exec.launch_info(i)["variant"] != L.WS_VARIANT for i in range(1, f.exec.launches()))


def test_tile_flags_select_variants():
    """EDB_TILE_LARGE puts every batch the large tile supports on it; EDB_NO_LARGE
    and EDB_NO_SPLIT_K restrict the choice; the two large-tile flags exclude each other."""
    w = WL.make_config(5, instances=12)
    base = L.DRYRUN | L.NO_FLOW
    f = edb.Forward(w, flags=base | L.TILE_LARGE)
    for i in range(1, f.exec.launches()):
        info = f.exec.launch_info(i)
        if info["part"] == L.PART_CHILD_SUM:
            assert info["grid"] == -(-info["m"] * (512 // 8) // 256)
            continue
        assert info["variant"] in L.LARGE_VARIANTS
        rows = LARGE_TILE_ROWS_G1 if info["part"] == L.PART_FORGET else LARGE_TILE_ROWS
        tm = rows[info["variant"]]
        assert info["grid"] == -(-(-(-info["m"] // tm) * (512 // LARGE_TILE_UNITS[info["variant"]])) // 8) * 8
    f = edb.Forward(w, flags=base | L.NO_LARGE | L.NO_SPLIT_K)
    for i in range(1, f.exec.launches()):
        assert f.exec.launch_info(i)["variant"] in (0, 1)
    w2 = WL.make_config(2, instances=6)
    f = edb.Forward(w2, flags=base | L.NO_SPLIT_K)
    for i in range(1, f.exec.launches()):
        assert f.exec.launch_info(i)["variant"] in (0, 1)
    big = WL.make_config(5)
    f = edb.Forward(big, flags=base)
    assert f.exec.launch_info(1)["kind"] == WL.CS_LEAF and f.exec.launch_info(1)["variant"] == L.WS_VARIANT
    f = edb.Forward(big, flags=base | L.NO_LARGE)
    assert f.exec.launch_info(1)["variant"] not in L.LARGE_VARIANTS + (L.WS_VARIANT,)
    with pytest.raises(L.EdbError) as ei:
        edb.Forward(w, flags=base | L.TILE_LARGE | L.NO_LARGE)
    assert ei.value.status == L.EDB_ERR_INVALID


@pytest.mark.parametrize("variant", [11, 12, 13, 14])
def test_forced_streamed_variant(variant, monkeypatch):
    """A forced streamed variant runs on every batch of a kind without a ragged
    phase, 64 * WK threads, one work-group per (16 RT rows, 16 units) tile
    rounded up to a multiple of 8 (the XCD-aware order); batches of ragged
    kinds (lattice characters, child-sum parents) get what forcing the staged
    variant with the same rows and reduction split gives them."""
    rt, wk = {11: (1, 4), 12: (2, 4), 13: (1, 8), 14: (1, 16)}[variant]
    for k in (1, 2, 3, 4, 5):
        w = WL.make_config(k, instances={1: 8, 2: 6, 3: 6, 4: 2, 5: 4}[k])
        monkeypatch.setenv("EDB_VARIANT", str(L.STREAM_STAGED[variant]))
        ref = edb.Forward(w, flags=L.DRYRUN | L.NO_FLOW)
        monkeypatch.setenv("EDB_VARIANT", str(variant))
        f = edb.Forward(w, flags=L.DRYRUN | L.NO_FLOW)
        assert f.exec.launches() == ref.exec.launches()
        hu = -(-w.hidden // 64) * 64
        for i in range(1, f.exec.launches()):
            info = f.exec.launch_info(i)
            if info["kind"] in (WL.LAT_CHAR, WL.CS_INTERNAL):
                assert info["variant"] == ref.exec.launch_info(i)["variant"]
                continue
            assert info["variant"] == variant
            assert info["block"] == 64 * wk
            tiles = -(-info["m"] // (16 * rt)) * (hu // 16)
            assert info["grid"] == -(-tiles // 8) * 8


def test_packed_weight_bytes_layout():
    # main [Hu/16][G][K/KG][64][16 B] + bias, 256-byte aligned
    c = edb.cell_struct(WL.NARY_INTERNAL, 0, 256, 2, L.F32)
    assert edb.packed_bytes(c) == 256 // 16 * 5 * (512 // 16) * 64 * 16 + 5 * 256 * 4
    c = edb.cell_struct(WL.CS_INTERNAL, 0, 512, 0, L.BF16)
    assert edb.packed_bytes(c) == (512 // 16 * 3 * 16 * 1024 + 3 * 512 * 4 + 512 // 16 * 16 * 1024 + 2048)


def test_forward_call_validates_before_any_device_work():
    """edb_forward: an arena smaller than the plan fails with EDB_ERR_INVALID
    (and reports the rows needed) before any HIP call; EDB_DRYRUN is rejected."""
    w = WL.make_config(2, instances=3)
    cells = [edb.cell_struct(k, w.in_dim, w.hidden, w.n_children[t] if k == WL.NARY_INTERNAL else 0, L.F32)
             for t, k in enumerate(w.kinds)]
    fc = edb.ForwardCall(w.op_type, w.child_ptr, w.child_idx, w.x_row, w.n_types, edb.operand_shapes(w), cells)
    with pytest.raises(L.EdbError) as ei:
        fc.call([256, 256], 256, 256, 256, 3, 0)
    assert ei.value.status == L.EDB_ERR_INVALID and "arena" in str(ei.value)
    g = edb.Graph(w.op_type, w.child_ptr, w.child_idx, w.x_row, w.n_types)
    pl = edb.Plan(g, edb.Schedule(g), edb.operand_shapes(w))
    assert fc.n_slots.value == pl.n_slots
    bad = edb.ForwardCall(w.op_type, w.child_ptr, w.child_idx, w.x_row, w.n_types, edb.operand_shapes(w), cells,
                          flags=L.DRYRUN)
    with pytest.raises(L.EdbError) as ei:
        bad.call([256, 256], 256, 256, 256, 10 ** 6, 0)
    assert ei.value.status == L.EDB_ERR_INVALID



@pytest.mark.parametrize("policy", [L.POLICY_TABLE, L.POLICY_AGENDA, L.POLICY_SUFFICIENT, L.POLICY_DEPTH])
def test_forward_call_rejects_cycles_before_any_device_work(policy):
    """edb_forward skips the ingest's own acyclicity check for the frontier
    policies (their schedule finds no ready node while nodes remain and
    reports the cycle); the depth policy keeps the ingest's check.  Either
    way a cycle fails with EDB_ERR_CYCLE before any HIP call.  The graph is a
    valid tree with a two-node cycle beside it."""
    w = WL.make_config(2, instances=2)
    cells = [edb.cell_struct(k, w.in_dim, w.hidden, w.n_children[t] if k == WL.NARY_INTERNAL else 0, L.F32)
             for t, k in enumerate(w.kinds)]
    V = len(w.op_type)
    internal = [t for t, k in enumerate(w.kinds) if k == WL.NARY_INTERNAL][0]
    n_ch = w.n_children[internal]
    # two extra internal nodes, each the other's first child (the rest absent)
    op = np.concatenate([np.asarray(w.op_type, np.int32), np.array([internal, internal], np.int32)])
    kids = [V + 1] + [-1] * (n_ch - 1) + [V] + [-1] * (n_ch - 1)
    idx = np.concatenate([np.asarray(w.child_idx, np.int32), np.array(kids, np.int32)])
    ptr = np.concatenate([np.asarray(w.child_ptr, np.int64),
                          w.child_ptr[-1] + np.array([n_ch, 2 * n_ch], np.int64)])
    xr = np.concatenate([np.asarray(w.x_row, np.int32), np.array([-1, -1], np.int32)])
    fc = edb.ForwardCall(op, ptr, idx, xr, w.n_types, edb.operand_shapes(w), cells, policy=policy)
    with pytest.raises(L.EdbError) as ei:
        fc.call([256, 256], 256, 256, 256, 10 ** 6, 0)
    assert ei.value.status == L.EDB_ERR_CYCLE and "cycle" in str(ei.value)
    # the same graph without the cycle's back edge goes past the ingest and
    # the schedule (it fails later, on the too-small arena)
    idx2 = idx.copy()
    idx2[len(w.child_idx)] = -1
    fc2 = edb.ForwardCall(op, ptr, idx2, xr, w.n_types, edb.operand_shapes(w), cells, policy=policy)
    with pytest.raises(L.EdbError) as ei:
        fc2.call([256, 256], 256, 256, 256, 3, 0)
    assert ei.value.status == L.EDB_ERR_INVALID and "arena" in str(ei.value)



@pytest.mark.parametrize("k", [2, 5])
def test_relabelled_mini_batch_has_the_same_launch_sequence(k):
    """workloads.relabel permutes node ids only: the oracle's states move with
    the permutation, and the executor's launch sequence (kernel kind, variant,
    part, block) is unchanged, so an EDB_USE_GRAPH execution of the relabelled
    mini-batch can reuse a kept graph."""
    from oracle.evaluate import evaluate
    w = WL.make_config(k, instances=2)
    w2, perm = WL.relabel(w, 5)
    assert sorted(perm.tolist()) == list(range(w.n_nodes))
    ref = evaluate(w.kinds, w.op_type, w.child_ptr, w.child_idx, w.x_row, w.x, w.weights, w.hidden,
                   n_fixed=w.n_children, dtype=w.dtype)
    got = evaluate(w2.kinds, w2.op_type, w2.child_ptr, w2.child_idx, w2.x_row, w2.x, w2.weights, w2.hidden,
                   n_fixed=w2.n_children, dtype=w2.dtype)
    for a, b in zip(ref, got):
        np.testing.assert_array_equal(np.asarray(b)[perm], np.asarray(a))

    def seq(v):
        f = edb.Forward(v, flags=L.DRYRUN)
        out = []
        for i in range(f.exec.launches()):
            inf = f.exec.launch_info(i)
            if inf["grid"] > 0:
                out.append((inf["kind"], inf["variant"], inf["part"], inf["block"]))
        return out

    assert seq(w) == seq(w2)


PQ_INSTANCES = {1: 8, 2: 16, 3: 8, 4: 3, 5: 8}


@pytest.mark.parametrize("k", [1, 2, 3, 4, 5])
def test_pq_plan_bit_exact_configs(k):
    """EDB_PLAN_PQ against the oracle's PQ-tree layout (smaller instances:
    the oracle's tree walks are slow)."""
    w = WL.make_config(k, instances=PQ_INSTANCES[k])
    table = edb.LATTICE_TABLE if k == 3 else None
    g = edb.Graph(w.op_type, w.child_ptr, w.child_idx, w.x_row, w.n_types)
    s = edb.Schedule(g, L.POLICY_TABLE, L.ENC_SORT, table)
    shapes = edb.operand_shapes(w)
    pl = edb.Plan(g, s, shapes, L.PLAN_PQ)
    batches, _ = _oracle_schedule(w, OS.POLICY_TABLE, table)
    ref = OP.plan_memory(w.op_type, w.child_ptr, w.child_idx, batches, shapes, OP.PLAN_PQ)
    _compare_plan(pl, ref, batches)
    OP.hazard_check(w.op_type, w.child_ptr, w.child_idx, batches, ref)


@settings(max_examples=400, deadline=None)
@given(random_graphs(), st.sampled_from([OS.POLICY_TABLE, OS.POLICY_DEPTH, OS.POLICY_AGENDA]))
def test_pq_plan_random_graphs_bit_exact(g, policy):
    op, children, T, shapes = g
    ptr = np.zeros(len(children) + 1, dtype=np.int64)
    for v, ch in enumerate(children):
        ptr[v + 1] = ptr[v] + len(ch)
    idx = np.array([c for ch in children for c in ch], dtype=np.int32)
    gr = edb.Graph(op, ptr, idx, np.full(len(op), -1, dtype=np.int32), T)
    s = edb.Schedule(gr, policy)
    batches, _ = OS.schedule(op, ptr, idx, T, policy)
    pl = edb.Plan(gr, s, shapes, L.PLAN_PQ)
    ref = OP.plan_memory(op, ptr, idx, batches, shapes, OP.PLAN_PQ)
    _compare_plan(pl, ref, batches)
    OP.hazard_check(op, ptr, idx, batches, ref)


def test_pq_plan_skipped_list_bit_exact():
    from tests.test_oracle_pq import SKIPPED_LIST_CASE
    op, children = SKIPPED_LIST_CASE
    op = np.array(op, dtype=np.int32)
    ptr = np.zeros(len(children) + 1, dtype=np.int64)
    for v, ch in enumerate(children):
        ptr[v + 1] = ptr[v] + len(ch)
    idx = np.array([c for ch in children for c in ch], dtype=np.int32)
    shapes = [(0, 0, 0), (2, 0, 0)]
    gr = edb.Graph(op, ptr, idx, np.full(len(op), -1, dtype=np.int32), 2)
    s = edb.Schedule(gr, L.POLICY_DEPTH)
    batches, _ = OS.schedule(op, ptr, idx, 2, OS.POLICY_DEPTH)
    pl = edb.Plan(gr, s, shapes, L.PLAN_PQ)
    ref = OP.plan_memory(op, ptr, idx, batches, shapes, OP.PLAN_PQ)
    _compare_plan(pl, ref, batches)
