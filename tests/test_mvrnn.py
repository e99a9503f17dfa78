"""MV-RNN (config 8): the batched path against the tree-level oracle
(oracle/mvrnn.py), node vectors and every column of every node matrix, on
every tile family; plus the host-side checks that need no GPU."""
import numpy as np
import pytest

from oracle.compare import normwise_rel_err
from oracle.mvrnn import mvrnn
from paper_2302_03851_amd import _lib as L
from paper_2302_03851_amd import edb, workloads as WL


def _reference(w):
    a = w.aux
    weights = w.weights
    return mvrnn(a["tree_left"], a["tree_right"], a["leaf_vec"], a["leaf_mat"], weights[2]["W"].T,
                 weights[2]["b"], weights[1]["W_M"].T)


def _split(w, h):
    """Node-ordered states -> per tree node (vector, matrix)."""
    a = w.aux
    d = w.hidden
    vec = h[a["vec_node"]]
    cols = h[a["mat_node"][:, None] + np.arange(d)[None, :]]    # [n_tree, j, :] = column j
    return vec, np.transpose(cols, (0, 2, 1))


def test_workload_structure():
    """Each tree node is d column nodes then a vector node; every vector node
    lists its children's vectors, then the left matrix's columns, then the
    right matrix's."""
    w = WL.make_config(8, instances=2)
    a, d = w.aux, w.hidden
    for t in range(len(a["tree_left"])):
        v, m0 = int(a["vec_node"][t]), int(a["mat_node"][t])
        assert v == m0 + d
        l, r = int(a["tree_left"][t]), int(a["tree_right"][t])
        ch = w.children(v)
        if l < 0:
            assert len(ch) == 0 and w.kinds[w.op_type[v]] == WL.LINEAR
            np.testing.assert_array_equal(w.x[w.x_row[v]], a["leaf_vec"][t])
            np.testing.assert_array_equal(w.x[w.x_row[m0 + 3]], a["leaf_mat"][t][:, 3])
        else:
            assert w.kinds[w.op_type[v]] == WL.MV_VEC
            ml, mr = int(a["mat_node"][l]), int(a["mat_node"][r])
            assert ch.tolist() == [int(a["vec_node"][l]), int(a["vec_node"][r])] + \
                list(range(ml, ml + d)) + list(range(mr, mr + d))
            assert w.children(m0 + 5).tolist() == [ml + 5, mr + 5]


def test_bf16_rejected():
    import ctypes as C
    nb = C.c_int64()
    for k in (WL.LINEAR, WL.MV_MAT, WL.MV_VEC):
        cell = edb.cell_struct(k, 64, 64, 0, L.BF16)
        assert L.load().edb_packed_weight_bytes(C.byref(cell), C.byref(nb)) == L.EDB_ERR_UNSUPPORTED
        cell = edb.cell_struct(k, 64, 64, 0, L.F32)
        assert L.load().edb_packed_weight_bytes(C.byref(cell), C.byref(nb)) == L.EDB_OK


def test_prepare_rejects_wrong_column_count():
    """An MV_VEC node must list exactly 2 * hidden matrix columns."""
    d = 16
    # two leaves (vector node + d column nodes each), then the parent's columns and vector
    op, ch, hx = [], [], []
    leaf_vec, leaf_mat0 = [], []
    for _ in range(2):
        leaf_mat0.append(len(op))
        for _j in range(d):
            op.append(0); ch.append([]); hx.append(True)
        leaf_vec.append(len(op))
        op.append(0); ch.append([]); hx.append(True)
    for j in range(d):
        op.append(1); ch.append([leaf_mat0[0] + j, leaf_mat0[1] + j]); hx.append(False)
    cols = [leaf_mat0[0] + j for j in range(d)] + [leaf_mat0[1] + j for j in range(d - 1)]   # one short
    op.append(2); ch.append(leaf_vec + cols); hx.append(False)
    w = WL.make_graph([WL.LINEAR, WL.MV_MAT, WL.MV_VEC], d, d, op, ch, hx)
    with pytest.raises(L.EdbError, match="2 \\* hidden"):
        edb.Forward(w, flags=L.DRYRUN)


@pytest.mark.gpu
@pytest.mark.parametrize("inst,flags", [(2, 0), (3, L.USE_GRAPH), (8, L.USE_GRAPH), (4, L.TILE_LARGE),
                                        (4, L.NO_LARGE), (5, L.FORCE_GATHER)])
def test_mvrnn_parity(inst, flags):
    w = WL.make_config(8, instances=inst)
    f = edb.Forward(w, flags=flags)
    f.run()
    h, c = f.states()
    V, M = _reference(w)
    gv, gm = _split(w, h)
    d = w.hidden
    ev = normwise_rel_err(gv, V)
    em = normwise_rel_err(np.transpose(gm, (0, 2, 1)).reshape(-1, d), np.transpose(M, (0, 2, 1)).reshape(-1, d))
    print(f"MV-RNN instances={inst} flags={flags}: vectors {ev:.2e}, matrix columns {em:.2e}")
    assert ev < 1e-4 and em < 1e-4
    np.testing.assert_array_equal(c, h)     # c mirrors h for the MV-RNN kinds


@pytest.mark.gpu
@pytest.mark.parametrize("variant", [0, 3, 6, 11, 13])
def test_mvrnn_forced_variants(variant, monkeypatch):
    """Every batch on one staged (0, 3, 6) or streamed (11, 13) tile variant."""
    monkeypatch.setenv("EDB_VARIANT", str(variant))
    w = WL.make_config(8, instances=3)
    f = edb.Forward(w, flags=L.NO_LARGE)
    used = {f.exec.launch_info(i)["variant"] for i in range(1, f.exec.launches())} - {-1}
    assert used == {variant}
    f.run()
    h, _ = f.states()
    V, M = _reference(w)
    gv, gm = _split(w, h)
    d = w.hidden
    assert normwise_rel_err(gv, V) < 1e-4
    assert normwise_rel_err(np.transpose(gm, (0, 2, 1)).reshape(-1, d), np.transpose(M, (0, 2, 1)).reshape(-1, d)) < 1e-4


@pytest.mark.gpu
def test_mvrnn_bias_and_replays():
    """A non-zero vector bias against the oracle, and three graph replays equal
    to the eager run bit for bit."""
    import torch
    w = WL.make_config(8, instances=3)
    rng = np.random.Generator(np.random.PCG64(5))
    w.weights[2]["b"] = rng.uniform(-0.3, 0.3, w.hidden).astype(np.float32)
    f0 = edb.Forward(w, flags=0)
    f0.run()
    h0, _ = f0.states()
    V, M = _reference(w)
    gv, gm = _split(w, h0)
    d = w.hidden
    assert normwise_rel_err(gv, V) < 1e-4
    assert normwise_rel_err(np.transpose(gm, (0, 2, 1)).reshape(-1, d), np.transpose(M, (0, 2, 1)).reshape(-1, d)) < 1e-4
    f1 = edb.Forward(w, flags=L.USE_GRAPH)
    for _ in range(3):
        f1.run()
        torch.cuda.synchronize()
        h1, _ = f1.states()
        np.testing.assert_array_equal(h1, h0)


@pytest.mark.gpu
def test_mvrnn_full_size_and_one_call_path():
    """The full workload (64 trees, 251 k graph nodes) in the benchmark's
    configurations: graph replay against the oracle on every tree node, and
    the one-call path (edb_forward, eager launches) bitwise equal to it."""
    import torch
    w = WL.make_config(8)
    f = edb.Forward(w, flags=L.USE_GRAPH)
    f.run()
    f.run()
    h, c = f.states()
    V, M = _reference(w)
    gv, gm = _split(w, h)
    d = w.hidden
    assert normwise_rel_err(gv, V) < 1e-4
    assert normwise_rel_err(np.transpose(gm, (0, 2, 1)).reshape(-1, d), np.transpose(M, (0, 2, 1)).reshape(-1, d)) < 1e-4
    fc = edb.ForwardCall(w.op_type, w.child_ptr, w.child_idx, w.x_row, w.n_types, edb.operand_shapes(w), f.cells)
    ah = torch.full_like(f.arena_h, 5.0)
    ac = torch.full_like(f.arena_c, 5.0)
    fc.call([b.data_ptr() for b in f.weights], f.x.data_ptr(), ah.data_ptr(), ac.data_ptr(), ah.shape[0],
            f.stream.cuda_stream)
    torch.cuda.synchronize()
    s = f.plan.slot
    np.testing.assert_array_equal(ah.cpu().numpy()[s], h)
    np.testing.assert_array_equal(ac.cpu().numpy()[s], c)
