"""Lattice GRU (config 9): the batched path against the lattice-level oracle
(oracle/latticegru.py), every position's state and every edge's proposal,
on every tile family the kinds run on; plus host-side checks."""
import numpy as np
import pytest

from oracle.compare import normwise_rel_err
from oracle.latticegru import lattice_gru
from paper_2302_03851_amd import _lib as L
from paper_2302_03851_amd import edb, workloads as WL


def _check(w, h, bx=None, bhn=None):
    """Max normwise errors of positions and of edge proposals."""
    a = w.aux
    bx = a["bx"] if bx is None else bx
    bhn = a["bhn"] if bhn is None else bhn
    ep = ee = 0.0
    for lat in a["lattices"]:
        xw = w.x[w.x_row[lat["word_edge"]]] if len(lat["words"]) else np.zeros((0, w.in_dim))
        hp, gc, gw = lattice_gru(lat["length"], lat["words"], w.x[w.x_row[lat["char_edge"]]], xw,
                                 a["Wx"], a["Wh"], bx, bhn)
        ep = max(ep, normwise_rel_err(h[lat["pos"]], hp))
        ee = max(ee, normwise_rel_err(h[lat["char_edge"]], gc))
        if len(lat["words"]):
            ee = max(ee, normwise_rel_err(h[lat["word_edge"]], gw))
    return ep, ee


def test_workload_structure():
    w = WL.make_config(9, instances=3)
    for lat in w.aux["lattices"]:
        pos, ce, we = lat["pos"], lat["char_edge"], lat["word_edge"]
        for j in range(lat["length"]):
            words = [k for k, (s, e) in enumerate(lat["words"]) if e == j]
            assert w.children(int(pos[j])).tolist() == [int(ce[j])] + [int(we[k]) for k in words]
            assert w.children(int(ce[j])).tolist() == [int(pos[j - 1]) if j else -1]
        for k, (s, e) in enumerate(lat["words"]):
            assert e - s + 1 in (2, 3, 4)
            assert w.children(int(we[k])).tolist() == [int(pos[s - 1]) if s else -1]


def test_bf16_rejected():
    import ctypes as C
    nb = C.c_int64()
    for k in (WL.LGRU_EDGE, WL.POOL_MEAN):
        cell = edb.cell_struct(k, 100, 200, 0, L.BF16)
        assert L.load().edb_packed_weight_bytes(C.byref(cell), C.byref(nb)) == L.EDB_ERR_UNSUPPORTED


def test_pool_runs_on_the_staged_tile_only():
    w = WL.make_config(9, instances=4)
    for flags in (L.DRYRUN, L.DRYRUN | L.TILE_LARGE):
        f = edb.Forward(w, flags=flags)
        for i in range(1, f.exec.launches()):
            info = f.exec.launch_info(i)
            if info["kind"] == WL.POOL_MEAN:
                assert 0 <= info["variant"] <= 7


@pytest.mark.gpu
@pytest.mark.parametrize("inst,flags", [(3, 0), (6, L.USE_GRAPH), (32, L.USE_GRAPH), (5, L.TILE_LARGE),
                                        (5, L.NO_LARGE), (5, L.FORCE_GATHER)])
def test_lattice_gru_parity(inst, flags):
    w = WL.make_config(9, instances=inst)
    f = edb.Forward(w, flags=flags)
    f.run()
    h, c = f.states()
    ep, ee = _check(w, h)
    assert ep < 1e-4 and ee < 1e-4, (ep, ee)
    np.testing.assert_array_equal(c, h)


@pytest.mark.gpu
@pytest.mark.parametrize("variant", [0, 3, 6, 11, 13])
def test_lattice_gru_forced_variants(variant, monkeypatch):
    """Every batch on one staged variant, or the edges on a streamed one (the
    pooling batches then take the staged counterpart)."""
    monkeypatch.setenv("EDB_VARIANT", str(variant))
    w = WL.make_config(9, instances=4)
    f = edb.Forward(w, flags=L.NO_LARGE)
    f.run()
    h, _ = f.states()
    ep, ee = _check(w, h)
    assert ep < 1e-4 and ee < 1e-4, (ep, ee)


@pytest.mark.gpu
def test_lattice_gru_biases_and_replays():
    """Non-zero input and candidate biases against the oracle; three graph
    replays equal to the eager run bit for bit."""
    import torch
    w = WL.make_config(9, instances=5)
    H = w.hidden
    rng = np.random.Generator(np.random.PCG64(9))
    bx = rng.uniform(-0.3, 0.3, 3 * H).astype(np.float32)
    bhn = rng.uniform(-0.3, 0.3, H).astype(np.float32)
    w.weights[0]["b"] = np.concatenate([bx, bhn]).astype(np.float32)
    f0 = edb.Forward(w, flags=0)
    f0.run()
    h0, _ = f0.states()
    ep, ee = _check(w, h0, bx, bhn)
    assert ep < 1e-4 and ee < 1e-4, (ep, ee)
    f1 = edb.Forward(w, flags=L.USE_GRAPH)
    for _ in range(3):
        f1.run()
        torch.cuda.synchronize()
        h1, _ = f1.states()
        np.testing.assert_array_equal(h1, h0)


@pytest.mark.gpu
def test_lattice_gru_one_call_path():
    """The full workload through the one-call path the benchmark times
    (edb_forward, eager launches): bitwise equal to a graph replay, which is
    within the bound of the oracle."""
    import torch
    w = WL.make_config(9)
    f = edb.Forward(w, flags=L.USE_GRAPH)
    f.run()
    f.run()
    h, c = f.states()
    ep, ee = _check(w, h)
    assert ep < 1e-4 and ee < 1e-4, (ep, ee)
    fc = edb.ForwardCall(w.op_type, w.child_ptr, w.child_idx, w.x_row, w.n_types, edb.operand_shapes(w), f.cells)
    ah = torch.full_like(f.arena_h, 5.0)
    ac = torch.full_like(f.arena_c, 5.0)
    fc.call([b.data_ptr() for b in f.weights], f.x.data_ptr(), ah.data_ptr(), ac.data_ptr(), ah.shape[0],
            f.stream.cuda_stream)
    torch.cuda.synchronize()
    s = f.plan.slot
    np.testing.assert_array_equal(ah.cpu().numpy()[s], h)
    np.testing.assert_array_equal(ac.cpu().numpy()[s], c)


@pytest.mark.gpu
@pytest.mark.parametrize("variant", [None, 0, 3])
def test_pool_mean_with_map_and_bias(variant, monkeypatch):
    """The pooling node as its kind defines it, h = mean(edges' h) W + b, with
    a non-identity W and non-zero biases in both kinds, against the graph
    oracle (every node)."""
    from oracle.compare import state_rel_err
    from oracle.evaluate import evaluate_workload
    if variant is not None:
        monkeypatch.setenv("EDB_VARIANT", str(variant))
    w = WL.make_config(9, instances=6)
    H = w.hidden
    rng = np.random.Generator(np.random.PCG64(31))
    w.weights[0]["b"] = rng.uniform(-0.3, 0.3, 4 * H).astype(np.float32)
    w.weights[1]["W"] = rng.uniform(-0.15, 0.15, (H, H)).astype(np.float32)
    w.weights[1]["b"] = rng.uniform(-0.5, 0.5, H).astype(np.float32)
    f = edb.Forward(w, flags=L.NO_LARGE)
    f.run()
    h, c = f.states()
    hr, cr = evaluate_workload(w)
    err = state_rel_err(h, c, hr, cr)
    print(f"pool with map and bias, variant {variant}: err {err:.3e}", flush=True)
    assert err < 1e-4, err
