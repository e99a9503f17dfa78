"""The allocation-free entry point (edb_forward_noalloc) through the C ABI:
bitwise the arena of edb_forward on the same mini-batch, on two calls in a
row (the second with a smaller mini-batch, so the fixed device array holds
the first call's contents when the second starts), with the oracle's states
at every node; and a mini-batch whose device memory exceeds the array is
rejected before anything runs."""
import numpy as np
import pytest

from oracle.compare import state_rel_err
from oracle_instances import evaluate_by_instance
from paper_2302_03851_amd import _lib as L
from paper_2302_03851_amd import workloads as WL

pytestmark = pytest.mark.gpu

TOL = {"f32": 1e-4, "bf16": 2e-2}


def _torch():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


def _arenas(torch, f, fill):
    return torch.full_like(f.arena_h, fill), torch.full_like(f.arena_c, -fill)


def _compare(torch, w, f, fc, call):
    """Run edb_forward and edb_forward_noalloc (`call`) on fresh arenas;
    return both node-ordered (h, c)."""
    a_ref = _arenas(torch, f, 3.0)
    a_na = _arenas(torch, f, 7.0)
    wp = [b.data_ptr() for b in f.weights]
    st = f.stream.cuda_stream
    fc.call(wp, f.x.data_ptr(), a_ref[0].data_ptr(), a_ref[1].data_ptr(), a_ref[0].shape[0], st)
    call(wp, f.x.data_ptr(), a_na[0].data_ptr(), a_na[1].data_ptr(), a_na[0].shape[0], st)
    torch.cuda.synchronize()
    s = f.plan.slot
    out = []
    for ah, ac in (a_ref, a_na):
        out.append((ah.float().cpu().numpy().astype(np.float64)[s], ac.cpu().numpy().astype(np.float64)[s]))
    return out


@pytest.mark.parametrize("k,inst,inst_small", [(2, None, 16), (4, None, 8), (5, 40, 10), (3, None, 8), (8, None, 16)])
def test_noalloc_matches_forward_two_calls(k, inst, inst_small):
    torch = _torch()
    from paper_2302_03851_amd import edb
    big = WL.make_config(k, instances=inst)
    small = WL.make_config(k, instances=inst_small)
    assert small.n_nodes < big.n_nodes
    for w in (big, small):
        f = edb.Forward(w)
        fc = edb.ForwardCall(w.op_type, w.child_ptr, w.child_idx, w.x_row, w.n_types, edb.operand_shapes(w),
                             f.cells, table=edb.LATTICE_TABLE if k == 3 else None)
        (h0, c0), (h1, c1) = _compare(torch, w, f, fc, fc.call_noalloc)
        print(f"noalloc k={k} V={w.n_nodes}", flush=True)
        np.testing.assert_array_equal(h1, h0)
        np.testing.assert_array_equal(c1, c0)
        if w.aux is None:   # MV-RNN: its own oracle runs in tests/test_mvrnn.py
            hr, cr = evaluate_by_instance(w)
            rows = np.array([w.kinds[t] != WL.LAT_WORD for t in w.op_type])
            assert state_rel_err(h1, c1, hr, cr, h_rows=rows) <= TOL[w.dtype]


def test_noalloc_rejects_oversized_and_bad_flags():
    torch = _torch()
    from paper_2302_03851_amd import edb
    w = WL.make_config(5)            # 52k nodes: about 68 MB of child-sum scratch rows, twice the array
    f = edb.Forward(w)
    fc = edb.ForwardCall(w.op_type, w.child_ptr, w.child_idx, w.x_row, w.n_types, edb.operand_shapes(w), f.cells)
    ah, ac = _arenas(torch, f, 5.0)
    with pytest.raises(L.EdbError) as ei:
        fc.call_noalloc([b.data_ptr() for b in f.weights], f.x.data_ptr(), ah.data_ptr(), ac.data_ptr(),
                        ah.shape[0], f.stream.cuda_stream)
    assert ei.value.status == L.EDB_ERR_UNSUPPORTED and "scratch" in str(ei.value)
    torch.cuda.synchronize()
    assert bool((ah == 5.0).all()) and bool((ac == -5.0).all())   # nothing ran
    fg = edb.ForwardCall(w.op_type, w.child_ptr, w.child_idx, w.x_row, w.n_types, edb.operand_shapes(w), f.cells,
                         flags=L.PROFILE)
    with pytest.raises(L.EdbError) as ei:
        fg.call_noalloc([b.data_ptr() for b in f.weights], f.x.data_ptr(), ah.data_ptr(), ac.data_ptr(),
                        ah.shape[0], f.stream.cuda_stream)
    assert ei.value.status == L.EDB_ERR_INVALID
