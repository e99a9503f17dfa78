"""Diagnostics: the split-phase copies (edb_split_phase) against a host
simulation of the same row copies, and the roofline probes (edb_probe_copy
copies bit-exactly; edb_probe_mfma's sums equal the product the MFMA lane
layout defines)."""
import numpy as np
import pytest

from paper_2302_03851_amd import _lib as L
from paper_2302_03851_amd import edb, workloads as WL


def _align16(v):
    return (v + 15) // 16 * 16


def _lists(plan, b):
    """Result list, then the operand lists of batch b (None = absent)."""
    out = []
    for kind, base, off, n in plan.segs[plan.seg_ptr[b]:plan.seg_ptr[b + 1]]:
        if kind == L.SEG_NONE:
            out.append(None)
        elif kind == L.SEG_CONTIG:
            out.append(np.arange(base, base + n))
        else:
            out.append(plan.idx_pool[off:off + n])
    return out


def simulate(f, ah, ac, xb, buf):
    """The split-phase copies on host byte arrays, in schedule order: the
    gather writes x rows, then per operand list its h rows and its c rows,
    densely (each list 16-byte aligned); the scatter copies m h rows and m c
    rows from the start of the buffer into the result slots.  Returns the
    buffer bytes the largest batch needs."""
    w, plan, sched = f.w, f.plan, f.sched
    esz = 2 if w.dtype == "bf16" else 4
    H = w.hidden
    shapes = edb.operand_shapes(w)
    need = 16
    for b in range(sched.n_batches):
        t = int(sched.batch_type[b])
        p0, p1 = int(sched.batch_ptr[b]), int(sched.batch_ptr[b + 1])
        nodes = plan.order[p0:p1]
        m = p1 - p0
        off = 0

        def put(rows):
            nonlocal off
            flat = rows.reshape(-1)
            if buf is not None:
                buf[off:off + flat.size] = flat
            off = _align16(off + flat.size)

        lists = _lists(plan, b)
        if shapes[t][2] and xb is not None:
            put(xb[w.x_row[nodes]])
        elif shapes[t][2]:
            off = _align16(m * w.in_dim * esz)
        for lst in lists[1:]:
            if lst is not None and len(lst):
                if ah is not None:
                    put(ah[lst])
                    put(ac[lst])
                else:
                    off = _align16(_align16(off + len(lst) * H * esz) + len(lst) * H * 4)
        hb = _align16(m * H * esz)
        need = max(need, off, hb + _align16(m * H * 4))
        if ah is not None:
            res = lists[0]
            newh = buf[:m * H * esz].reshape(m, H * esz).copy()
            newc = buf[hb:hb + m * H * 4].reshape(m, H * 4).copy()
            ah[res] = newh
            ac[res] = newc
    return need


SPLIT_CASES = [(1, 3), (2, 4), (3, 3), (4, 2), (5, 3), (6, 4), (7, 4)]


@pytest.mark.parametrize("k,inst", SPLIT_CASES)
def test_split_phase_bytes(k, inst):
    """Buffer size of a dry-run executor = the largest batch's dense lists."""
    w = WL.make_config(k, instances=inst)
    f = edb.Forward(w, flags=L.DRYRUN)
    assert f.exec.split_phase_bytes() == simulate(f, None, None, None, None)


@pytest.mark.gpu
@pytest.mark.parametrize("k,inst", SPLIT_CASES + [(5, 24)])
def test_split_phase_copies(k, inst):
    """Every batch's gather and scatter move exactly the rows the simulation
    moves (arenas and the final buffer compared byte for byte); (5, 24) puts
    child-sum batches on the large tile, whose descriptors the diagnostic
    takes from the child-sum part."""
    import torch
    w = WL.make_config(k, instances=inst)
    f = edb.Forward(w, flags=L.USE_GRAPH)
    f.run()
    torch.cuda.synchronize()
    ah = f.arena_h.view(torch.uint8).cpu().numpy().copy()
    ac = f.arena_c.view(torch.uint8).cpu().numpy().copy()
    xb = f.x.view(torch.uint8).cpu().numpy()
    nb = f.exec.split_phase_bytes()
    buf = torch.zeros(nb, dtype=torch.uint8, device="cuda")
    B = f.sched.n_batches
    ms = f.exec.split_phase(f.x.data_ptr(), f.arena_h.data_ptr(), f.arena_c.data_ptr(), buf.data_ptr(), nb,
                            f.stream.cuda_stream, B)
    torch.cuda.synchronize()
    assert ms.shape == (B, 2) and np.all(np.isfinite(ms)) and np.all(ms >= 0)
    hbuf = np.zeros(nb, dtype=np.uint8)
    assert simulate(f, ah, ac, xb, hbuf) == nb
    np.testing.assert_array_equal(buf.cpu().numpy(), hbuf)
    np.testing.assert_array_equal(f.arena_h.view(torch.uint8).cpu().numpy(), ah)
    np.testing.assert_array_equal(f.arena_c.view(torch.uint8).cpu().numpy(), ac)


@pytest.mark.gpu
def test_split_phase_errors():
    import torch
    w = WL.make_config(2, instances=2)
    f = edb.Forward(w, flags=L.USE_GRAPH)
    nb = f.exec.split_phase_bytes()
    buf = torch.zeros(nb, dtype=torch.uint8, device="cuda")
    B = f.sched.n_batches
    with pytest.raises(L.EdbError, match="edb_execute first"):
        f.exec.split_phase(f.x.data_ptr(), f.arena_h.data_ptr(), f.arena_c.data_ptr(), buf.data_ptr(), nb,
                           f.stream.cuda_stream, B)
    f.run()
    with pytest.raises(L.EdbError, match="needed"):
        f.exec.split_phase(f.x.data_ptr(), f.arena_h.data_ptr(), f.arena_c.data_ptr(), buf.data_ptr(), nb - 16,
                           f.stream.cuda_stream, B)
    torch.cuda.synchronize()


@pytest.mark.gpu
@pytest.mark.parametrize("nbytes,wg", [(16, 1), (16 * 1000003, 64), (1 << 24, 4096)])
def test_probe_copy_exact(nbytes, wg):
    import torch
    st = torch.cuda.current_stream().cuda_stream
    g = torch.Generator(device="cpu").manual_seed(nbytes)
    src = torch.randint(0, 256, (nbytes,), dtype=torch.uint8, generator=g).cuda()
    dst = torch.zeros(nbytes + 64, dtype=torch.uint8, device="cuda")
    ms = edb.probe_copy(src.data_ptr(), dst.data_ptr(), nbytes, wg, st)
    assert ms > 0
    assert torch.equal(dst[:nbytes], src)
    assert int(dst[nbytes:].sum()) == 0   # nothing past the end


def _probe_expected(bf16, iters):
    """Per thread of a work-group: 8 chains x iters x the 4 entries of the
    lane's D fragment, with D = A B over the operands each lane supplies.
    Layouts (16x16 output, k split in 4 groups of lanes): A[i][k] comes from
    lane i + 16*(k // KL), B[k][j] from lane j + 16*(k // KL), D[4*(l // 16) + v][l % 16]
    is register v of lane l; KL = 1 (f32, 16x16x4) or 8 (bf16, 16x16x32, entry k % 8 of the lane's vector)."""
    out = np.zeros(256)
    for wv in range(4):
        t = 64 * wv + np.arange(64)
        if bf16:
            K = 32
            A = np.zeros((16, K))
            Bm = np.zeros((K, 16))
            for kk in range(K):
                for r in range(16):
                    lane = r + 16 * (kk // 8)
                    A[r, kk] = 0.125 * ((t[lane] + kk % 8) & 7)
                    Bm[kk, r] = 0.0625 * ((t[lane] * 3 + kk % 8) & 15)
        else:
            K = 4
            A = np.zeros((16, K))
            Bm = np.zeros((K, 16))
            for kk in range(K):
                for r in range(16):
                    lane = r + 16 * kk
                    A[r, kk] = 0.125 * (t[lane] & 7)
                    Bm[kk, r] = 0.0625 * ((t[lane] * 3) & 15)
        D = A @ Bm
        for lane in range(64):
            out[64 * wv + lane] = 8 * iters * sum(D[4 * (lane // 16) + v, lane % 16] for v in range(4))
    return out


@pytest.mark.gpu
@pytest.mark.parametrize("bf16", [False, True])
def test_probe_mfma_values(bf16):
    import torch
    st = torch.cuda.current_stream().cuda_stream
    n_wg, iters = 3, 5
    out = torch.full((n_wg * 256,), -1.0, dtype=torch.float32, device="cuda")
    ms = edb.probe_mfma(L.BF16 if bf16 else L.F32, n_wg, iters, out.data_ptr(), st)
    assert ms > 0
    exp = _probe_expected(bf16, iters)
    got = out.cpu().numpy().reshape(n_wg, 256)
    for g in range(n_wg):
        np.testing.assert_array_equal(got[g], exp.astype(np.float32))


def test_probe_argument_checks():
    """Rejected on the host before any launch (no GPU needed)."""
    ms = np.zeros(1, dtype=np.float32)
    lib = L.load()
    import ctypes as C
    msp = ms.ctypes.data_as(C.POINTER(C.c_float))
    assert lib.edb_probe_mfma(7, 1, 1, C.cast(C.c_void_p(16), C.POINTER(C.c_float)), None, msp) == L.EDB_ERR_INVALID
    assert lib.edb_probe_mfma(L.F32, 0, 1, C.cast(C.c_void_p(16), C.POINTER(C.c_float)), None, msp) == L.EDB_ERR_INVALID
    assert lib.edb_probe_copy(C.c_void_p(16), C.c_void_p(32), 24, 1, None, msp) == L.EDB_ERR_INVALID
    assert lib.edb_probe_copy(None, C.c_void_p(32), 32, 1, None, msp) == L.EDB_ERR_INVALID
