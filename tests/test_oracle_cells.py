"""Pins of the oracle's cell equations against things other than itself:
library routines (torch.nn.LSTM in float64), closed forms with zero weights,
symmetries and exact rational hand values.  CPU only."""
import math

import numpy as np
import pytest
import torch

from oracle import cells as C
from oracle.evaluate import evaluate, evaluate_workload, round_to_bf16, topo_order
from paper_2302_03851_amd import workloads as WL


def torch_lstm(xs, W_ih, W_hh, b, h0=None, c0=None):
    """Reference: torch.nn.LSTM (float64, CPU), gates [i, f, g, o].
    W_ih [4H, E], W_hh [4H, H], b [4H]; returns h, c per step [T, H]."""
    H = W_hh.shape[1]
    E = W_ih.shape[1]
    m = torch.nn.LSTM(E, H, batch_first=False).double()
    with torch.no_grad():
        m.weight_ih_l0.copy_(torch.from_numpy(np.ascontiguousarray(W_ih, dtype=np.float64)))
        m.weight_hh_l0.copy_(torch.from_numpy(np.ascontiguousarray(W_hh, dtype=np.float64)))
        m.bias_ih_l0.copy_(torch.from_numpy(np.asarray(b, dtype=np.float64)))
        m.bias_hh_l0.zero_()
    hs, cs = [], []
    h = torch.zeros(1, 1, H, dtype=torch.float64) if h0 is None else torch.from_numpy(h0).reshape(1, 1, H)
    c = torch.zeros(1, 1, H, dtype=torch.float64) if c0 is None else torch.from_numpy(c0).reshape(1, 1, H)
    with torch.no_grad():
        for t in range(xs.shape[0]):
            xt = torch.from_numpy(np.asarray(xs[t:t + 1], dtype=np.float64)).reshape(1, 1, E)
            _, (h, c) = m(xt, (h, c))
            hs.append(h.reshape(H).numpy().copy())
            cs.append(c.reshape(H).numpy().copy())
    return np.array(hs), np.array(cs)


def chain_graph(L, t=0, children_of=lambda prev: [prev]):
    op, ch = [], []
    prev = -1
    for i in range(L):
        op.append(t)
        ch.append(children_of(prev))
        prev = i
    return op, ch


def test_p1_chain_equals_torch_lstm():
    w = WL.make_config(1, instances=3)
    # non-zero biases exercise the bias path
    rng = np.random.default_rng(7)
    w.weights[0]["b"] = rng.uniform(-0.5, 0.5, size=4 * w.hidden).astype(np.float32)
    hs, cs = evaluate_workload(w)
    W, b = w.weights[0]["W"].astype(np.float64), w.weights[0]["b"]
    E = w.in_dim
    # walk each chain
    starts = [v for v in range(w.n_nodes) if w.children(v)[0] < 0]
    ends = starts[1:] + [w.n_nodes]
    for s, e in zip(starts, ends):
        xs = w.x[w.x_row[s:e]]
        rh, rc = torch_lstm(xs, W[:E].T, W[E:].T, b)
        np.testing.assert_allclose(hs[s:e], rh, rtol=0, atol=1e-12)
        np.testing.assert_allclose(cs[s:e], rc, rtol=0, atol=1e-12)


def test_p2_lattice_without_words_equals_lstm():
    E, H = 6, 5
    op, ch = chain_graph(9)
    w = WL.make_graph([WL.LAT_CHAR, WL.LAT_WORD], E, H, op, ch, [True] * 9, seed=3, scale=0.4,
                      bias_scale=0.3)
    hs, cs = evaluate_workload(w)
    Wc, b = w.weights[0]["W"].astype(np.float64), w.weights[0]["b"].astype(np.float64)
    blk = lambda a, g: a[..., g * H:(g + 1) * H]
    # lattice gates [i, f, o, u] -> LSTM gates [i, f, g=u, o]
    perm = lambda a: np.concatenate([blk(a, 0), blk(a, 1), blk(a, 3), blk(a, 2)], axis=-1)
    Wl, bl = perm(Wc), perm(b)
    rh, rc = torch_lstm(w.x, Wl[:E].T, Wl[E:].T, bl)
    np.testing.assert_allclose(hs, rh, rtol=0, atol=1e-12)
    np.testing.assert_allclose(cs, rc, rtol=0, atol=1e-12)


@pytest.mark.parametrize("axis", ["row", "col"])
def test_p3_grid_line_equals_lstm(axis):
    E, H, n = 4, 3, 8
    if axis == "row":
        op, ch = chain_graph(n, children_of=lambda p: [p, -1])
    else:
        op, ch = chain_graph(n, children_of=lambda p: [-1, p])
    w = WL.make_graph([WL.GRID], E, H, op, ch, [True] * n, seed=11, scale=0.5, bias_scale=0.4)
    hs, cs = evaluate_workload(w)
    W, b = w.weights[0]["W"].astype(np.float64), w.weights[0]["b"].astype(np.float64)
    blk = lambda a, g: a[..., g * H:(g + 1) * H]
    fg = 1 if axis == "row" else 2         # f_left or f_top
    perm = lambda a: np.concatenate([blk(a, 0), blk(a, fg), blk(a, 4), blk(a, 3)], axis=-1)
    rows = slice(E, E + H) if axis == "row" else slice(E + H, E + 2 * H)
    rh, rc = torch_lstm(w.x, perm(W[:E]).T, perm(W[rows]).T, perm(b))
    np.testing.assert_allclose(hs, rh, rtol=0, atol=1e-12)
    np.testing.assert_allclose(cs, rc, rtol=0, atol=1e-12)


def test_p4_unary_childsum_chain_equals_lstm():
    E, H, L = 3, 4, 7
    op = [0] + [1] * L
    ch = [[]] + [[i] for i in range(L)]
    w = WL.make_graph([WL.CS_LEAF, WL.CS_INTERNAL], E, H, op, ch, [True] + [False] * L,
                      seed=5, scale=0.6, bias_scale=0.4)
    hs, cs = evaluate_workload(w)
    p = w.weights[1]
    Ui, Uf = p["U_iou"].astype(np.float64), p["U_f"].astype(np.float64)
    bi, bf = p["b_iou"].astype(np.float64), p["b_f"].astype(np.float64)
    blk = lambda a, g: a[..., g * H:(g + 1) * H]
    W_hh = np.concatenate([blk(Ui, 0), Uf, blk(Ui, 2), blk(Ui, 1)], axis=1)
    bb = np.concatenate([blk(bi, 0), bf, blk(bi, 2), blk(bi, 1)])
    rh, rc = torch_lstm(np.zeros((L, 1)), np.zeros((4 * H, 1)), W_hh.T, bb, h0=hs[0].copy(), c0=cs[0].copy())
    np.testing.assert_allclose(hs[1:], rh, rtol=0, atol=1e-12)
    np.testing.assert_allclose(cs[1:], rc, rtol=0, atol=1e-12)


@pytest.mark.parametrize("pos", [0, 1])
def test_p4b_nary_one_sided_chain_equals_lstm(pos):
    """An N-ary internal chain whose other child is absent is an LSTM with zero
    input over the present child's U row block, forget gate f_pos."""
    E, H, L = 3, 4, 6
    op = [0] + [1] * L
    ch = [[]] + [([i, -1] if pos == 0 else [-1, i]) for i in range(L)]
    w = WL.make_graph([WL.NARY_LEAF, WL.NARY_INTERNAL], E, H, op, ch, [True] + [False] * L,
                      seed=9, scale=0.6, bias_scale=0.4)
    hs, cs = evaluate_workload(w)
    U, b = w.weights[1]["W"].astype(np.float64), w.weights[1]["b"].astype(np.float64)
    blk = lambda a, g: a[..., g * H:(g + 1) * H]
    perm = lambda a: np.concatenate([blk(a, 0), blk(a, 1 + pos), blk(a, 4), blk(a, 3)], axis=-1)
    W_hh = perm(U[pos * H:(pos + 1) * H])
    rh, rc = torch_lstm(np.zeros((L, 1)), np.zeros((4 * H, 1)), W_hh.T, perm(b),
                        h0=hs[0].copy(), c0=cs[0].copy())
    np.testing.assert_allclose(hs[1:], rh, rtol=0, atol=1e-12)
    np.testing.assert_allclose(cs[1:], rc, rtol=0, atol=1e-12)


def test_p5_nary_child_swap_symmetry():
    w = WL.make_config(2, instances=3)
    rng = np.random.default_rng(1)
    H = w.hidden
    w.weights[1]["b"] = rng.uniform(-0.3, 0.3, size=5 * H).astype(np.float32)
    hs, cs = evaluate_workload(w)
    U = w.weights[1]["W"]
    U2 = np.concatenate([U[H:2 * H], U[:H]], axis=0)
    blk = lambda a, g: a[..., g * H:(g + 1) * H]
    sw = lambda a: np.concatenate([blk(a, 0), blk(a, 2), blk(a, 1), blk(a, 3), blk(a, 4)], axis=-1)
    U2 = sw(U2)
    b2 = sw(w.weights[1]["b"])
    idx = w.child_idx.copy()
    for v in range(w.n_nodes):
        s, e = w.child_ptr[v], w.child_ptr[v + 1]
        if e - s == 2:
            idx[s], idx[s + 1] = idx[s + 1], idx[s]
    w2 = WL.Workload(**{**w.__dict__, "child_idx": idx,
                        "weights": [w.weights[0], {"W": U2, "b": b2}]})
    hs2, cs2 = evaluate_workload(w2)
    np.testing.assert_allclose(hs2, hs, rtol=0, atol=1e-12)
    np.testing.assert_allclose(cs2, cs, rtol=0, atol=1e-12)


def test_p5_hand_values_h1_tree():
    """H = E = 1, zero weights, biases ln 3 (sigma = 3/4), ln 2 (tanh = 3/5) and
    0 (sigma = 1/2): leaf c = 3/4 * 3/5 = 9/20; root with forget gates 3/4 and
    1/2 has c = 9/20 + 3/4 * 9/20 + 1/2 * 9/20 = 81/80."""
    ln2, ln3 = math.log(2.0), math.log(3.0)
    w = WL.make_graph([WL.NARY_LEAF, WL.NARY_INTERNAL], 1, 1, [0, 0, 1], [[], [], [0, 1]],
                      [True, True, False], scale=0.0)
    w.weights[0]["W"][:] = 0
    w.weights[0]["b"][:] = np.array([ln3, ln3, ln2], dtype=np.float32)
    w.weights[1]["W"][:] = 0
    w.weights[1]["b"][:] = np.array([ln3, ln3, 0.0, ln3, ln2], dtype=np.float32)
    # the biases were rounded to fp32; the exact values follow from those
    bl = w.weights[0]["b"].astype(np.float64)
    br = w.weights[1]["b"].astype(np.float64)
    hs, cs = evaluate_workload(w)
    s = lambda z: 1 / (1 + math.exp(-z))
    leaf_c = s(bl[0]) * math.tanh(bl[2])
    assert abs(leaf_c - 9 / 20) < 1e-7
    root_c = s(br[0]) * math.tanh(br[4]) + (s(br[1]) + s(br[2])) * leaf_c
    assert abs(root_c - 81 / 80) < 1e-7
    assert abs(cs[2, 0] - 81 / 80) < 1e-6
    assert abs(cs[0, 0] - 9 / 20) < 1e-7
    assert abs(hs[2, 0] - 0.75 * math.tanh(81 / 80)) < 1e-6


def _biases(kind, H, rng, E=4):
    return {n: rng.uniform(-1.0, 1.0, size=s).astype(np.float32)
            for n, s in WL.weight_shapes(kind, E, H) if n.startswith("b")}


def test_p6_zero_weight_chain_closed_form():
    H, L = 3, 9
    op, ch = chain_graph(L)
    w = WL.make_graph([WL.LSTM_CHAIN], 4, H, op, ch, [True] * L, scale=0.0)
    rng = np.random.default_rng(2)
    w.weights[0].update(_biases(WL.LSTM_CHAIN, H, rng))
    b = w.weights[0]["b"].astype(np.float64)
    sg = lambda z: 1 / (1 + np.exp(-z))
    bi, bf, bg = b[:H], b[H:2 * H], b[2 * H:3 * H]
    hs, cs = evaluate_workload(w)
    for t in range(L):
        ref = sg(bi) * np.tanh(bg) * (1 - sg(bf) ** (t + 1)) / (1 - sg(bf))
        np.testing.assert_allclose(cs[t], ref, rtol=1e-12, atol=1e-14)


def test_p6_zero_weight_full_binary_tree():
    H, height = 3, 4
    op, ch = [], []
    level = []
    for _ in range(2 ** height):
        op.append(0)
        ch.append([])
        level.append(len(op) - 1)
    heights = [0] * len(op)
    while len(level) > 1:
        nxt = []
        for a, bnode in zip(level[0::2], level[1::2]):
            op.append(1)
            ch.append([a, bnode])
            heights.append(heights[a] + 1)
            nxt.append(len(op) - 1)
        level = nxt
    w = WL.make_graph([WL.NARY_LEAF, WL.NARY_INTERNAL], 4, H, op, ch, [k == 0 for k in op], scale=0.0)
    rng = np.random.default_rng(3)
    for t, k in enumerate([WL.NARY_LEAF, WL.NARY_INTERNAL]):
        w.weights[t].update(_biases(k, H, rng))
    bl = w.weights[0]["b"].astype(np.float64)
    b = w.weights[1]["b"].astype(np.float64)
    sg = lambda z: 1 / (1 + np.exp(-z))
    g = lambda a, i: a[i * H:(i + 1) * H]
    c = [sg(g(bl, 0)) * np.tanh(g(bl, 2))]
    for k in range(1, height + 1):
        c.append(sg(g(b, 0)) * np.tanh(g(b, 4)) + (sg(g(b, 1)) + sg(g(b, 2))) * c[-1])
    hs, cs = evaluate_workload(w)
    for v in range(len(op)):
        np.testing.assert_allclose(cs[v], c[heights[v]], rtol=1e-12, atol=1e-14)


def test_p6_zero_weight_grid_lattice_path_sum():
    H, R, Cn = 2, 5, 6
    op, ch = [], []
    ids = {}
    for i in range(R):
        for j in range(Cn):
            ids[i, j] = len(op)
            op.append(0)
            ch.append([ids.get((i, j - 1), -1), ids.get((i - 1, j), -1)])
    w = WL.make_graph([WL.GRID], 3, H, op, ch, [True] * len(op), scale=0.0)
    w.weights[0].update(_biases(WL.GRID, H, np.random.default_rng(4)))
    b = w.weights[0]["b"].astype(np.float64)
    sg = lambda z: 1 / (1 + np.exp(-z))
    g = lambda i: b[i * H:(i + 1) * H]
    a = sg(g(0)) * np.tanh(g(4))
    al, be = sg(g(1)), sg(g(2))
    hs, cs = evaluate_workload(w)
    for (i, j), v in ids.items():
        ref = sum(math.comb(p + q, p) * be ** p * al ** q for p in range(i + 1) for q in range(j + 1)) * a
        np.testing.assert_allclose(cs[v], ref, rtol=1e-12)


def test_p6_zero_weight_lattice_fusion():
    """A char with K >= 1 words ending at it: c = (e^{s(b_i)} tanh(b_u) +
    e^{s(b_l)} sum_k c_w^k) / (e^{s(b_i)} + K e^{s(b_l)})."""
    H = 3
    # chars 0..4; words from char 0 -> ends at char 2, from char 1 -> ends at char 2,
    # from char 2 -> ends at char 4
    op = [0, 1, 0, 1, 0, 1, 0, 0]
    ch = [[-1], [0], [0], [2], [2, 1, 3], [4], [4], [6, 5]]
    w = WL.make_graph([WL.LAT_CHAR, WL.LAT_WORD], 4, H, op, ch, [True] * len(op), scale=0.0)
    rng = np.random.default_rng(5)
    w.weights[0].update(_biases(WL.LAT_CHAR, H, rng))
    w.weights[1].update(_biases(WL.LAT_WORD, H, rng))
    hs, cs = evaluate_workload(w)
    sg = lambda z: 1 / (1 + np.exp(-z))
    b = w.weights[0]["b"].astype(np.float64)
    bl = w.weights[0]["b_l"].astype(np.float64)
    g = lambda i: b[i * H:(i + 1) * H]
    e0, el = np.exp(sg(g(0))), np.exp(sg(bl))
    for v, words in [(4, [1, 3]), (7, [5])]:
        K = len(words)
        ref = (e0 * np.tanh(g(3)) + el * sum(cs[k] for k in words)) / (e0 + K * el)
        np.testing.assert_allclose(cs[v], ref, rtol=1e-12)
    # words have no hidden output; their c follows the word-cell closed form
    bw = w.weights[1]["b"].astype(np.float64)
    gw = lambda i: bw[i * H:(i + 1) * H]
    for wv, cb in [(1, 0), (3, 2), (5, 4)]:
        np.testing.assert_array_equal(hs[wv], 0)
        np.testing.assert_allclose(cs[wv], sg(gw(1)) * cs[cb] + sg(gw(0)) * np.tanh(gw(2)), rtol=1e-12)


def test_bf16_rounding_matches_torch():
    rng = np.random.default_rng(0)
    a = np.concatenate([rng.standard_normal(10000) * 10.0 ** rng.integers(-6, 6, 10000),
                        # exact ties between two bf16 neighbours
                        (np.arange(1, 200, dtype=np.uint32) << 16 | 0x8000).view(np.float32),
                        ((np.arange(1, 200, dtype=np.uint32) << 16) | 0x18000).view(np.float32),
                        np.array([0.0, -0.0, 1e-40, -3.3e38], dtype=np.float32)]).astype(np.float32)
    ref = torch.from_numpy(a).to(torch.bfloat16).to(torch.float32).numpy()
    np.testing.assert_array_equal(round_to_bf16(a).astype(np.float32), ref)
    np.testing.assert_array_equal(WL.round_bf16(a), ref)


def test_bf16_mode_rounds_node_outputs():
    w = WL.make_config(5, instances=2)
    hs, cs = evaluate_workload(w)
    np.testing.assert_array_equal(round_to_bf16(hs), hs)
    np.testing.assert_array_equal(cs.astype(np.float32).astype(np.float64), cs)


def _batched_eval(w, batches):
    """Test-local batched evaluation: per batch, stack the rows of all nodes
    and multiply as matrices (N-ary, chain and grid kinds)."""
    V, H = w.n_nodes, w.hidden
    hs, cs = np.zeros((V, H)), np.zeros((V, H))
    sg = lambda z: 1 / (1 + np.exp(-z))
    for batch in batches:
        t = int(w.op_type[batch[0]])
        k, p = w.kinds[t], w.weights[t]
        kids = np.array([w.children(v) for v in batch]).reshape(len(batch), -1)
        get = lambda arr, col: np.where((kids[:, col] >= 0)[:, None], arr[np.maximum(kids[:, col], 0)], 0.0)
        X = w.x[w.x_row[batch]].astype(np.float64) if w.x_row[batch[0]] >= 0 else None
        W, b = p["W"].astype(np.float64), p["b"].astype(np.float64)
        if k == WL.NARY_LEAF:
            Z = X @ W + b
            i, o, u = np.split(Z, 3, axis=1)
            c = sg(i) * np.tanh(u)
        elif k == WL.NARY_INTERNAL:
            A = np.concatenate([get(hs, 0), get(hs, 1)], axis=1)
            i, f0, f1, o, u = np.split(A @ W + b, 5, axis=1)
            c = sg(i) * np.tanh(u) + sg(f0) * get(cs, 0) + sg(f1) * get(cs, 1)
        elif k == WL.LSTM_CHAIN:
            A = np.concatenate([X, get(hs, 0)], axis=1)
            i, f, g, o = np.split(A @ W + b, 4, axis=1)
            c = sg(f) * get(cs, 0) + sg(i) * np.tanh(g)
        elif k == WL.GRID:
            A = np.concatenate([X, get(hs, 0), get(hs, 1)], axis=1)
            i, fl, ft, o, u = np.split(A @ W + b, 5, axis=1)
            c = sg(i) * np.tanh(u) + sg(fl) * get(cs, 0) + sg(ft) * get(cs, 1)
        hs[batch] = sg(o) * np.tanh(c)
        cs[batch] = c
    return hs, cs


@pytest.mark.parametrize("cfg", [1, 2, 4])
def test_p7_batched_equals_node_at_a_time(cfg):
    from oracle.schedule import schedule
    w = WL.make_config(cfg, instances=3)
    batches, _ = schedule(w.op_type, w.child_ptr, w.child_idx, w.n_types)
    hb, cb = _batched_eval(w, batches)
    hs, cs = evaluate_workload(w)
    np.testing.assert_allclose(hb, hs, rtol=0, atol=1e-12)
    np.testing.assert_allclose(cb, cs, rtol=0, atol=1e-12)
    # any topological order gives bitwise the same node results
    order = [v for b in batches for v in b]
    h2, c2 = evaluate_workload(w, order=order)
    np.testing.assert_array_equal(h2, hs)
    np.testing.assert_array_equal(c2, cs)


def test_topo_order_rejects_cycle():
    with pytest.raises(ValueError):
        topo_order(2, np.array([0, 1, 2]), np.array([1, 0]))


# ---- TreeGRU ---------------------------------------------------------------

def torch_gru_step(h, W_hh, b_hh):
    """Reference: torch.nn.GRUCell (float64, CPU) with a zero input; gates in
    torch's order [r, z, n]: n = tanh(r * (W_hn h + b_hn)), h' = (1 - z) n + z h."""
    H = h.shape[0]
    m = torch.nn.GRUCell(1, H).double()
    with torch.no_grad():
        m.weight_ih.zero_()
        m.bias_ih.zero_()
        m.weight_hh.copy_(torch.from_numpy(np.ascontiguousarray(W_hh, dtype=np.float64)))
        m.bias_hh.copy_(torch.from_numpy(np.asarray(b_hh, dtype=np.float64)))
        out = m(torch.zeros(1, 1, dtype=torch.float64), torch.from_numpy(h).reshape(1, H))
    return out.numpy().reshape(H)


def test_gru_internal_with_equal_children_equals_torch_gru():
    # With h_0 = h_1 = h and the n_1 column block and bias zero, the internal
    # node is one GRU step from h with zero input: the z and r_0 columns act
    # through U[:H] + U[H:], the candidate through U[:H, n_0].
    rng = np.random.default_rng(7)
    H = 5
    U = rng.uniform(-0.6, 0.6, size=(2 * H, 5 * H))
    b = rng.uniform(-0.3, 0.3, size=5 * H)
    U[:, 4 * H:] = 0.0
    b[4 * H:] = 0.0
    h = rng.standard_normal(H)
    got, c = C.gru_internal([h, h], U, b)
    Wsum = U[:H] + U[H:]
    W_hh = np.concatenate([Wsum[:, H:2 * H].T, Wsum[:, 0:H].T, U[:H, 3 * H:4 * H].T])   # [r, z, n]
    b_hh = np.concatenate([b[H:2 * H], b[0:H], b[3 * H:4 * H]])
    np.testing.assert_allclose(got, torch_gru_step(h, W_hh, b_hh), rtol=1e-12, atol=1e-14)
    np.testing.assert_array_equal(got, c)


def test_gru_leaf_equals_torch_gru_from_zero_state():
    # A leaf is one GRU step from h = 0: h' = (1 - z) tanh(W_in x + b_in + r * b_hn)
    # with b_hn = 0.
    rng = np.random.default_rng(8)
    E, H = 6, 4
    W = rng.uniform(-0.5, 0.5, size=(E, 2 * H))
    b = rng.uniform(-0.2, 0.2, size=2 * H)
    x = rng.standard_normal(E)
    got, _ = C.gru_leaf(x, W, b)
    m = torch.nn.GRUCell(E, H).double()
    with torch.no_grad():
        m.weight_hh.zero_()
        m.bias_hh.zero_()
        W_ih = np.concatenate([np.zeros((H, E)), W[:, 0:H].T, W[:, H:].T])   # [r, z, n]
        m.weight_ih.copy_(torch.from_numpy(W_ih))
        m.bias_ih.copy_(torch.from_numpy(np.concatenate([np.zeros(H), b[0:H], b[H:]])))
        ref = m(torch.from_numpy(x).reshape(1, E), torch.zeros(1, H, dtype=torch.float64)).numpy().reshape(H)
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-14)


def test_gru_internal_closed_forms():
    rng = np.random.default_rng(9)
    H = 3
    h0, h1 = rng.standard_normal(H), rng.standard_normal(H)
    # zero weights and biases: z = 1/2, candidate tanh(0) = 0
    h, _ = C.gru_internal([h0, h1], np.zeros((2 * H, 5 * H)), np.zeros(5 * H))
    np.testing.assert_allclose(h, 0.25 * (h0 + h1), rtol=0, atol=1e-15)
    # a saturated update gate keeps the children's mean; a closed one takes the candidate
    U = rng.uniform(-0.5, 0.5, size=(2 * H, 5 * H))
    b = np.zeros(5 * H)
    b[0:H] = 60.0
    h, _ = C.gru_internal([h0, h1], U, b)
    np.testing.assert_allclose(h, (h0 + h1) / 2, rtol=0, atol=1e-12)
    b[0:H] = -60.0
    h, _ = C.gru_internal([h0, h1], U, b)
    n0 = h0 @ U[0:H, 3 * H:4 * H]
    n1 = h1 @ U[H:, 4 * H:]
    r0 = 1 / (1 + np.exp(-(np.concatenate([h0, h1]) @ U[:, H:2 * H])))
    r1 = 1 / (1 + np.exp(-(np.concatenate([h0, h1]) @ U[:, 2 * H:3 * H])))
    np.testing.assert_allclose(h, np.tanh(r0 * n0 + r1 * n1), rtol=0, atol=1e-12)
    # the unused blocks of the n columns do not matter
    U2 = U.copy()
    U2[H:, 3 * H:4 * H] = 9.0
    U2[:H, 4 * H:] = -9.0
    np.testing.assert_array_equal(C.gru_internal([h0, h1], U2, b)[0], C.gru_internal([h0, h1], U, b)[0])


def test_gru_hand_values_one_unit():
    # H = 1 by hand: h_0 = 0.5, h_1 = -0.25, U rows [h_0; h_1], columns [z, r_0, r_1, n_0, n_1]
    U = np.array([[0.2, 1.0, 0.0, 2.0, 7.0],
                  [0.4, 0.0, -1.0, 5.0, -1.0]])
    b = np.array([0.0, 0.0, 0.0, 0.0, 0.0])
    h, _ = C.gru_internal([np.array([0.5]), np.array([-0.25])], U, b)
    z = 0.2 * 0.5 + 0.4 * -0.25            # 0.0   -> sigma = 1/2
    r0 = 0.5                                # sigma(0.5)
    r1 = 0.25                               # -1 * -0.25
    n0 = 2.0 * 0.5                          # 1.0 (n_0 reads h_0 only)
    n1 = -1.0 * -0.25                       # 0.25 (n_1 reads h_1 only)
    s = lambda v: 1 / (1 + np.exp(-v))
    ht = np.tanh(s(r0) * n0 + s(r1) * n1)
    assert z == 0.0
    assert abs(h[0] - (0.5 * 0.125 + 0.5 * ht)) < 1e-15
