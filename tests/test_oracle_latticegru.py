"""Pins of the lattice GRU oracle (oracle/latticegru.py):

* a lattice without words is torch.nn.GRU over its characters (the GRU form
  with the reset gate after the recurrent product, bias b_hn on that product);
* a word from the lattice start with the first character's input proposes
  exactly the first position's state;
* a position's state is the mean of its edges' proposals, each one a
  torch.nn.GRUCell step from its own source (checked per position on a
  lattice with overlapping words).
"""
import numpy as np
import torch

from oracle.latticegru import lattice_gru


def _weights(rng, E, H, scale=0.4):
    return (rng.uniform(-scale, scale, (E, 3 * H)), rng.uniform(-scale, scale, (H, 3 * H)),
            rng.uniform(-0.2, 0.2, 3 * H), rng.uniform(-0.2, 0.2, H))


def _cell(E, H, Wx, Wh, bx, bhn):
    c = torch.nn.GRUCell(E, H).double()
    with torch.no_grad():
        # torch gate order [r, z, n]; the oracle's columns are [z, r, n]
        perm = lambda m: np.concatenate([m[H:2 * H], m[:H], m[2 * H:]])
        c.weight_ih.copy_(torch.from_numpy(perm(Wx.T)))
        c.weight_hh.copy_(torch.from_numpy(perm(Wh.T)))
        c.bias_ih.copy_(torch.from_numpy(perm(bx)))
        c.bias_hh.copy_(torch.from_numpy(np.concatenate([np.zeros(2 * H), bhn])))
    return c


def test_no_words_is_torch_gru():
    rng = np.random.Generator(np.random.PCG64(3))
    E, H, L = 5, 4, 9
    Wx, Wh, bx, bhn = _weights(rng, E, H)
    xc = rng.normal(size=(L, E))
    h, gc, _ = lattice_gru(L, [], xc, np.zeros((0, E)), Wx, Wh, bx, bhn)
    g = torch.nn.GRU(E, H).double()
    c = _cell(E, H, Wx, Wh, bx, bhn)
    with torch.no_grad():
        g.weight_ih_l0.copy_(c.weight_ih)
        g.weight_hh_l0.copy_(c.weight_hh)
        g.bias_ih_l0.copy_(c.bias_ih)
        g.bias_hh_l0.copy_(c.bias_hh)
        out, _ = g(torch.from_numpy(xc)[:, None])
    np.testing.assert_allclose(h, out[:, 0].numpy(), rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(gc, h, rtol=0, atol=0)


def test_word_from_the_start_repeats_the_first_step():
    """A word (0, 1) with input x_char[0] starts, like position 0's character
    edge, from the zero state: its proposal is h_0, and position 1 is the mean
    of its character proposal and h_0."""
    rng = np.random.Generator(np.random.PCG64(4))
    E, H = 3, 5
    Wx, Wh, bx, bhn = _weights(rng, E, H)
    xc = rng.normal(size=(3, E))
    # word (0, 1): source = zero state, input = x_char[0]; position 0's char edge
    # also starts from zero with x_char[0]: position 1 then averages g(x_c[1], h_0)
    # with g(x_c[0], 0) = h_0
    h_w, _, gw = lattice_gru(3, [(0, 1)], xc, xc[:1], Wx, Wh, bx, bhn)
    h_0, gc0, _ = lattice_gru(3, [], xc, np.zeros((0, E)), Wx, Wh, bx, bhn)
    np.testing.assert_allclose(gw[0], h_0[0], rtol=0, atol=0)
    np.testing.assert_allclose(h_w[1], (gc0[1] + h_0[0]) / 2, rtol=1e-15, atol=1e-15)


def test_mean_of_gru_cells():
    rng = np.random.Generator(np.random.PCG64(5))
    E, H, L = 4, 6, 8
    Wx, Wh, bx, bhn = _weights(rng, E, H)
    words = [(0, 2), (1, 3), (2, 3), (3, 6), (5, 7), (0, 7)]
    xc = rng.normal(size=(L, E))
    xw = rng.normal(size=(len(words), E))
    h, gc, gw = lattice_gru(L, words, xc, xw, Wx, Wh, bx, bhn)
    c = _cell(E, H, Wx, Wh, bx, bhn)
    t = lambda a: torch.from_numpy(np.asarray(a, dtype=np.float64))[None]
    zero = np.zeros(H)
    with torch.no_grad():
        for j in range(L):
            props = [c(t(xc[j]), t(h[j - 1] if j else zero))[0].numpy()]
            for k, (s, e) in enumerate(words):
                if e == j:
                    props.append(c(t(xw[k]), t(h[s - 1] if s else zero))[0].numpy())
            np.testing.assert_allclose(h[j], np.mean(props, axis=0), rtol=1e-12, atol=1e-13)


# ---- the node-level cells of the lattice GRU in the graph oracle -----------

def test_lgru_edge_is_torch_gru_cell():
    """oracle.cells.lgru_edge: W [(E+H) x 4H] with gate columns [z, r, n_x,
    n_h] (n_x over the x rows, n_h over the h rows, b_nh on the recurrent
    candidate product) is one torch.nn.GRUCell step."""
    from oracle import cells as C
    rng = np.random.Generator(np.random.PCG64(11))
    E, H = 5, 4
    W = rng.uniform(-0.5, 0.5, (E + H, 4 * H))
    b = rng.uniform(-0.3, 0.3, 4 * H)
    x, h = rng.normal(size=E), rng.normal(size=H)
    got, c = C.lgru_edge(x, h, W, b)
    cell = torch.nn.GRUCell(E, H).double()
    blk = lambda m, g: m[:, g * H:(g + 1) * H]
    with torch.no_grad():
        # torch rows [r, z, n]
        cell.weight_ih.copy_(torch.from_numpy(np.concatenate([blk(W[:E], 1), blk(W[:E], 0), blk(W[:E], 2)], 1).T))
        cell.weight_hh.copy_(torch.from_numpy(np.concatenate([blk(W[E:], 1), blk(W[E:], 0), blk(W[E:], 3)], 1).T))
        cell.bias_ih.copy_(torch.from_numpy(np.concatenate([b[H:2 * H], b[:H], b[2 * H:3 * H]])))
        cell.bias_hh.copy_(torch.from_numpy(np.concatenate([np.zeros(2 * H), b[3 * H:]])))
        ref = cell(torch.from_numpy(x)[None], torch.from_numpy(h)[None]).numpy()[0]
    np.testing.assert_allclose(got, ref, rtol=0, atol=1e-13)
    np.testing.assert_array_equal(got, c)


def test_pool_mean_hand_values():
    """mean([1, 2], [3, 4]) = [2, 3]; W = [[1, 2], [0, 1]] maps it to [2, 7];
    b = [1, -1] gives [3, 6].  With no edge the state is b."""
    from oracle import cells as C
    W = np.array([[1.0, 2.0], [0.0, 1.0]])
    b = np.array([1.0, -1.0])
    h, c = C.pool_mean([np.array([1.0, 2.0]), np.array([3.0, 4.0])], W, b)
    np.testing.assert_array_equal(h, [3.0, 6.0])
    np.testing.assert_array_equal(c, h)
    np.testing.assert_array_equal(C.pool_mean([], W, b)[0], b)


def test_graph_oracle_equals_lattice_oracle():
    """The graph oracle (oracle.evaluate over the lattice GRU's LGRU_EDGE and
    POOL_MEAN nodes, identity pooling, zero biases) gives the lattice-level
    oracle's position states and edge proposals."""
    from oracle.evaluate import evaluate_workload
    from paper_2302_03851_amd import workloads as WL
    w = WL.make_config(9, instances=4)
    h, c = evaluate_workload(w)
    a = w.aux
    for lat in a["lattices"]:
        xw = w.x[w.x_row[lat["word_edge"]]] if len(lat["words"]) else np.zeros((0, w.in_dim))
        hp, gc, gw = lattice_gru(lat["length"], lat["words"], w.x[w.x_row[lat["char_edge"]]], xw,
                                 a["Wx"], a["Wh"], a["bx"], a["bhn"])
        np.testing.assert_allclose(h[lat["pos"]], hp, rtol=0, atol=1e-12)
        np.testing.assert_allclose(h[lat["char_edge"]], gc, rtol=0, atol=1e-12)
        if len(lat["words"]):
            np.testing.assert_allclose(h[lat["word_edge"]], gw, rtol=0, atol=1e-12)
    np.testing.assert_array_equal(c, h)
