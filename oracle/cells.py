"""Cell equations of the recurrent / recursive models evaluated in the paper.

The paper names its workloads (Section 5.1, Table 2: BiLSTM tagger, N-ary
TreeLSTM, TreeGRU, lattice LSTM; the gated grid RNN of the introduction's
structured data examples) but prints no cell equations; each function below writes out
the published definition of the cited model.  All arithmetic is float64.

Conventions: weight matrices are K x N with rows ordered
[x ; child-position-0 h ; child-position-1 h ; ...] and columns gate-major;
z = a . W + b for the row vector a; sigma is the logistic function; an absent
child contributes a zero state (h, c) = (0, 0).
"""
from __future__ import annotations

import numpy as np

# Cell kind ids (the library's interface numbering).
LSTM_CHAIN = 0
NARY_LEAF = 1
NARY_INTERNAL = 2
GRID = 3
CS_LEAF = 4
CS_INTERNAL = 5
LAT_CHAR = 6
LAT_WORD = 7
GRU_LEAF = 8
GRU_INTERNAL = 9
LGRU_EDGE = 13
POOL_MEAN = 14


def sigmoid(z):
    return 1.0 / (1.0 + np.exp(-z))


def _f64(a):
    return np.asarray(a, dtype=np.float64)


def _split(z, n):
    return np.split(z, n)


def lstm_chain(x, h_prev, c_prev, W, b):
    """One LSTM time step (the tagger's recurrent cell, Table 2).

    z = [x ; h_prev] W + b split into gates [i, f, g, o];
    c = sigma(f) * c_prev + sigma(i) * tanh(g);  h = sigma(o) * tanh(c).
    """
    z = np.concatenate([_f64(x), _f64(h_prev)]) @ _f64(W) + _f64(b)
    i, f, g, o = _split(z, 4)
    c = sigmoid(f) * _f64(c_prev) + sigmoid(i) * np.tanh(g)
    h = sigmoid(o) * np.tanh(c)
    return h, c


def tree_leaf(x, W, b):
    """Leaf of an N-ary or child-sum TreeLSTM (Table 2's TreeLSTM, cited model
    Tai et al.): with no children the forget terms vanish.

    z = x W + b split into [i, o, u];  c = sigma(i) * tanh(u);  h = sigma(o) * tanh(c).
    """
    z = _f64(x) @ _f64(W) + _f64(b)
    i, o, u = _split(z, 3)
    c = sigmoid(i) * np.tanh(u)
    h = sigmoid(o) * np.tanh(c)
    return h, c


def nary_internal(hs, cs, U, b):
    """Internal node of an N-ary TreeLSTM (Table 2, cited model Tai et al.).

    z = [h_0 ; ... ; h_{N-1}] U + b split into [i, f_0 .. f_{N-1}, o, u], where
    the f_k columns of U hold the per-child forget blocks over all children;
    c = sigma(i) * tanh(u) + sum_k sigma(f_k) * c_k;  h = sigma(o) * tanh(c).
    """
    N = len(hs)
    z = np.concatenate([_f64(h) for h in hs]) @ _f64(U) + _f64(b)
    parts = _split(z, 3 + N)
    i, fs, o, u = parts[0], parts[1:1 + N], parts[1 + N], parts[2 + N]
    c = sigmoid(i) * np.tanh(u)
    for f, ck in zip(fs, cs):
        c = c + sigmoid(f) * _f64(ck)
    h = sigmoid(o) * np.tanh(c)
    return h, c


def grid(x, h_left, c_left, h_top, c_top, W, b):
    """Gated 2-D grid cell (multi-dimensional LSTM without peepholes): the
    cell reads its left and top neighbours.

    z = [x ; h_left ; h_top] W + b split into [i, f_left, f_top, o, u];
    c = sigma(i) tanh(u) + sigma(f_left) c_left + sigma(f_top) c_top;  h = sigma(o) tanh(c).
    """
    z = np.concatenate([_f64(x), _f64(h_left), _f64(h_top)]) @ _f64(W) + _f64(b)
    i, fl, ft, o, u = _split(z, 5)
    c = sigmoid(i) * np.tanh(u) + sigmoid(fl) * _f64(c_left) + sigmoid(ft) * _f64(c_top)
    h = sigmoid(o) * np.tanh(c)
    return h, c


def childsum_internal(hs, cs, U_iou, U_f, b_iou, b_f):
    """Internal node of a child-sum TreeLSTM (cited TreeLSTM model, Tai et al.).

    h_sum = sum_k h_k;  z = h_sum U_iou + b_iou split into [i, o, u];
    f_k = sigma(h_k U_f + b_f) per child;
    c = sigma(i) tanh(u) + sum_k f_k * c_k;  h = sigma(o) tanh(c).
    """
    h_sum = np.zeros(_f64(U_f).shape[0])
    for h in hs:
        h_sum = h_sum + _f64(h)
    z = h_sum @ _f64(U_iou) + _f64(b_iou)
    i, o, u = _split(z, 3)
    c = sigmoid(i) * np.tanh(u)
    for h, ck in zip(hs, cs):
        f = sigmoid(_f64(h) @ _f64(U_f) + _f64(b_f))
        c = c + f * _f64(ck)
    h_out = sigmoid(o) * np.tanh(c)
    return h_out, c


def lattice_word(x_w, h_b, c_b, W, b):
    """Word cell of the lattice LSTM (Table 2, cited model Zhang and Yang): a
    word spanning chars b..e reads the state of its first char b.

    z = [x_w ; h_b] W + b split into [i, f, u];
    c_w = sigma(f) c_b + sigma(i) tanh(u).  The word cell has no hidden output.
    """
    z = np.concatenate([_f64(x_w), _f64(h_b)]) @ _f64(W) + _f64(b)
    i, f, u = _split(z, 3)
    c_w = sigmoid(f) * _f64(c_b) + sigmoid(i) * np.tanh(u)
    return np.zeros_like(c_w), c_w


def lattice_char(x, h_prev, c_prev, word_cs, W, W_lx, W_lc, b, b_l):
    """Character cell of the lattice LSTM (cited model Zhang and Yang).

    z = [x ; h_prev] W + b split into [i, f, o, u].
    No word ends at this char: c = sigma(f) c_prev + sigma(i) tanh(u).
    Words k = 1..K end here with cell states c_w^k: link gates
    l_k = sigma(x W_lx + c_w^k W_lc + b_l); the input gate and the link gates
    are normalised together, element-wise,
    a_0 = exp(sigma(i)) / (exp(sigma(i)) + sum_k exp(l_k)),  a_k = exp(l_k) / (same),
    and c = a_0 tanh(u) + sum_k a_k c_w^k (the forget gate is not used).
    Then h = sigma(o) tanh(c).
    """
    z = np.concatenate([_f64(x), _f64(h_prev)]) @ _f64(W) + _f64(b)
    i, f, o, u = _split(z, 4)
    if len(word_cs) == 0:
        c = sigmoid(f) * _f64(c_prev) + sigmoid(i) * np.tanh(u)
    else:
        xl = _f64(x) @ _f64(W_lx)
        e0 = np.exp(sigmoid(i))
        es = [np.exp(sigmoid(xl + _f64(cw) @ _f64(W_lc) + _f64(b_l))) for cw in word_cs]
        den = e0 + sum(es)
        c = (e0 / den) * np.tanh(u)
        for ek, cw in zip(es, word_cs):
            c = c + (ek / den) * _f64(cw)
    h = sigmoid(o) * np.tanh(c)
    return h, c


def gru_leaf(x, W, b):
    """Leaf of a binary TreeGRU (Table 2's TreeGRU): the gated recurrent unit
    (Cho et al. 2014) with no children.

    z = x W + b split into [z, n];  h = (1 - sigma(z)) * tanh(n).  A GRU node's
    state is h alone; it is returned as the cell state too."""
    zz = _f64(x) @ _f64(W) + _f64(b)
    z, n = _split(zz, 2)
    h = (1.0 - sigmoid(z)) * np.tanh(n)
    return h, h


def gru_internal(hs, U, b):
    """Internal node of a binary TreeGRU: the gated recurrent unit extended to
    two ordered children the way the N-ary TreeLSTM extends the LSTM, with
    each child's reset gate applied after its recurrent product (the GRU form
    whose candidate is tanh(W x + b + r * (U h + b_h))).

    Columns of U [2H x 5H] and b [5H]: [z, r_0, r_1, n_0, n_1].  z, r_0 and r_1
    read both children; n_0 reads only h_0 (rows 0..H-1), n_1 only h_1 (rows
    H..2H-1); the other blocks of the n columns are not used.
      h~ = tanh(sigma(r_0) * n_0 + sigma(r_1) * n_1)
      h  = sigma(z) * (h_0 + h_1) / 2 + (1 - sigma(z)) * h~
    """
    h0, h1 = _f64(hs[0]), _f64(hs[1])
    U, b = _f64(U), _f64(b)
    H = h0.shape[0]
    a = np.concatenate([h0, h1])
    z = a @ U[:, 0:H] + b[0:H]
    r0 = a @ U[:, H:2 * H] + b[H:2 * H]
    r1 = a @ U[:, 2 * H:3 * H] + b[2 * H:3 * H]
    n0 = h0 @ U[0:H, 3 * H:4 * H] + b[3 * H:4 * H]
    n1 = h1 @ U[H:2 * H, 4 * H:5 * H] + b[4 * H:5 * H]
    ht = np.tanh(sigmoid(r0) * n0 + sigmoid(r1) * n1)
    h = sigmoid(z) * (h0 + h1) / 2.0 + (1.0 - sigmoid(z)) * ht
    return h, h


def lgru_edge(x, h_src, W, b):
    """One edge of the lattice GRU (Table 2's lattice-based GRU): a GRU step
    (Cho et al. 2014, reset gate applied after the recurrent product) from the
    edge's source position state with the edge's own input.

    W [(E+H) x 4H] with rows [x ; h_src] and gate columns [z, r, n_x, n_h];
    n_x reads only the x rows, n_h only the h_src rows:
      z = [x ; h] W_z + b_z,  r = [x ; h] W_r + b_r,
      n = tanh(x W_nx + b_nx + sigma(r) * (h W_nh + b_nh)),
      h' = (1 - sigma(z)) * n + sigma(z) * h.
    The edge's state is h' (returned as the cell state too)."""
    x, h = _f64(x), _f64(h_src)
    W, b = _f64(W), _f64(b)
    E, H = x.shape[0], h.shape[0]
    a = np.concatenate([x, h])
    z = a @ W[:, 0:H] + b[0:H]
    r = a @ W[:, H:2 * H] + b[H:2 * H]
    nx = x @ W[:E, 2 * H:3 * H] + b[2 * H:3 * H]
    nh = h @ W[E:, 3 * H:4 * H] + b[3 * H:4 * H]
    n = np.tanh(nx + sigmoid(r) * nh)
    out = (1.0 - sigmoid(z)) * n + sigmoid(z) * h
    return out, out


def pool_mean(hs, W, b):
    """A lattice position's state: the mean of its incoming edges' states,
    mapped by W [H x H] and shifted by b: h = mean_k(h_k) W + b (with no
    edge, the mean is taken as 0 and h = b).  The lattice GRU uses W = I,
    b = 0.  Returned as the cell state too."""
    W, b = _f64(W), _f64(b)
    m = np.mean([_f64(h) for h in hs], axis=0) if len(hs) else np.zeros(W.shape[0])
    out = m @ W + b
    return out, out
