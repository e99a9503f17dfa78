"""Cell equations of the recurrent / recursive models evaluated in the paper.

The paper names its workloads (Section 5.1, Table 2: BiLSTM tagger, N-ary
TreeLSTM, lattice LSTM; the gated grid RNN of the introduction's structured
data examples) but prints no cell equations; each function below writes out
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
