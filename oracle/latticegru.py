"""Lattice GRU (the LatticeGRU of Table 2), in float64.

Test infrastructure only: imported by tests/, __graft_entry__.smoke() and
bench.py's cpu_baseline, never by the library.

The paper names the model (a lattice-based GRU encoder for translation) and
gives no equations.  Reading: a lattice over L positions (characters) has,
into every position j, one character edge from position j-1 and one word edge
per lexicon word that ends at j, from the position before the word's first
character.  Every incoming edge e proposes a GRU step from its source
position's state with its own input, and the position's state is the mean of
its edges' proposals:

    g_e = GRU(x_e, h_src(e))          (h_src = 0 before the first position)
    h_j = (1 / |E_j|) sum_{e in E_j} g_e

GRU is the gated recurrent unit with the reset gate applied after the
recurrent product (the form of PyTorch's GRUCell):
    z = sigma(W_z x + b_z + U_z h),  r = sigma(W_r x + b_r + U_r h),
    n = tanh(W_n x + b_n + r * (U_n h + b_hn)),  g = (1 - z) n + z h.
"""
from __future__ import annotations

import numpy as np


def _sig(v):
    return 1.0 / (1.0 + np.exp(-v))


def gru(x, h, Wx, Wh, bx, bhn):
    """One GRU step.  Wx: [E x 3H] input weights (gate columns z, r, n), Wh:
    [H x 3H] recurrent weights, bx: [3H] input bias, bhn: [H] bias of the
    recurrent candidate product."""
    H = h.shape[0]
    a = x @ Wx + bx
    b = h @ Wh
    z = _sig(a[:H] + b[:H])
    r = _sig(a[H:2 * H] + b[H:2 * H])
    n = np.tanh(a[2 * H:] + r * (b[2 * H:] + bhn))
    return (1.0 - z) * n + z * h


def lattice_gru(length, words, x_char, x_word, Wx, Wh, bx, bhn):
    """One lattice: `length` positions, words = [(start, end)] (inclusive
    character span); x_char: [length, E], x_word: [n_words, E].  Returns
    (h [length, H], g_char [length, H], g_word [n_words, H]): position states
    and every edge's proposal."""
    Wx = np.asarray(Wx, dtype=np.float64)
    Wh = np.asarray(Wh, dtype=np.float64)
    bx = np.asarray(bx, dtype=np.float64)
    bhn = np.asarray(bhn, dtype=np.float64)
    H = Wh.shape[0]
    h = np.zeros((length, H))
    g_char = np.zeros((length, H))
    g_word = np.zeros((len(words), H))
    ends = {}
    for k, (s, e) in enumerate(words):
        assert 0 <= s < e < length, "a word spans at least two positions inside the lattice"
        ends.setdefault(e, []).append(k)
    zero = np.zeros(H)
    for j in range(length):
        g_char[j] = gru(np.asarray(x_char[j], dtype=np.float64), h[j - 1] if j else zero, Wx, Wh, bx, bhn)
        props = [g_char[j]]
        for k in ends.get(j, []):
            s = words[k][0]
            g_word[k] = gru(np.asarray(x_word[k], dtype=np.float64), h[s - 1] if s else zero, Wx, Wh, bx, bhn)
            props.append(g_word[k])
        h[j] = np.mean(props, axis=0)
    return h, g_char, g_word
