"""Matrix-vector recursive neural network (MV-RNN, one of the tree models of
Table 2; the model of Socher, Huval, Manning and Ng, 2012) on binary trees,
in float64.

Test infrastructure only: imported by tests/, __graft_entry__.smoke() and
bench.py's cpu_baseline, never by the library.

Every tree node n carries a vector v_n (length d) and a matrix M_n (d x d).
A leaf's pair is its input (the word's vector and the word's matrix).  An
internal node with left child (a, A) and right child (b, B) computes

    v = tanh(W [B a ; A b] + b_W)        W  : d x 2d,  b_W : d
    M = W_M [A ; B]                        W_M: d x 2d

so each child's matrix transforms the other child's vector, and the parent's
matrix is a linear map of the two children's matrices stacked.  The paper
names the model and its dataset only; the definition is the published one.
"""
from __future__ import annotations

import numpy as np


def mvrnn(left, right, leaf_vec, leaf_mat, W, bW, WM):
    """Evaluate every node of a forest of binary trees.

    left, right: [n] child ids, -1 for both children of a leaf; a node's
    children precede it (ids in children-before-parents order).
    leaf_vec: [n, d] (read for leaves only); leaf_mat: [n, d, d] (leaves only).
    Returns (V [n, d], M [n, d, d]) in float64."""
    left = np.asarray(left)
    right = np.asarray(right)
    n = left.shape[0]
    d = np.asarray(W).shape[0]
    W = np.asarray(W, dtype=np.float64)
    bW = np.asarray(bW, dtype=np.float64)
    WM = np.asarray(WM, dtype=np.float64)
    V = np.zeros((n, d))
    M = np.zeros((n, d, d))
    for v in range(n):
        l, r = int(left[v]), int(right[v])
        if l < 0:
            V[v] = np.asarray(leaf_vec[v], dtype=np.float64)
            M[v] = np.asarray(leaf_mat[v], dtype=np.float64)
            continue
        assert 0 <= l < v and 0 <= r < v, "children must precede their parent"
        a, A, b, B = V[l], M[l], V[r], M[r]
        V[v] = np.tanh(W @ np.concatenate([B @ a, A @ b]) + bW)
        M[v] = WM @ np.concatenate([A, B], axis=0)
    return V, M
