"""Pins of the MV-RNN oracle (oracle/mvrnn.py) against what the model's
definition fixes independently of the oracle's code:

* identity matrices everywhere reduce the vector recursion to the plain
  recursive network v = tanh(W_1 a + W_2 b + b_W): a two-leaf tree is one
  torch.nn.RNNCell step (input b, hidden a), a left-branching tree is
  torch.nn.RNN over the leaves with the first leaf as initial state;
* W_M = [alpha I, beta I] makes the matrix recursion linear with a closed
  form: the root matrix is the sum over leaves of alpha^(left turns) *
  beta^(right turns) * (leaf matrix) along the root-to-leaf path;
* a swap of the two children's matrices must swap which vector each one
  transforms (a sign/operand check on a hand-sized tree, computed from the
  definition with explicit loops).
"""
import numpy as np
import pytest
import torch

from oracle.mvrnn import mvrnn


def _rng(seed):
    return np.random.Generator(np.random.PCG64(seed))


def _left_chain(n_leaves):
    """((((l0 l1) l2) l3) ...): leaves 0..n-1, internal nodes after them."""
    left, right = [-1] * n_leaves, [-1] * n_leaves
    prev = 0
    for i in range(1, n_leaves):
        left.append(prev)
        right.append(i)
        prev = len(left) - 1
    return np.array(left), np.array(right)


def _random_tree(rng, n_leaves):
    """Random binary tree: leaves first, internal nodes in creation order."""
    left, right = [-1] * n_leaves, [-1] * n_leaves
    pool = list(range(n_leaves))
    while len(pool) > 1:
        i = int(rng.integers(0, len(pool) - 1))
        l, r = pool[i], pool[i + 1]
        left.append(l)
        right.append(r)
        pool[i:i + 2] = [len(left) - 1]
    return np.array(left), np.array(right)


def test_two_leaves_is_rnn_cell():
    rng = _rng(1)
    d = 6
    W = rng.uniform(-0.5, 0.5, (d, 2 * d))
    bW = rng.uniform(-0.2, 0.2, d)
    a, b = rng.normal(size=d), rng.normal(size=d)
    eye = np.eye(d)
    V, M = mvrnn([-1, -1, 0], [-1, -1, 1], np.stack([a, b, a * 0]), np.stack([eye, eye, eye]), W, bW,
                 rng.normal(size=(d, 2 * d)))
    cell = torch.nn.RNNCell(d, d, nonlinearity="tanh").double()
    with torch.no_grad():
        cell.weight_hh.copy_(torch.from_numpy(W[:, :d]))
        cell.weight_ih.copy_(torch.from_numpy(W[:, d:]))
        cell.bias_hh.copy_(torch.from_numpy(bW))
        cell.bias_ih.zero_()
        ref = cell(torch.from_numpy(b)[None], torch.from_numpy(a)[None])[0].numpy()
    np.testing.assert_allclose(V[2], ref, rtol=1e-13, atol=1e-13)


@pytest.mark.parametrize("n_leaves", [2, 5, 9])
def test_left_chain_is_rnn(n_leaves):
    rng = _rng(10 + n_leaves)
    d = 5
    W = rng.uniform(-0.6, 0.6, (d, 2 * d))
    bW = rng.uniform(-0.2, 0.2, d)
    left, right = _left_chain(n_leaves)
    n = left.shape[0]
    vec = np.zeros((n, d))
    vec[:n_leaves] = rng.normal(size=(n_leaves, d))
    mats = np.broadcast_to(np.eye(d), (n, d, d))
    WM = np.concatenate([np.eye(d), np.eye(d)], axis=1) * 0.5   # keeps every matrix the identity
    V, M = mvrnn(left, right, vec, mats, W, bW, WM)
    rnn = torch.nn.RNN(d, d, nonlinearity="tanh").double()
    with torch.no_grad():
        rnn.weight_hh_l0.copy_(torch.from_numpy(W[:, :d]))
        rnn.weight_ih_l0.copy_(torch.from_numpy(W[:, d:]))
        rnn.bias_hh_l0.copy_(torch.from_numpy(bW))
        rnn.bias_ih_l0.zero_()
        out, _ = rnn(torch.from_numpy(vec[1:n_leaves])[:, None], torch.from_numpy(vec[0])[None, None])
    np.testing.assert_allclose(V[n_leaves:], out[:, 0].numpy(), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(M[-1], np.eye(d), atol=1e-15)


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_matrix_closed_form(seed):
    rng = _rng(100 + seed)
    d = 4
    n_leaves = int(rng.integers(2, 12))
    left, right = _random_tree(rng, n_leaves)
    n = left.shape[0]
    alpha, beta = 0.7, -1.3
    WM = np.concatenate([alpha * np.eye(d), beta * np.eye(d)], axis=1)
    mats = np.zeros((n, d, d))
    mats[:n_leaves] = rng.normal(size=(n_leaves, d, d))
    _, M = mvrnn(left, right, np.zeros((n, d)), mats, rng.normal(size=(d, 2 * d)), np.zeros(d), WM)
    # path weights from the root down
    wgt = {n - 1: 1.0}
    for v in range(n - 1, -1, -1):
        if left[v] >= 0:
            wgt[int(left[v])] = wgt[v] * alpha
            wgt[int(right[v])] = wgt[v] * beta
    expect = sum(wgt[i] * mats[i] for i in range(n_leaves))
    np.testing.assert_allclose(M[-1], expect, rtol=1e-12, atol=1e-12)


def test_hand_tree_loops():
    """Three leaves ((x y) z), evaluated from the definition with explicit
    loops; leaf matrices differ so that a swapped operand shows."""
    rng = _rng(7)
    d = 3
    W = rng.uniform(-1, 1, (d, 2 * d))
    bW = rng.uniform(-0.3, 0.3, d)
    WM = rng.uniform(-1, 1, (d, 2 * d))
    vec = rng.normal(size=(5, d))
    mats = rng.normal(size=(5, d, d))
    left, right = np.array([-1, -1, -1, 0, 3]), np.array([-1, -1, -1, 1, 2])

    def node(a, A, b, B):
        u = [sum(B[i][k] * a[k] for k in range(d)) for i in range(d)] + \
            [sum(A[i][k] * b[k] for k in range(d)) for i in range(d)]
        v = [np.tanh(sum(W[i][k] * u[k] for k in range(2 * d)) + bW[i]) for i in range(d)]
        S = [list(A[k]) for k in range(d)] + [list(B[k]) for k in range(d)]
        Mp = [[sum(WM[i][k] * S[k][j] for k in range(2 * d)) for j in range(d)] for i in range(d)]
        return np.array(v), np.array(Mp)

    v3, m3 = node(vec[0], mats[0], vec[1], mats[1])
    v4, m4 = node(v3, m3, vec[2], mats[2])
    V, M = mvrnn(left, right, vec, mats, W, bW, WM)
    np.testing.assert_allclose(V[3], v3, rtol=1e-13, atol=1e-14)
    np.testing.assert_allclose(M[3], m3, rtol=1e-13, atol=1e-14)
    np.testing.assert_allclose(V[4], v4, rtol=1e-13, atol=1e-14)
    np.testing.assert_allclose(M[4], m4, rtol=1e-13, atol=1e-14)
