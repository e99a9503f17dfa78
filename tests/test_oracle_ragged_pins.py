"""Pins of the oracle's ragged cells and of its error measure, CPU only.

The child-sum TreeLSTM (Table 2's TreeLSTM, cited model Tai et al.) with two
or more children, the lattice LSTM character cell (Table 2, cited model Zhang
and Yang) with words whose link gates carry non-zero input and cell weights,
and the normwise error that every parity bound is stated in.  Each case is
chosen so that a plausible slip fails it: a forget gate computed from the
child sum instead of each child's own h, a link gate without its x term or
reading the previous char's cell instead of the word's, a transposed weight,
a 2-norm or a mean in the error measure.
"""
import math

import numpy as np
import pytest
import torch

from oracle import cells as C
from oracle.compare import elementwise_rel_err, normwise_rel_err, state_rel_err
from oracle.evaluate import evaluate_workload
from paper_2302_03851_amd import workloads as WL

LN2, LN3 = math.log(2.0), math.log(3.0)
# sigma(ln 3) = 3/4, sigma(0) = 1/2, sigma(-ln 3) = 1/4, tanh(ln 2) = 3/5


# ---- child-sum TreeLSTM, two or more children -------------------------------

def test_childsum_three_children_hand_values():
    """H = 1.  Children h = (ln 3, 0, 0), c = (1, 2, 4); U_iou = [1 1 1],
    b_iou = (0, 0, ln 2 - ln 3), U_f = [1], b_f = 0.
    The child sum ln 3 gives i = o = sigma(ln 3) = 3/4 and u = ln 2 (tanh 3/5);
    the per-child forget gates are sigma(h_k) = 3/4, 1/2, 1/2, so
    c = 9/20 + 3/4 + 1 + 2 = 21/5 and h = 3/4 tanh(21/5).
    (Forget gates from the child sum would give 3/4 each and c = 57/10.)"""
    hs = [np.array([LN3]), np.array([0.0]), np.array([0.0])]
    cs = [np.array([1.0]), np.array([2.0]), np.array([4.0])]
    h, c = C.childsum_internal(hs, cs, np.array([[1.0, 1.0, 1.0]]), np.array([[1.0]]),
                               np.array([0.0, 0.0, LN2 - LN3]), np.array([0.0]))
    assert c[0] == pytest.approx(21 / 5, abs=1e-12)
    assert h[0] == pytest.approx(0.75 * math.tanh(21 / 5), abs=1e-12)


def test_childsum_two_children_hand_values():
    """H = 1.  Children h = (ln 3, -ln 3) sum to 0, so U_iou does not act;
    b_iou = (ln 3, 0, ln 2): i = 3/4, o = 1/2, tanh(u) = 3/5.  Forget gates
    3/4 and 1/4 on c = (2, -4): c = 9/20 + 3/2 - 1 = 19/20, h = tanh(19/20)/2.
    (From the child sum both gates would be 1/2 and c = -11/20.)"""
    hs = [np.array([LN3]), np.array([-LN3])]
    cs = [np.array([2.0]), np.array([-4.0])]
    h, c = C.childsum_internal(hs, cs, np.array([[5.0, -7.0, 2.0]]), np.array([[1.0]]),
                               np.array([LN3, 0.0, LN2]), np.array([0.0]))
    assert c[0] == pytest.approx(19 / 20, abs=1e-12)
    assert h[0] == pytest.approx(0.5 * math.tanh(19 / 20), abs=1e-12)


def test_childsum_four_children_two_units_hand_values():
    """H = 2, U_f = [[1, 1], [0, 2]] (not symmetric, so a transposed U_f
    fails): h_k U_f = (h_0, h_0 + 2 h_1).
      child   h             h U_f           f            c
      1    (ln 3, 0)       (ln 3, ln 3)    (3/4, 3/4)   (1, 2)
      2    (0, ln3/2)      (0, ln 3)       (1/2, 3/4)   (2, 1)
      3    (-ln 3, 0)      (-ln 3, -ln 3)  (1/4, 1/4)   (4, -4)
      4    (0, -ln3/2)     (0, -ln 3)      (1/2, 1/4)   (8, 8)
    sum_k f_k c_k = (27/4, 13/4).  The child sum is 0; b_iou gives
    i = (3/4, 3/4), o = (1/2, 3/4), tanh(u) = (3/5, -3/5):
    c = (9/20 + 27/4, -9/20 + 13/4) = (36/5, 14/5)."""
    hs = [np.array([LN3, 0.0]), np.array([0.0, LN3 / 2]), np.array([-LN3, 0.0]),
          np.array([0.0, -LN3 / 2])]
    cs = [np.array([1.0, 2.0]), np.array([2.0, 1.0]), np.array([4.0, -4.0]), np.array([8.0, 8.0])]
    U_iou = np.arange(12, dtype=np.float64).reshape(2, 6) - 5.0     # acts on the zero child sum
    U_f = np.array([[1.0, 1.0], [0.0, 2.0]])
    b_iou = np.array([LN3, LN3, 0.0, LN3, LN2, -LN2])
    h, c = C.childsum_internal(hs, cs, U_iou, U_f, b_iou, np.zeros(2))
    np.testing.assert_allclose(c, [36 / 5, 14 / 5], rtol=0, atol=1e-12)
    np.testing.assert_allclose(h, [0.5 * math.tanh(36 / 5), 0.75 * math.tanh(14 / 5)], rtol=0, atol=1e-12)


def test_childsum_graph_zero_weight_closed_form():
    """Through the graph evaluator: internal weights zero, biases non-zero,
    leaves with distinct states.  Every gate is then a constant and
    c_v = sigma(b_i) tanh(b_u) + sigma(b_f) sum_k c_k over the node's present
    children (2, 3 and 4 of them, leaves and internal nodes mixed; an absent
    child -1 is dropped)."""
    H = 3
    op = [0, 0, 0, 0, 0, 0, 1, 1, 1, 1]
    ch = [[], [], [], [], [], [], [0, 1], [2, 3, -1, 4], [6, 5, 7], [8, 0, 1, 2]]
    w = WL.make_graph([WL.CS_LEAF, WL.CS_INTERNAL], 4, H, op, ch, [k == 0 for k in op],
                      seed=21, scale=0.7, bias_scale=0.6)
    w.weights[1]["U_iou"][:] = 0
    w.weights[1]["U_f"][:] = 0
    b = w.weights[1]["b_iou"].astype(np.float64)
    bf = w.weights[1]["b_f"].astype(np.float64)
    sg = lambda z: 1 / (1 + np.exp(-z))
    a = sg(b[:H]) * np.tanh(b[2 * H:])
    hs, cs = evaluate_workload(w)
    assert np.ptp(cs[:6], axis=0).min() > 1e-3          # leaves really differ
    for v in range(6, 10):
        kids = [k for k in ch[v] if k >= 0]
        np.testing.assert_allclose(cs[v], a + sg(bf) * cs[kids].sum(axis=0), rtol=1e-12, atol=1e-15)
        np.testing.assert_allclose(hs[v], sg(b[H:2 * H]) * np.tanh(cs[v]), rtol=1e-12, atol=1e-15)


# ---- lattice LSTM character cell with words ---------------------------------

def test_lattice_char_link_gates_hand_values():
    """H = E = 1, x = 1, previous char c = 7 (never a word's cell), char
    weights 0, b = (0, 5, ln 3, ln 2): sigma(i) = 1/2, o = 3/4, tanh(u) = 3/5
    (f is not used when words arrive).  W_lx = ln 3, W_lc = 1, b_l = 0 and two
    words with cells 0 and -ln 3: l_1 = sigma(ln 3) = 3/4, l_2 = sigma(0) = 1/2.
    With D = e^{1/2} + e^{3/4} + e^{1/2}:
    c = (e^{1/2} 3/5 + e^{3/4} 0 + e^{1/2} (-ln 3)) / D."""
    h, c = C.lattice_char(np.array([1.0]), np.array([0.5]), np.array([7.0]),
                          [np.array([0.0]), np.array([-LN3])],
                          np.zeros((2, 4)), np.array([[LN3]]), np.array([[1.0]]),
                          np.array([0.0, 5.0, LN3, LN2]), np.array([0.0]))
    D = 2 * math.exp(0.5) + math.exp(0.75)
    ref = math.exp(0.5) * (0.6 - LN3) / D
    assert c[0] == pytest.approx(ref, abs=1e-12)
    assert h[0] == pytest.approx(0.75 * math.tanh(ref), abs=1e-12)


def test_lattice_char_one_word_is_a_two_way_logistic():
    """H = E = 1, one word: the normalisation over {sigma(i), l} is a logistic
    of the difference, a_1 = sigma(l - sigma(i)), a_0 = 1 - a_1.  x = 2,
    W_lx = ln 3 / 2, W_lc = 1/2, b_l = -1, c_w = 2: l = sigma(ln 3) = 3/4;
    b_i = 0: sigma(i) = 1/2; tanh(u) = 3/5."""
    h, c = C.lattice_char(np.array([2.0]), np.array([0.0]), np.array([-3.0]), [np.array([2.0])],
                          np.zeros((2, 4)), np.array([[LN3 / 2]]), np.array([[0.5]]),
                          np.array([0.0, 0.0, 0.0, LN2]), np.array([-1.0]))
    a1 = 1 / (1 + math.exp(-(0.75 - 0.5)))
    assert c[0] == pytest.approx((1 - a1) * 0.6 + a1 * 2.0, abs=1e-12)
    assert h[0] == pytest.approx(0.5 * math.tanh(c[0]), abs=1e-12)


def _linear(W, b, a):
    """torch.nn.Linear (float64, CPU) with weight W^T and bias b applied to a."""
    m = torch.nn.Linear(W.shape[0], W.shape[1]).double()
    with torch.no_grad():
        m.weight.copy_(torch.from_numpy(np.ascontiguousarray(W.T, dtype=np.float64)))
        m.bias.copy_(torch.from_numpy(np.asarray(b, dtype=np.float64)))
        return m(torch.from_numpy(np.asarray(a, dtype=np.float64)))


def test_lattice_char_fusion_against_torch_linear_and_softmax():
    """A lattice of 4 chars and 3 words with every weight non-zero (H = 6,
    E = 5): char 2 receives two words, char 3 one.  Each char with words
    equals torch: the gates and the link gates as torch.nn.Linear layers
    followed by torch.sigmoid (the link layer over [x ; c_w] with weight
    [W_lx ; W_lc]), the normalisation as torch.softmax over
    {sigma(i), l_1, .., l_K} per element, c the softmax-weighted sum of
    {tanh(u), c_w^1, .., c_w^K}, h = sigma(o) tanh(c)."""
    E, H = 5, 6
    # ids: c0, w0 (reads c0, ends at c2), c1, w1 (reads c1, ends at c2), c2, w2 (reads c2, ends at c3), c3
    op = [0, 1, 0, 1, 0, 1, 0]
    ch = [[-1], [0], [0], [2], [2, 1, 3], [4], [4, 5]]
    w = WL.make_graph([WL.LAT_CHAR, WL.LAT_WORD], E, H, op, ch, [True] * len(op), seed=17,
                      scale=0.6, bias_scale=0.5)
    p = {k: v.astype(np.float64) for k, v in w.weights[0].items()}
    assert min(np.abs(p["W_lx"]).min(), np.abs(p["W_lc"]).min()) > 0
    hs, cs = evaluate_workload(w)
    g = lambda a, k: a[..., k * H:(k + 1) * H]
    W_link = np.concatenate([p["W_lx"], p["W_lc"]], axis=0)
    for v, prev, words in [(4, 2, [1, 3]), (6, 4, [5])]:
        x = w.x[w.x_row[v]].astype(np.float64)
        a = np.concatenate([x, hs[prev]])
        si = torch.sigmoid(_linear(g(p["W"], 0), g(p["b"], 0), a))
        so = torch.sigmoid(_linear(g(p["W"], 2), g(p["b"], 2), a))
        tu = torch.tanh(_linear(g(p["W"], 3), g(p["b"], 3), a))
        ls = [torch.sigmoid(_linear(W_link, p["b_l"], np.concatenate([x, cs[k]]))) for k in words]
        wts = torch.softmax(torch.stack([si] + ls), dim=0)
        vals = torch.stack([tu] + [torch.from_numpy(cs[k]) for k in words])
        c_ref = (wts * vals).sum(dim=0)
        h_ref = so * torch.tanh(c_ref)
        np.testing.assert_allclose(cs[v], c_ref.numpy(), rtol=0, atol=1e-12)
        np.testing.assert_allclose(hs[v], h_ref.numpy(), rtol=0, atol=1e-12)
        # the previous char's cell differs from every word's: a link gate reading it would differ
        assert all(np.abs(cs[prev] - cs[k]).max() > 1e-2 for k in words)


# ---- the error measure -------------------------------------------------------

def test_normwise_rel_err_hand_values():
    """Rows: |g - r|_inf / max(|r|_inf, 1e-6).
      (1, 2) vs (1, 1):    1 / 1            = 1
      (3, 4) vs (3, 5):    1 / 5            = 0.2  (2-norms would give 1/sqrt(34))
      (0, 1e-7) vs (0, 0): 1e-7 / 1e-6 floor = 0.1
    The measure is the maximum over rows (the mean would be 13/30)."""
    got = np.array([[1.0, 2.0], [3.0, 4.0], [0.0, 1e-7]])
    ref = np.array([[1.0, 1.0], [3.0, 5.0], [0.0, 0.0]])
    assert normwise_rel_err(got, ref) == pytest.approx(1.0, rel=1e-15)
    assert normwise_rel_err(got, ref, rows=[1, 2]) == pytest.approx(0.2, rel=1e-15)
    assert normwise_rel_err(got, ref, rows=[2]) == pytest.approx(0.1, rel=1e-9)
    assert normwise_rel_err(got[1:2], ref[1:2]) == pytest.approx(0.2, rel=1e-15)
    assert normwise_rel_err(got[:0], ref[:0]) == 0.0
    # the floor is a parameter
    assert normwise_rel_err(got[2:], ref[2:], floor=1e-3) == pytest.approx(1e-4, rel=1e-9)


def test_elementwise_rel_err_hand_values():
    """|g - r| / max(|r|, 1e-3), maximum over elements:
    1.5 vs 1 -> 0.5;  0.0011 vs 0.001 -> 0.1;  1e-4 vs 0 -> 0.1."""
    got = np.array([[1.5, 0.0011, 1e-4]])
    ref = np.array([[1.0, 0.001, 0.0]])
    assert elementwise_rel_err(got, ref) == pytest.approx(0.5, rel=1e-15)
    assert elementwise_rel_err(got[:, 1:], ref[:, 1:]) == pytest.approx(0.1, rel=1e-9)


def test_state_rel_err_takes_the_worse_state():
    """The larger of the h and c measures; h rows can be restricted (lattice
    words have no h)."""
    h = np.array([[1.0, 0.0], [9.0, 9.0]])
    hr = np.array([[1.0, 0.5], [1.0, 1.0]])       # row 0: 0.5 / 1; row 1: 8 / 1
    c = np.array([[2.0, 2.0]])
    cr = np.array([[2.0, 2.5]])                   # 0.5 / 2.5 = 0.2
    assert state_rel_err(h, c, hr, cr) == pytest.approx(8.0)
    assert state_rel_err(h, c, hr, cr, h_rows=[0]) == pytest.approx(0.5)
    assert state_rel_err(h[:1], c, h[:1], cr) == pytest.approx(0.2)
