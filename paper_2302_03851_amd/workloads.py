"""Seeded synthetic workloads for batched dynamic-dataflow-graph execution.

This module only builds inputs: the graph structure of a mini-batch of
per-instance dataflow graphs (chains, binary trees, lattices, 2-D grids and
child-sum trees), the logical weight matrices of each cell type and the node
inputs x.  It holds none of the method's arithmetic (no cell math, no
schedule, no memory plan), so both the oracle and the GPU path may use it.

Graph format (the union of the instance graphs of one mini-batch, Section 2.1
of the paper: every operation carries a type; a mini-batch is executed as one
graph):

  op_type[V]     int32  type id of every node
  child_ptr[V+1] int64  CSR offsets into child_idx
  child_idx[E]   int32  children of node v are child_idx[child_ptr[v]:child_ptr[v+1]],
                        fixed positions first, then ragged children; -1 marks an
                        absent child (its state is zero)
  x_row[V]       int32  row of x holding the node's input vector, -1 if none

Node ids are instance-major and children-before-parents.

Random draw order (numpy PCG64, seed 1000 + config index by default):
  1. structure, instance by instance (size first, then the shape draws in
     pre-order);
  2. weights, type by type, each logical matrix row-major (biases are zero
     and draw nothing);
  3. x, node by node in node-id order.
bf16 configurations store W and x rounded to bf16 (round-to-nearest-even)
from the fp32 draws; the arrays returned here are float32 holding exactly
those bf16 values.
"""
from __future__ import annotations

import dataclasses
import hashlib
from typing import Dict, List, Optional, Tuple

import numpy as np

# Cell kinds (values mirror EDB_CELL_* in include/edb.h).
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
# MV-RNN: each tree node's d x d matrix is held as d nodes, node j = column j
LINEAR = 10
MV_MAT = 11
MV_VEC = 12
# lattice GRU: one GRU proposal per incoming edge, averaged per position
LGRU_EDGE = 13
POOL_MEAN = 14

KIND_NAMES = {
    LSTM_CHAIN: "lstm_chain", NARY_LEAF: "nary_leaf", NARY_INTERNAL: "nary_internal",
    GRID: "grid", CS_LEAF: "cs_leaf", CS_INTERNAL: "cs_internal",
    LAT_CHAR: "lat_char", LAT_WORD: "lat_word", GRU_LEAF: "gru_leaf", GRU_INTERNAL: "gru_internal",
    LINEAR: "linear", MV_MAT: "mv_mat", MV_VEC: "mv_vec", LGRU_EDGE: "lgru_edge", POOL_MEAN: "pool_mean",
}

# Per kind: (n_fixed children, ragged children allowed, has x input).
KIND_SHAPE = {
    LSTM_CHAIN: (1, False, True),
    NARY_LEAF: (0, False, True),
    NARY_INTERNAL: (2, False, False),
    GRID: (2, False, True),
    CS_LEAF: (0, False, True),
    CS_INTERNAL: (0, True, False),
    LAT_CHAR: (1, True, True),
    LAT_WORD: (1, False, True),
    GRU_LEAF: (0, False, True),
    GRU_INTERNAL: (2, False, False),
    LINEAR: (0, False, True),
    MV_MAT: (2, False, False),
    MV_VEC: (2, True, False),
    LGRU_EDGE: (1, False, True),
    POOL_MEAN: (0, True, False),
}


def weight_shapes(kind: int, E: int, H: int, n_children: int = 2) -> List[Tuple[str, Tuple[int, ...]]]:
    """Logical weight matrices of one cell type, in draw order (row-major).

    Matrices are K x N with rows ordered [x ; child-position-0 h ; ...] and
    columns gate-major in the gate order of the kind:
      LSTM_CHAIN     W[(E+H) x 4H]  gates [i, f, g, o]
      NARY_LEAF      W[E x 3H]      gates [i, o, u]
      NARY_INTERNAL  U[NH x (3+N)H] gates [i, f_0 .. f_{N-1}, o, u]
      GRID           W[(E+2H) x 5H] gates [i, f_left, f_top, o, u]
      CS_LEAF        W[E x 3H]      gates [i, o, u]
      CS_INTERNAL    U_iou[H x 3H] gates [i, o, u];  U_f[H x H]
      LAT_WORD       W_w[(E+H) x 3H] gates [i, f, u]
      LAT_CHAR       W_c[(E+H) x 4H] gates [i, f, o, u];  W_lx[E x H];  W_lc[H x H]
      GRU_LEAF       W[E x 2H]      gates [z, n]
      GRU_INTERNAL   U[2H x 5H]     gates [z, r_0, r_1, n_0, n_1] (n_k reads child k only)
      LINEAR         W[E x H]       h = x W + b
      MV_MAT         W_M[2H x H]    rows: column j of the left matrix, then of the right (W_M transposed)
      MV_VEC         W[2H x H]      rows: [B a ; A b] (the model's W transposed), tanh
      LGRU_EDGE      W[(E+H) x 4H]  gates [z, r, n_x, n_h] (n_x reads x only, n_h the source h only)
      POOL_MEAN      W[H x H]       h = (mean of the ragged children's h) W + b
    Biases follow the matrices (float32).
    """
    if kind == LSTM_CHAIN:
        return [("W", (E + H, 4 * H)), ("b", (4 * H,))]
    if kind in (NARY_LEAF, CS_LEAF):
        return [("W", (E, 3 * H)), ("b", (3 * H,))]
    if kind == NARY_INTERNAL:
        N = n_children
        return [("W", (N * H, (3 + N) * H)), ("b", ((3 + N) * H,))]
    if kind == GRID:
        return [("W", (E + 2 * H, 5 * H)), ("b", (5 * H,))]
    if kind == CS_INTERNAL:
        return [("U_iou", (H, 3 * H)), ("U_f", (H, H)), ("b_iou", (3 * H,)), ("b_f", (H,))]
    if kind == LAT_WORD:
        return [("W", (E + H, 3 * H)), ("b", (3 * H,))]
    if kind == LAT_CHAR:
        return [("W", (E + H, 4 * H)), ("W_lx", (E, H)), ("W_lc", (H, H)),
                ("b", (4 * H,)), ("b_l", (H,))]
    if kind == GRU_LEAF:
        return [("W", (E, 2 * H)), ("b", (2 * H,))]
    if kind == GRU_INTERNAL:
        return [("W", (2 * H, 5 * H)), ("b", (5 * H,))]
    if kind == LINEAR:
        return [("W", (E, H)), ("b", (H,))]
    if kind == MV_MAT:
        return [("W_M", (2 * H, H)), ("b", (H,))]
    if kind == MV_VEC:
        return [("W", (2 * H, H)), ("b", (H,))]
    if kind == LGRU_EDGE:
        return [("W", (E + H, 4 * H)), ("b", (4 * H,))]
    if kind == POOL_MEAN:
        return [("W", (H, H)), ("b", (H,))]
    raise ValueError(f"unknown cell kind {kind}")


@dataclasses.dataclass
class Workload:
    name: str
    dtype: str                      # "f32" or "bf16" (storage of W, x and h)
    kinds: List[int]                # cell kind per type id
    in_dim: int                     # E (0 if no type has an input)
    hidden: int                     # H
    op_type: np.ndarray
    child_ptr: np.ndarray
    child_idx: np.ndarray
    x_row: np.ndarray
    x: np.ndarray                   # float32 [n_x_rows, in_dim]
    weights: List[Dict[str, np.ndarray]]  # per type id, float32 logical matrices
    n_children: List[int]           # N for NARY_INTERNAL types (0 otherwise)
    instances: int
    aux: Optional[Dict[str, np.ndarray]] = None   # model-level view (MV-RNN: trees and weights)

    @property
    def n_nodes(self) -> int:
        return int(self.op_type.shape[0])

    @property
    def n_types(self) -> int:
        return len(self.kinds)

    def shapes(self) -> List[Tuple[int, int]]:
        """(n_fixed, ragged) per type."""
        out = []
        for t, k in enumerate(self.kinds):
            nf, rg, _ = KIND_SHAPE[k]
            if k == NARY_INTERNAL:
                nf = self.n_children[t]
            out.append((nf, int(rg)))
        return out

    def children(self, v: int) -> np.ndarray:
        return self.child_idx[self.child_ptr[v]:self.child_ptr[v + 1]]

    def digest(self) -> str:
        h = hashlib.sha256()
        for a in (self.op_type, self.child_ptr, self.child_idx, self.x_row, self.x):
            h.update(np.ascontiguousarray(a).tobytes())
        for w in self.weights:
            for key in sorted(w):
                h.update(key.encode())
                h.update(np.ascontiguousarray(w[key]).tobytes())
        return h.hexdigest()


def round_bf16(a: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bf16 (ties to even); return float32."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32).astype(np.uint64)
    lsb = (u >> 16) & 1
    r = ((u + 0x7FFF + lsb) >> 16) << 16
    nan = np.isnan(a)
    out = (r & 0xFFFFFFFF).astype(np.uint32).view(np.float32).copy()
    out[nan] = np.float32(np.nan)
    return out


class _GraphBuilder:
    def __init__(self) -> None:
        self.op_type: List[int] = []
        self.children: List[List[int]] = []
        self.has_x: List[bool] = []

    def add(self, t: int, children: List[int], has_x: bool) -> int:
        self.op_type.append(t)
        self.children.append(list(children))
        self.has_x.append(has_x)
        return len(self.op_type) - 1

    def finish(self):
        V = len(self.op_type)
        ptr = np.zeros(V + 1, dtype=np.int64)
        for v, ch in enumerate(self.children):
            ptr[v + 1] = ptr[v] + len(ch)
        idx = np.array([c for ch in self.children for c in ch], dtype=np.int32)
        x_row = np.full(V, -1, dtype=np.int32)
        n = 0
        for v in range(V):
            if self.has_x[v]:
                x_row[v] = n
                n += 1
        return (np.array(self.op_type, dtype=np.int32), ptr, idx, x_row, n)


def _build_binary(rng, n: int, g: _GraphBuilder) -> int:
    # n = 1: leaf; else split k ~ U{1..n-1}, children build(k), build(n-k).
    if n == 1:
        return g.add(0, [], True)
    k = int(rng.integers(1, n))
    left = _build_binary(rng, k, g)
    right = _build_binary(rng, n - k, g)
    return g.add(1, [left, right], False)


def _build_childsum(rng, n: int, g: _GraphBuilder) -> int:
    # n = 1: leaf.  Else a ~ U{1..4}; a = 1 gives a unary node over build(n);
    # otherwise a = min(a, n) parts cut at a-1 distinct uniform points of {1..n-1}.
    if n == 1:
        return g.add(0, [], True)
    a = int(rng.integers(1, 5))
    if a == 1:
        child = _build_childsum(rng, n, g)
        return g.add(1, [child], False)
    a = min(a, n)
    cuts = np.sort(rng.choice(np.arange(1, n), size=a - 1, replace=False))
    bounds = [0] + [int(c) for c in cuts] + [n]
    kids = [_build_childsum(rng, bounds[i + 1] - bounds[i], g) for i in range(a)]
    return g.add(1, kids, False)


def _draw_weights(rng, kinds, E, H, scale, n_children, bf16):
    out = []
    for t, k in enumerate(kinds):
        w = {}
        for name, shape in weight_shapes(k, E, H, n_children[t] or 2):
            if name.startswith("b"):
                w[name] = np.zeros(shape, dtype=np.float32)
            else:
                m = rng.uniform(-scale, scale, size=shape).astype(np.float32)
                w[name] = round_bf16(m) if bf16 else m
        out.append(w)
    return out


CONFIG_NAMES = {
    1: "chain_lstm_f32",
    2: "binary_treelstm_h256_f32",
    3: "lattice_lstm_f32",
    4: "grid_rnn_f32",
    5: "childsum_treelstm_h512_bf16",
    6: "treelstm_2type_h256_f32",
    7: "binary_treegru_h256_f32",
    8: "mvrnn_d64_f32",
    9: "lattice_gru_f32",
}


def relabel(w: Workload, seed: int) -> Tuple[Workload, np.ndarray]:
    """The same mini-batch with its node ids permuted: node v becomes
    perm[v] (children keep their positions, x rows and weights are shared).
    A different input graph whose schedule has the same batch sizes."""
    rng = np.random.default_rng(seed)
    V = w.n_nodes
    perm = rng.permutation(V)
    inv = np.argsort(perm)
    kids = [w.children(int(v)) for v in inv]
    ptr = np.zeros(V + 1, dtype=np.int64)
    ptr[1:] = np.cumsum([len(c) for c in kids])
    idx = (np.concatenate([np.where(c >= 0, perm[np.maximum(c, 0)], -1) for c in kids]).astype(np.int32)
           if V else np.zeros(0, dtype=np.int32))
    w2 = dataclasses.replace(w, op_type=np.ascontiguousarray(w.op_type[inv], dtype=np.int32), child_ptr=ptr,
                             child_idx=idx, x_row=np.ascontiguousarray(w.x_row[inv], dtype=np.int32))
    return w2, perm


def make_config(k: int, seed: Optional[int] = None, instances: Optional[int] = None) -> Workload:
    """Build synthetic config k (1..5; 6 is the two-internal-type TreeLSTM of
    the batching study, 7 the binary TreeGRU, 8 the MV-RNN, 9 the lattice GRU).  `instances` overrides the number of
    instance graphs (chains / trees / lattices / grids) for small test cases
    and scale sweeps; all other sizes and distributions stay as stated."""
    if seed is None:
        seed = 1000 + k
    rng = np.random.Generator(np.random.PCG64(seed))
    g = _GraphBuilder()
    n_children = [0, 0]
    bf16 = False
    if k == 1:
        # 8 chain LSTMs, lengths U{5..20}, E = H = 64, W ~ U(-0.1, 0.1).
        inst = 8 if instances is None else instances
        kinds, E, H, scale = [LSTM_CHAIN], 64, 64, 0.1
        n_children = [0]
        for _ in range(inst):
            L = int(rng.integers(5, 21))
            prev = -1
            for _t in range(L):
                prev = g.add(0, [prev], True)
    elif k == 2:
        # 64 binary trees, leaves U{10..50}, E = H = 256, W ~ U(-0.08, 0.08).
        inst = 64 if instances is None else instances
        kinds, E, H, scale = [NARY_LEAF, NARY_INTERNAL], 256, 256, 0.08
        n_children = [0, 2]
        for _ in range(inst):
            n = int(rng.integers(10, 51))
            _build_binary(rng, n, g)
    elif k == 3:
        # 32 lattices: char chains of length U{20..60}; at each start position a
        # word with probability 0.3 spanning s ~ U{2,3,4} chars (dropped if it
        # runs past the end).  E = 100 (chars and words), H = 200.
        inst = 32 if instances is None else instances
        kinds, E, H, scale = [LAT_CHAR, LAT_WORD], 100, 200, 0.1
        n_children = [0, 0]
        for _ in range(inst):
            L = int(rng.integers(20, 61))
            spans = []
            for b in range(L):
                if rng.random() < 0.3:
                    s = int(rng.integers(2, 5))
                    spans.append(s if b + s - 1 <= L - 1 else 0)
                else:
                    spans.append(0)
            ending: Dict[int, List[int]] = {}
            prev = -1
            for j in range(L):
                c = g.add(0, [prev] + ending.get(j, []), True)
                prev = c
                if spans[j]:
                    w = g.add(1, [c], True)
                    ending.setdefault(j + spans[j] - 1, []).append(w)
    elif k == 4:
        # 32 grids of 16 x 16; each cell reads its left and top neighbours.
        inst = 32 if instances is None else instances
        kinds, E, H, scale = [GRID], 128, 256, 0.08
        n_children = [0]
        R = C = 16
        for _ in range(inst):
            ids = np.full((R, C), -1, dtype=np.int64)
            for i in range(R):
                for j in range(C):
                    left = int(ids[i, j - 1]) if j > 0 else -1
                    top = int(ids[i - 1, j]) if i > 0 else -1
                    ids[i, j] = g.add(0, [left, top], True)
    elif k == 5:
        # 256 child-sum trees, leaves U{20..200}, arity U{1..4}, E = H = 512, bf16.
        inst = 256 if instances is None else instances
        kinds, E, H, scale = [CS_LEAF, CS_INTERNAL], 512, 512, 0.05
        n_children = [0, 0]
        bf16 = True
        for _ in range(inst):
            n = int(rng.integers(20, 201))
            _build_childsum(rng, n, g)
    elif k == 6:
        # TreeLSTM with two internal cell types (a batching study workload):
        # the binary trees of config 2, each internal node of type 1 or 2
        # (U{0,1} per internal node, node order, after the tree's shape),
        # with separate weights per type.
        inst = 64 if instances is None else instances
        kinds, E, H, scale = [NARY_LEAF, NARY_INTERNAL, NARY_INTERNAL], 256, 256, 0.08
        n_children = [0, 2, 2]
        for _ in range(inst):
            n = int(rng.integers(10, 51))
            first = len(g.op_type)
            _build_binary(rng, n, g)
            for v in range(first, len(g.op_type)):
                if g.op_type[v] == 1:
                    g.op_type[v] = 1 + int(rng.integers(0, 2))
    elif k == 7:
        # binary TreeGRU: trees drawn as in config 2 (its own seed), GRU cells
        inst = 64 if instances is None else instances
        kinds, E, H, scale = [GRU_LEAF, GRU_INTERNAL], 256, 256, 0.08
        n_children = [0, 0]
        for _ in range(inst):
            n = int(rng.integers(10, 51))
            _build_binary(rng, n, g)
    elif k == 8:
        return _mvrnn_config(rng, 64 if instances is None else instances)
    elif k == 9:
        return _lattice_gru_config(rng, 32 if instances is None else instances)
    else:
        raise ValueError("config index must be 1..9")

    op_type, ptr, idx, x_row, n_x = g.finish()
    weights = _draw_weights(rng, kinds, E, H, scale, n_children, bf16)
    x = rng.standard_normal(size=(n_x, E), dtype=np.float32)
    if bf16:
        x = round_bf16(x)
    return Workload(
        name=CONFIG_NAMES[k], dtype="bf16" if bf16 else "f32", kinds=kinds,
        in_dim=E, hidden=H, op_type=op_type, child_ptr=ptr, child_idx=idx,
        x_row=x_row, x=x, weights=weights, n_children=n_children, instances=inst)


def _mvrnn_config(rng, inst: int, d: int = 64) -> Workload:
    """MV-RNN over binary trees drawn as in config 2 (leaves U{10..50}), d = 64,
    fp32.  Every tree node becomes d matrix-column nodes (type 1, MV_MAT; leaf:
    type 0, LINEAR) followed by one vector node (type 2, MV_VEC; leaf: type 0).
    Draws: (1) the tree shapes; (2) W_M = [I I] / 2 + U(-0.05, 0.05) (d x 2d)
    and W ~ U(-0.1, 0.1) (d x 2d), row-major; biases 0, the leaf LINEAR
    weights are the identity; (3) per leaf in node order its vector ~ N(0, 1),
    then its matrix I + U(-0.1, 0.1) (row-major).  Word vectors and matrices
    follow the initialisation the model's authors describe (matrices near the
    identity)."""
    tb = _GraphBuilder()
    for _ in range(inst):
        _build_binary(rng, int(rng.integers(10, 51)), tb)
    n_tree = len(tb.op_type)
    left = np.array([c[0] if c else -1 for c in tb.children], dtype=np.int64)
    right = np.array([c[1] if c else -1 for c in tb.children], dtype=np.int64)
    WM = np.concatenate([np.eye(d), np.eye(d)], axis=1) / 2 + rng.uniform(-0.05, 0.05, size=(d, 2 * d))
    WM = WM.astype(np.float32)
    W = rng.uniform(-0.1, 0.1, size=(d, 2 * d)).astype(np.float32)
    leaf_vec = np.zeros((n_tree, d), dtype=np.float32)
    leaf_mat = np.zeros((n_tree, d, d), dtype=np.float32)
    for t in range(n_tree):
        if left[t] < 0:
            leaf_vec[t] = rng.standard_normal(size=d, dtype=np.float32)
            leaf_mat[t] = np.eye(d, dtype=np.float32) + rng.uniform(-0.1, 0.1, size=(d, d)).astype(np.float32)
    g = _GraphBuilder()
    vec_node = np.zeros(n_tree, dtype=np.int64)
    mat_node = np.zeros(n_tree, dtype=np.int64)   # first of the d column nodes
    xs = []
    for t in range(n_tree):
        l, r = int(left[t]), int(right[t])
        if l < 0:
            mat_node[t] = g.add(0, [], True)
            xs.append(leaf_mat[t][:, 0])
            for j in range(1, d):
                g.add(0, [], True)
                xs.append(leaf_mat[t][:, j])
            vec_node[t] = g.add(0, [], True)
            xs.append(leaf_vec[t])
        else:
            ml, mr = int(mat_node[l]), int(mat_node[r])
            mat_node[t] = g.add(1, [ml, mr], False)
            for j in range(1, d):
                g.add(1, [ml + j, mr + j], False)
            cols = [ml + j for j in range(d)] + [mr + j for j in range(d)]
            vec_node[t] = g.add(2, [int(vec_node[l]), int(vec_node[r])] + cols, False)
    op_type, ptr, idx, x_row, n_x = g.finish()
    weights = [{"W": np.eye(d, dtype=np.float32), "b": np.zeros(d, dtype=np.float32)},
               {"W_M": np.ascontiguousarray(WM.T), "b": np.zeros(d, dtype=np.float32)},
               {"W": np.ascontiguousarray(W.T), "b": np.zeros(d, dtype=np.float32)}]
    aux = {"tree_left": left, "tree_right": right, "vec_node": vec_node, "mat_node": mat_node,
           "leaf_vec": leaf_vec, "leaf_mat": leaf_mat, "W": W, "bW": np.zeros(d, dtype=np.float32), "WM": WM}
    return Workload(name=CONFIG_NAMES[8], dtype="f32", kinds=[LINEAR, MV_MAT, MV_VEC], in_dim=d, hidden=d,
                    op_type=op_type, child_ptr=ptr, child_idx=idx, x_row=x_row,
                    x=np.stack(xs).astype(np.float32), weights=weights, n_children=[0, 0, 0], instances=inst,
                    aux=aux)


def _lattice_gru_config(rng, inst: int, E: int = 100, H: int = 200) -> Workload:
    """Lattice GRU over lattices drawn as in config 3 (lengths U{20..60}; at
    each start position a word with probability 0.3 spanning U{2,3,4}
    characters, dropped past the end), E = 100, H = 200, fp32.  Per position
    j: its character-edge node (type 0, LGRU_EDGE; x = the character's input,
    source = position j-1), one word-edge node (type 0; x = the word's input,
    source = the position before the word's first character) per word ending
    at j, then the position node (type 1, POOL_MEAN over those edges).
    Draws: (1) the structure; (2) the GRU weights Wx [E x 3H] then Wh [H x 3H]
    ~ U(-0.1, 0.1) (gate columns z, r, n), biases 0, the pooling map the
    identity; (3) the edges' inputs ~ N(0, 1) in node order."""
    g = _GraphBuilder()
    lattices = []
    for _ in range(inst):
        L = int(rng.integers(20, 61))
        spans = []
        for b in range(L):
            if rng.random() < 0.3:
                sp = int(rng.integers(2, 5))
                spans.append(sp if b + sp - 1 <= L - 1 else 0)
            else:
                spans.append(0)
        words = [(b, b + sp - 1) for b, sp in enumerate(spans) if sp]
        ending: Dict[int, List[int]] = {}
        for k, (b, e) in enumerate(words):
            ending.setdefault(e, []).append(k)
        pos = []
        char_edge = []
        word_edge = [0] * len(words)
        for j in range(L):
            ce = g.add(0, [pos[j - 1] if j else -1], True)
            char_edge.append(ce)
            edges = [ce]
            for k in ending.get(j, []):
                b = words[k][0]
                word_edge[k] = g.add(0, [pos[b - 1] if b else -1], True)
                edges.append(word_edge[k])
            pos.append(g.add(1, edges, False))
        lattices.append({"length": L, "words": words, "pos": np.array(pos), "char_edge": np.array(char_edge),
                         "word_edge": np.array(word_edge, dtype=np.int64)})
    op_type, ptr, idx, x_row, n_x = g.finish()
    Wx = rng.uniform(-0.1, 0.1, size=(E, 3 * H)).astype(np.float32)
    Wh = rng.uniform(-0.1, 0.1, size=(H, 3 * H)).astype(np.float32)
    x = rng.standard_normal(size=(n_x, E), dtype=np.float32)
    W = np.zeros((E + H, 4 * H), dtype=np.float32)
    W[:E, :3 * H] = Wx                       # z, r, n_x over x
    W[E:, :2 * H] = Wh[:, :2 * H]            # z, r over the source state
    W[E:, 3 * H:] = Wh[:, 2 * H:]            # n_h over the source state
    weights = [{"W": W, "b": np.zeros(4 * H, dtype=np.float32)},
               {"W": np.eye(H, dtype=np.float32), "b": np.zeros(H, dtype=np.float32)}]
    aux = {"lattices": lattices, "Wx": Wx, "Wh": Wh, "bx": np.zeros(3 * H, dtype=np.float32),
           "bhn": np.zeros(H, dtype=np.float32)}
    return Workload(name=CONFIG_NAMES[9], dtype="f32", kinds=[LGRU_EDGE, POOL_MEAN], in_dim=E, hidden=H,
                    op_type=op_type, child_ptr=ptr, child_idx=idx, x_row=x_row, x=x, weights=weights,
                    n_children=[0, 0], instances=inst, aux=aux)


def make_graph(kinds: List[int], E: int, H: int, op_type, children: List[List[int]],
               has_x: List[bool], seed: int = 0, scale: float = 0.1, dtype: str = "f32",
               n_children: Optional[List[int]] = None, bias_scale: float = 0.0) -> Workload:
    """Workload from an explicit small graph (tests).  Weights ~ U(-scale, scale),
    biases ~ U(-bias_scale, bias_scale), x ~ N(0, 1)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    g = _GraphBuilder()
    for t, ch, hx in zip(op_type, children, has_x):
        g.add(int(t), list(ch), bool(hx))
    op, ptr, idx, x_row, n_x = g.finish()
    if n_children is None:
        n_children = [2 if k == NARY_INTERNAL else 0 for k in kinds]
    bf16 = dtype == "bf16"
    weights = []
    for t, k in enumerate(kinds):
        w = {}
        for name, shape in weight_shapes(k, E, H, n_children[t] or 2):
            if name.startswith("b"):
                m = rng.uniform(-bias_scale, bias_scale, size=shape).astype(np.float32) \
                    if bias_scale else np.zeros(shape, dtype=np.float32)
                w[name] = m
            else:
                m = rng.uniform(-scale, scale, size=shape).astype(np.float32)
                w[name] = round_bf16(m) if bf16 else m
        weights.append(w)
    x = rng.standard_normal(size=(n_x, E), dtype=np.float32)
    if bf16:
        x = round_bf16(x)
    return Workload(name="custom", dtype=dtype, kinds=list(kinds), in_dim=E, hidden=H,
                    op_type=op, child_ptr=ptr, child_idx=idx, x_row=x_row, x=x,
                    weights=weights, n_children=list(n_children), instances=1)


def make_typed_trees(shape: str, n_trees: int, leaves=(10, 50), seed: int = 0):
    """Typed dataflow graphs for batch-count studies (schedules only; no cells).

    shape "outputs": the tree of Figure 1 at scale.  Binary trees (the C2 shape
      draw, leaves U{lo..hi}) whose leaves (type 0) and internal nodes (type 1)
      each feed an output operation (type 2), and one reduction (type 3) per
      tree over all of its outputs.
    shape "two_type": binary trees whose internal nodes take one of two types
      (1 or 2, probability 1/2 each), as in a TreeLSTM with two internal cell
      types; leaves are type 0.
    Returns (op_type, child_ptr, child_idx, n_types); node ids are
    children-before-parents, instance by instance."""
    rng = np.random.Generator(np.random.PCG64(seed))
    g = _GraphBuilder()
    for _ in range(n_trees):
        n = int(rng.integers(leaves[0], leaves[1] + 1))
        first = len(g.op_type)
        _build_binary(rng, n, g)
        tree = range(first, len(g.op_type))
        if shape == "outputs":
            outs = [g.add(2, [v], False) for v in tree]
            g.add(3, outs, False)
        elif shape == "two_type":
            for v in tree:
                if g.op_type[v] == 1:
                    g.op_type[v] = 1 + int(rng.integers(0, 2))
        else:
            raise ValueError(f"unknown shape {shape}")
    op, ptr, idx, _x_row, _n = g.finish()
    return op, ptr, idx, 4 if shape == "outputs" else 3
