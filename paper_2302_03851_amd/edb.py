"""Python front end of libedb: handles for the graph, schedule, plan and
executor, plus a `Forward` helper that owns the device buffers of one
mini-batch.  PyTorch provides device memory and the stream only; all work is
done by libedb's host code and HIP kernels."""
from __future__ import annotations

import ctypes as C
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

from . import _lib as L
from .workloads import KIND_SHAPE, NARY_INTERNAL, weight_shapes


def _i32(a):
    return np.ascontiguousarray(a, dtype=np.int32)


def _ptr(a, ctype):
    return a.ctypes.data_as(C.POINTER(ctype))


class Graph:
    def __init__(self, op_type, child_ptr, child_idx, x_row, n_types):
        lib = L.load()
        self._op = _i32(op_type)
        self._ptr = np.ascontiguousarray(child_ptr, dtype=np.int64)
        self._idx = _i32(child_idx) if len(child_idx) else np.zeros(1, dtype=np.int32)
        self._xr = _i32(x_row)
        self.n_nodes = int(self._op.shape[0])
        self.n_types = int(n_types)
        h = C.c_void_p()
        L.check(lib.edb_build_graph(self.n_nodes, self.n_types, _ptr(self._op, C.c_int32),
                                    _ptr(self._ptr, C.c_int64), _ptr(self._idx, C.c_int32),
                                    _ptr(self._xr, C.c_int32), C.byref(h)), "edb_build_graph")
        self.handle = h

    def __del__(self):
        if getattr(self, "handle", None) and L is not None and L._lib is not None:
            L._lib.edb_graph_free(self.handle)
            self.handle = None


class Schedule:
    def __init__(self, graph: Graph, kind=L.POLICY_TABLE, encoding=L.ENC_SORT, table=None):
        lib = L.load()
        self.graph = graph
        flat = None
        if table:
            if isinstance(table, dict):
                flat = [len(table)]
                for key, action in table.items():
                    flat += [len(key)] + list(key) + [action]
            else:
                flat = list(table)
        self._tab = _i32(flat) if flat else None
        pol = L.Policy(kind, encoding, _ptr(self._tab, C.c_int32) if flat else None,
                       len(flat) if flat else 0)
        h = C.c_void_p()
        L.check(lib.edb_schedule(graph.handle, C.byref(pol), C.byref(h)), "edb_schedule")
        self.handle = h
        self._view = None

    def _load_view(self):
        if self._view is None:
            lib = L.load()
            nb = C.c_int32()
            bp, bn, bt = C.POINTER(C.c_int32)(), C.POINTER(C.c_int32)(), C.POINTER(C.c_int32)()
            L.check(lib.edb_schedule_view(self.handle, C.byref(nb), C.byref(bp), C.byref(bn), C.byref(bt)))
            B, V = nb.value, self.graph.n_nodes
            self._view = (np.ctypeslib.as_array(bp, shape=(B + 1,)).copy(),
                          np.ctypeslib.as_array(bn, shape=(V,)).copy() if V else np.zeros(0, dtype=np.int32),
                          np.ctypeslib.as_array(bt, shape=(B,)).copy() if B else np.zeros(0, dtype=np.int32))
        return self._view

    @property
    def batch_ptr(self):
        return self._load_view()[0]

    @property
    def batch_nodes(self):
        return self._load_view()[1]

    @property
    def batch_type(self):
        return self._load_view()[2]

    @property
    def n_batches(self):
        return int(self.batch_type.shape[0])

    def batches(self) -> List[List[int]]:
        return [self.batch_nodes[self.batch_ptr[b]:self.batch_ptr[b + 1]].tolist()
                for b in range(self.n_batches)]

    def __del__(self):
        if getattr(self, "handle", None) and L is not None and L._lib is not None:
            L._lib.edb_schedule_free(self.handle)
            self.handle = None


def lower_bound(graph: Graph) -> int:
    """edb_lower_bound: the Appendix A.3 bound on the number of batches."""
    out = C.c_int64()
    L.check(L.load().edb_lower_bound(graph.handle, C.byref(out)), "edb_lower_bound")
    return int(out.value)


def learn_policy(graph: Graph, encoding=L.ENC_SORT, **params):
    """edb_learn_policy: learns an FSM policy table by N-step Q-learning.
    Keyword arguments override the library defaults (trials, check_every,
    n_step, alpha, epsilon, lr, gamma, seed).  Returns (flat table, stats dict,
    Q) with Q = {key tuple: float64[n_types]}."""
    lib = L.load()
    p = L.LearnParams()
    lib.edb_learn_defaults(C.byref(p))
    p.encoding = encoding
    for k, v in params.items():
        if not hasattr(p, k):
            raise TypeError(f"unknown learning parameter {k}")
        setattr(p, k, v)
    h = C.c_void_p()
    L.check(lib.edb_learn_policy(graph.handle, C.byref(p), C.byref(h)), "edb_learn_policy")
    try:
        tab, tlen, st = C.POINTER(C.c_int32)(), C.c_int64(), L.LearnStats()
        L.check(lib.edb_learned_view(h, C.byref(tab), C.byref(tlen), C.byref(st)))
        table = np.ctypeslib.as_array(tab, shape=(tlen.value,)).tolist() if tlen.value else []
        stats = {"trials": st.trials, "batches": st.batches, "lower_bound": st.lower_bound,
                 "states": st.n_states}
        ns, keys, klen, q = C.c_int32(), C.POINTER(C.c_int32)(), C.c_int64(), C.POINTER(C.c_double)()
        L.check(lib.edb_learned_q(h, C.byref(ns), C.byref(keys), C.byref(klen), C.byref(q)))
        Q = {}
        if ns.value:
            flat = np.ctypeslib.as_array(keys, shape=(klen.value,)).tolist()
            vals = np.ctypeslib.as_array(q, shape=(ns.value * graph.n_types,)).copy()
            pos = 0
            for i in range(ns.value):
                kl = flat[pos]
                Q[tuple(flat[pos + 1:pos + 1 + kl])] = vals[i * graph.n_types:(i + 1) * graph.n_types]
                pos += 1 + kl
    finally:
        lib.edb_learned_free(h)
    return table, stats, Q


class Plan:
    def __init__(self, graph: Graph, sched: Schedule, shapes: Sequence[Tuple[int, int, int]], mode=L.PLAN_RC):
        lib = L.load()
        self.graph, self.sched = graph, sched
        arr = (L.OperandShape * len(shapes))(*[L.OperandShape(*s) for s in shapes])
        h = C.c_void_p()
        L.check(lib.edb_plan_memory(graph.handle, sched.handle, arr, mode, C.byref(h)), "edb_plan_memory")
        self.handle = h
        self._loaded = False

    def __getattr__(self, name):
        # plan arrays are copied out of the library on first use only
        if name in ("n_slots", "slot", "order", "x_slot", "seg_ptr", "segs", "idx_pool", "ragged_off",
                    "ragged_pool", "pads") and not self.__dict__.get("_loaded", True):
            self._load_view()
            return self.__dict__[name]
        raise AttributeError(name)

    def _load_view(self):
        v = L.PlanView()
        L.check(L.load().edb_plan_view(self.handle, C.byref(v)))
        V, B = v.n_nodes, v.n_batches
        asarr = lambda p, n, dt=np.int32: np.ctypeslib.as_array(p, shape=(n,)).copy() if n else np.zeros(0, dt)
        d = self.__dict__
        d["n_slots"] = v.n_slots
        d["slot"] = asarr(v.slot, V)
        d["order"] = asarr(v.order, V)
        d["x_slot"] = asarr(v.x_slot, V)
        d["seg_ptr"] = asarr(v.seg_ptr, B + 1)
        nseg = int(d["seg_ptr"][-1]) if B else 0
        d["segs"] = [(v.segs[i].kind, v.segs[i].base, v.segs[i].idx_off, v.segs[i].len) for i in range(nseg)]
        d["idx_pool"] = asarr(v.idx_pool, v.idx_len)
        d["ragged_off"] = asarr(v.ragged_off, B, np.int64)
        d["ragged_pool"] = asarr(v.ragged_pool, v.ragged_len)
        d["pads"] = asarr(v.pads, v.n_pads)
        d["_loaded"] = True

    def batch_segments(self, b):
        """[(kind, slot list)] for batch b: result first, then the operand lists."""
        out = []
        for kind, base, off, n in self.segs[self.seg_ptr[b]:self.seg_ptr[b + 1]]:
            out.append((kind, [] if kind == L.SEG_NONE else self.idx_pool[off:off + n].tolist()))
        return out

    def __del__(self):
        if getattr(self, "handle", None) and L is not None and L._lib is not None:
            L._lib.edb_plan_free(self.handle)
            self.handle = None


def cell_struct(kind, in_dim, hidden, n_children, dtype) -> L.Cell:
    return L.Cell(kind, in_dim, hidden, n_children, dtype)


def packed_bytes(cell: L.Cell) -> int:
    n = C.c_int64()
    L.check(L.load().edb_packed_weight_bytes(C.byref(cell), C.byref(n)), "edb_packed_weight_bytes")
    return int(n.value)


def pack_weights(cell: L.Cell, logical: Sequence[np.ndarray], dest_ptr: int, stream: int = 0):
    mats = [np.ascontiguousarray(m, dtype=np.float32) for m in logical]
    arr = (C.POINTER(C.c_float) * len(mats))(*[_ptr(m, C.c_float) for m in mats])
    L.check(L.load().edb_pack_weights(C.byref(cell), arr, C.c_void_p(dest_ptr), C.c_void_p(stream)),
            "edb_pack_weights")


class Exec:
    def __init__(self, graph: Graph, sched: Schedule, plan: Plan, cells: Sequence[L.Cell], flags=L.USE_GRAPH):
        lib = L.load()
        self.graph, self.sched, self.plan = graph, sched, plan
        self._cells = (L.Cell * len(cells))(*cells)
        h = C.c_void_p()
        L.check(lib.edb_prepare(graph.handle, sched.handle, plan.handle, self._cells, flags, C.byref(h)),
                "edb_prepare")
        self.handle = h
        self.flags = flags

    def launches(self) -> int:
        n = C.c_int32()
        L.check(L.load().edb_exec_launches(self.handle, C.byref(n)))
        return n.value

    def launch_info(self, i) -> Dict:
        info = L.LaunchInfo()
        L.check(L.load().edb_exec_launch_info(self.handle, i, C.byref(info)))
        return {f: (list(getattr(info, f)) if f == "seg_kind" else getattr(info, f)) for f, _ in info._fields_}

    def launch_times(self) -> np.ndarray:
        """Per-launch milliseconds of the last profiled execution."""
        n = self.launches()
        out = (C.c_float * n)()
        L.check(L.load().edb_exec_launch_times(self.handle, out, n), "edb_exec_launch_times")
        return np.array(out[:], dtype=np.float64)

    def validate(self, n_workers: int = 512) -> int:
        """edb_exec_validate: host-side check of the device descriptors (raises
        on the first problem); returns the launches and row tiles checked."""
        n = C.c_int64()
        L.check(L.load().edb_exec_validate(self.handle, n_workers, C.byref(n)), "edb_exec_validate")
        return int(n.value)

    def check(self, stream: int = 0):
        """Synchronise and raise if a dataflow wait of the last execution timed out."""
        L.check(L.load().edb_exec_check(self.handle, C.c_void_p(stream)), "edb_exec_check")

    def execute(self, weight_ptrs: Sequence[int], x_ptr: int, arena_h_ptr: int, arena_c_ptr: int, stream: int):
        arr = (C.c_void_p * len(weight_ptrs))(*weight_ptrs)
        L.check(L.load().edb_execute(self.handle, arr, C.c_void_p(x_ptr), C.c_void_p(arena_h_ptr),
                                     C.c_void_p(arena_c_ptr), C.c_void_p(stream)), "edb_execute")

    def split_phase_bytes(self) -> int:
        n = C.c_int64()
        L.check(L.load().edb_split_phase_bytes(self.handle, C.byref(n)), "edb_split_phase_bytes")
        return n.value

    def split_phase(self, x_ptr: int, arena_h_ptr: int, arena_c_ptr: int, buf_ptr: int, buf_bytes: int,
                    stream: int, n_batches: int) -> np.ndarray:
        """Unfused gather and scatter of every batch (edb_split_phase); returns
        [n_batches, 2] kernel durations in ms (gather, scatter)."""
        out = (C.c_float * (2 * n_batches))()
        L.check(L.load().edb_split_phase(self.handle, C.c_void_p(x_ptr), C.c_void_p(arena_h_ptr),
                                         C.c_void_p(arena_c_ptr), C.c_void_p(buf_ptr), buf_bytes,
                                         C.c_void_p(stream), out, 2 * n_batches), "edb_split_phase")
        return np.array(out[:], dtype=np.float64).reshape(n_batches, 2)

    def __del__(self):
        if getattr(self, "handle", None) and L is not None and L._lib is not None:
            L._lib.edb_exec_free(self.handle)
            self.handle = None


class ForwardCall:
    """Argument block of edb_forward for one graph, marshalled once; call()
    then runs the whole path for that mini-batch in a single C call."""

    def __init__(self, op_type, child_ptr, child_idx, x_row, n_types, shapes, cells, policy=L.POLICY_TABLE,
                 encoding=L.ENC_SORT, table=None, plan_mode=L.PLAN_RC, flags=0):
        self._op = _i32(op_type)
        self._ptr = np.ascontiguousarray(child_ptr, dtype=np.int64)
        self._idx = _i32(child_idx) if len(child_idx) else np.zeros(1, dtype=np.int32)
        self._xr = _i32(x_row)
        flat = None
        if table:
            if isinstance(table, dict):
                flat = [len(table)]
                for key, action in table.items():
                    flat += [len(key)] + list(key) + [action]
            else:
                flat = list(table)
        self._tab = _i32(flat) if flat else None
        self._pol = L.Policy(policy, encoding, _ptr(self._tab, C.c_int32) if flat else None, len(flat) if flat else 0)
        self._shapes = (L.OperandShape * len(shapes))(*[L.OperandShape(*s) for s in shapes])
        self._cells = (L.Cell * len(cells))(*cells)
        self.n_nodes, self.n_types = int(self._op.shape[0]), int(n_types)
        self.plan_mode, self.flags = plan_mode, flags
        self._args = (self.n_nodes, self.n_types, _ptr(self._op, C.c_int32), _ptr(self._ptr, C.c_int64),
                      _ptr(self._idx, C.c_int32), _ptr(self._xr, C.c_int32), C.byref(self._pol), self._shapes,
                      plan_mode, self._cells, flags)
        self.n_slots = C.c_int32()

    def call(self, weight_ptrs, x_ptr, arena_h_ptr, arena_c_ptr, arena_rows, stream, keep=False):
        """Run the path; with keep=True return the executor (ExecRecord) for its
        launch records and, under EDB_PROFILE, its per-launch times."""
        arr = (C.c_void_p * len(weight_ptrs))(*weight_ptrs)
        h = C.c_void_p()
        L.check(L.load().edb_forward(*self._args, arr, C.c_void_p(x_ptr), C.c_void_p(arena_h_ptr),
                                     C.c_void_p(arena_c_ptr), arena_rows, C.c_void_p(stream),
                                     C.byref(self.n_slots), C.byref(h) if keep else None), "edb_forward")
        return ExecRecord(h) if keep else None

    def bind(self, weight_ptrs, x_ptr, arena_h_ptr, arena_c_ptr, arena_rows, stream):
        """The arguments of call() marshalled once, for a caller that repeats
        them (a worker with its own stream and arena): returns a function of no
        arguments that runs the path with them."""
        arr = (C.c_void_p * len(weight_ptrs))(*weight_ptrs)
        n_slots = C.c_int32()
        args = self._args + (arr, C.c_void_p(x_ptr), C.c_void_p(arena_h_ptr), C.c_void_p(arena_c_ptr),
                             arena_rows, C.c_void_p(stream), C.byref(n_slots), None)
        fn = L.load().edb_forward

        def run():
            st = fn(*args)
            if st:
                L.check(st, "edb_forward")
        run.keep = (arr, n_slots)   # the marshalled arrays live as long as the function
        return run

    @staticmethod
    def release_stream(stream):
        """edb_stream_release: return the device block that call() keeps for
        `stream` on the current device."""
        L.check(L.load().edb_stream_release(C.c_void_p(stream)), "edb_stream_release")

    def call_noalloc(self, weight_ptrs, x_ptr, arena_h_ptr, arena_c_ptr, arena_rows, stream):
        """The same mini-batch through edb_forward_noalloc (no device
        allocation; the library's fixed per-device array holds the
        executor's device memory)."""
        arr = (C.c_void_p * len(weight_ptrs))(*weight_ptrs)
        L.check(L.load().edb_forward_noalloc(*self._args, arr, C.c_void_p(x_ptr), C.c_void_p(arena_h_ptr),
                                             C.c_void_p(arena_c_ptr), arena_rows, C.c_void_p(stream),
                                             C.byref(self.n_slots)), "edb_forward_noalloc")


class ExecRecord:
    """An executor handed back by edb_forward: launch records and times."""

    def __init__(self, handle):
        self.handle = handle

    def launches(self) -> int:
        n = C.c_int32()
        L.check(L.load().edb_exec_launches(self.handle, C.byref(n)))
        return n.value

    def launch_info(self, i) -> Dict:
        info = L.LaunchInfo()
        L.check(L.load().edb_exec_launch_info(self.handle, i, C.byref(info)))
        return {f: (list(getattr(info, f)) if f == "seg_kind" else getattr(info, f)) for f, _ in info._fields_}

    def launch_times(self) -> np.ndarray:
        n = self.launches()
        out = (C.c_float * n)()
        L.check(L.load().edb_exec_launch_times(self.handle, out, n), "edb_exec_launch_times")
        return np.array(out[:], dtype=np.float64)

    def __del__(self):
        if getattr(self, "handle", None) and L is not None and L._lib is not None:
            L._lib.edb_exec_free(self.handle)
            self.handle = None


def graph_stats() -> Tuple[int, int]:
    """edb_graph_stats: (kernel sequences instantiated as new HIP graphs,
    executions that updated a kept graph in place) in this process."""
    a, b = C.c_int64(), C.c_int64()
    L.check(L.load().edb_graph_stats(C.byref(a), C.byref(b)), "edb_graph_stats")
    return int(a.value), int(b.value)


def operand_shapes(w) -> List[Tuple[int, int, int]]:
    return [(nf, rg, int(KIND_SHAPE[k][2])) for (nf, rg), k in zip(w.shapes(), w.kinds)]


def logical_weights(w, t) -> List[np.ndarray]:
    k = w.kinds[t]
    names = [n for n, _ in weight_shapes(k, w.in_dim, w.hidden, w.n_children[t] or 2)]
    return [w.weights[t][n] for n in names]


def probe_mfma(dtype, n_workgroups: int, iters: int, out_ptr: int, stream: int) -> float:
    """Matrix-core probe (edb_probe_mfma): kernel duration in ms."""
    ms = C.c_float()
    L.check(L.load().edb_probe_mfma(dtype, n_workgroups, iters, C.cast(C.c_void_p(out_ptr), C.POINTER(C.c_float)),
                                    C.c_void_p(stream), C.byref(ms)), "edb_probe_mfma")
    return ms.value


def probe_copy(src_ptr: int, dst_ptr: int, nbytes: int, n_workgroups: int, stream: int) -> float:
    """Device-memory copy probe (edb_probe_copy): kernel duration in ms."""
    ms = C.c_float()
    L.check(L.load().edb_probe_copy(C.c_void_p(src_ptr), C.c_void_p(dst_ptr), nbytes, n_workgroups,
                                    C.c_void_p(stream), C.byref(ms)), "edb_probe_copy")
    return ms.value


LATTICE_TABLE = {(0,): 0, (1,): 1, (0, 1): 0, (1, 0): 1}


class Forward:
    """Everything needed to run the batched forward pass of one workload on
    the current GPU: graph, schedule, plan, packed weights, x, arena."""

    def __init__(self, w, policy=L.POLICY_TABLE, table=None, plan_mode=L.PLAN_RC, flags=L.USE_GRAPH,
                 device="cuda", encoding=L.ENC_SORT):
        import torch
        self.w = w
        self.torch = torch
        if table is None and policy == L.POLICY_TABLE and w.kinds == [6, 7]:
            table = LATTICE_TABLE
        self.graph = Graph(w.op_type, w.child_ptr, w.child_idx, w.x_row, w.n_types)
        self.sched = Schedule(self.graph, policy, encoding, table)
        self.plan = Plan(self.graph, self.sched, operand_shapes(w), plan_mode)
        dt = L.BF16 if w.dtype == "bf16" else L.F32
        self.dtype = dt
        self.cells = [cell_struct(k, w.in_dim, w.hidden, w.n_children[t] if k == NARY_INTERNAL else 0, dt)
                      for t, k in enumerate(w.kinds)]
        self.exec = Exec(self.graph, self.sched, self.plan, self.cells, flags)
        self.flags = flags
        if flags & L.DRYRUN:
            return
        tdt = torch.bfloat16 if dt == L.BF16 else torch.float32
        self.tdt = tdt
        dev = torch.device(device)
        self.stream = torch.cuda.current_stream(dev)
        self.weights = []
        for t in range(w.n_types):
            nb = packed_bytes(self.cells[t])
            buf = torch.empty(nb, dtype=torch.uint8, device=dev)
            pack_weights(self.cells[t], logical_weights(w, t), buf.data_ptr(), self.stream.cuda_stream)
            self.weights.append(buf)
        n_x = max(1, int(w.x.shape[0]))
        if w.x.shape[0] and int(w.x_row.max()) >= w.x.shape[0]:
            raise ValueError("x_row points past the end of x")
        xt = torch.zeros((n_x, max(1, w.in_dim)), dtype=torch.float32)
        if w.x.shape[0]:
            xt[: w.x.shape[0], : w.in_dim] = torch.from_numpy(w.x)
        self.x = xt.to(dev).to(tdt).contiguous()
        H = w.hidden
        self.arena_h = torch.empty((self.plan.n_slots, H), dtype=tdt, device=dev)
        self.arena_c = torch.empty((self.plan.n_slots, H), dtype=torch.float32, device=dev)

    def run(self):
        self.exec.execute([b.data_ptr() for b in self.weights], self.x.data_ptr(), self.arena_h.data_ptr(),
                          self.arena_c.data_ptr(), self.stream.cuda_stream)

    def states(self):
        """Node-ordered (h, c) as float64 numpy arrays (synchronises and checks
        the dataflow launches)."""
        self.exec.check(self.stream.cuda_stream)
        self.torch.cuda.synchronize()
        ah = self.arena_h.float().cpu().numpy().astype(np.float64)
        ac = self.arena_c.cpu().numpy().astype(np.float64)
        s = self.plan.slot
        return ah[s], ac[s]
