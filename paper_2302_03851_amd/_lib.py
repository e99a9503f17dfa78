"""ctypes binding of libedb (include/edb.h).  Argument marshalling only: the
graph, schedule, plan and every kernel run inside the library.  Loading
fails loudly when the library has not been built."""
from __future__ import annotations

import ctypes as C
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libedb.so")

EDB_OK = 0
EDB_ERR_INVALID = -1
EDB_ERR_CYCLE = -2
EDB_ERR_OOM = -3
EDB_ERR_UNSUPPORTED = -4
EDB_ERR_TABLE = -5
EDB_ERR_HIP = -6

POLICY_TABLE, POLICY_AGENDA, POLICY_DEPTH, POLICY_SUFFICIENT = 0, 1, 2, 3
ENC_SORT, ENC_BASE, ENC_MAX = 0, 1, 2
PLAN_RC, PLAN_IDENTITY, PLAN_PQ = 0, 1, 2
SEG_NONE, SEG_CONTIG, SEG_GATHER, SEG_SCATTER = 0, 1, 2, 3
F32, BF16 = 0, 1
USE_GRAPH, DRYRUN, FORCE_GATHER, X_DIRECT, PROFILE, NO_FLOW = 1, 2, 4, 8, 16, 32
NO_SPLIT_K, TILE_LARGE, NO_LARGE, FLOW_DRYRUN = 64, 128, 256, 512
LARGE_VARIANTS = (8, 9, 10, 15, 16)      # large tile size classes 0, 1, 2, 3, 4
LARGE_CLASS = {8: 0, 9: 1, 10: 2, 15: 3, 16: 4}
WS_VARIANT = 17                          # weight-stationary tile (bf16 x-only leaf batches)
STREAM_VARIANTS = (11, 12, 13, 14)        # streamed tile: (rows / 16, waves) = (1, 4), (2, 4), (1, 8), (1, 16)
STREAM_STAGED = {11: 3, 12: 6, 13: 4, 14: 5}   # the staged variant with the same rows and reduction split
PART_CELL, PART_CHILD_SUM, PART_FORGET = 0, 1, 2
FLOW_VARIANT = 100
NOALLOC_SCRATCH_BYTES = 32 << 20   # EDB_NOALLOC_SCRATCH_BYTES

# every symbol include/edb.h declares
EXPORTS = [
    "edb_last_error", "edb_version",
    "edb_build_graph", "edb_graph_free", "edb_graph_info",
    "edb_schedule", "edb_schedule_view", "edb_schedule_free", "edb_lower_bound",
    "edb_learn_defaults", "edb_learn_policy", "edb_learned_view", "edb_learned_q", "edb_learned_free",
    "edb_plan_memory", "edb_plan_view", "edb_plan_free",
    "edb_packed_weight_bytes", "edb_pack_weights",
    "edb_prepare", "edb_execute", "edb_graph_stats", "edb_exec_launches", "edb_exec_launch_info", "edb_exec_launch_times",
    "edb_exec_check", "edb_exec_validate", "edb_exec_free", "edb_forward", "edb_stream_release",
    "edb_forward_noalloc",
    "edb_split_phase_bytes", "edb_split_phase", "edb_probe_mfma", "edb_probe_copy",
]


class EdbError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__(f"edb error {status}: {msg}")
        self.status = status


class Policy(C.Structure):
    _fields_ = [("kind", C.c_int32), ("encoding", C.c_int32),
                ("table", C.POINTER(C.c_int32)), ("table_len", C.c_int64)]


class LearnParams(C.Structure):
    _fields_ = [("encoding", C.c_int32), ("trials", C.c_int32), ("check_every", C.c_int32),
                ("n_step", C.c_int32), ("alpha", C.c_double), ("epsilon", C.c_double), ("lr", C.c_double),
                ("gamma", C.c_double), ("seed", C.c_uint64)]


class LearnStats(C.Structure):
    _fields_ = [("trials", C.c_int32), ("batches", C.c_int32), ("lower_bound", C.c_int64),
                ("n_states", C.c_int32)]


class OperandShape(C.Structure):
    _fields_ = [("n_fixed", C.c_int32), ("ragged", C.c_int32), ("has_x", C.c_int32)]


class Seg(C.Structure):
    _fields_ = [("kind", C.c_int32), ("base", C.c_int32), ("idx_off", C.c_int64),
                ("len", C.c_int32), ("reserved", C.c_int32)]


class PlanView(C.Structure):
    _fields_ = [("n_nodes", C.c_int32), ("n_batches", C.c_int32), ("n_slots", C.c_int32),
                ("n_pads", C.c_int32),
                ("slot", C.POINTER(C.c_int32)), ("order", C.POINTER(C.c_int32)),
                ("x_slot", C.POINTER(C.c_int32)), ("seg_ptr", C.POINTER(C.c_int32)),
                ("segs", C.POINTER(Seg)), ("idx_pool", C.POINTER(C.c_int32)), ("idx_len", C.c_int64),
                ("ragged_off", C.POINTER(C.c_int64)), ("ragged_pool", C.POINTER(C.c_int32)),
                ("ragged_len", C.c_int64), ("pads", C.POINTER(C.c_int32))]


class Cell(C.Structure):
    _fields_ = [("kind", C.c_int32), ("in_dim", C.c_int32), ("hidden", C.c_int32),
                ("n_children", C.c_int32), ("dtype", C.c_int32)]


class LaunchInfo(C.Structure):
    _fields_ = [("batch", C.c_int32), ("kind", C.c_int32), ("m", C.c_int32), ("k", C.c_int32),
                ("n", C.c_int32), ("variant", C.c_int32), ("grid", C.c_int32), ("block", C.c_int32),
                ("seg_kind", C.c_int32 * 4), ("n_batches", C.c_int32), ("part", C.c_int32)]


_lib = None


def load():
    """Load libedb.so and declare its signatures; raises if it is missing."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"libedb.so not built ({LIB_PATH}); run __graft_entry__.build() "
                           "or python -m paper_2302_03851_amd.build")
    lib = C.CDLL(LIB_PATH)
    P = C.POINTER
    vp = C.c_void_p
    sig = {
        "edb_last_error": (C.c_char_p, []),
        "edb_version": (C.c_int32, []),
        "edb_build_graph": (C.c_int32, [C.c_int32, C.c_int32, P(C.c_int32), P(C.c_int64), P(C.c_int32),
                                        P(C.c_int32), P(vp)]),
        "edb_graph_free": (None, [vp]),
        "edb_graph_info": (C.c_int32, [vp, P(C.c_int32), P(C.c_int32), P(C.c_int64)]),
        "edb_schedule": (C.c_int32, [vp, P(Policy), P(vp)]),
        "edb_schedule_view": (C.c_int32, [vp, P(C.c_int32), P(P(C.c_int32)), P(P(C.c_int32)),
                                          P(P(C.c_int32))]),
        "edb_schedule_free": (None, [vp]),
        "edb_lower_bound": (C.c_int32, [vp, P(C.c_int64)]),
        "edb_learn_defaults": (None, [P(LearnParams)]),
        "edb_learn_policy": (C.c_int32, [vp, P(LearnParams), P(vp)]),
        "edb_learned_view": (C.c_int32, [vp, P(P(C.c_int32)), P(C.c_int64), P(LearnStats)]),
        "edb_learned_q": (C.c_int32, [vp, P(C.c_int32), P(P(C.c_int32)), P(C.c_int64), P(P(C.c_double))]),
        "edb_learned_free": (None, [vp]),
        "edb_plan_memory": (C.c_int32, [vp, vp, P(OperandShape), C.c_int32, P(vp)]),
        "edb_plan_view": (C.c_int32, [vp, P(PlanView)]),
        "edb_plan_free": (None, [vp]),
        "edb_packed_weight_bytes": (C.c_int32, [P(Cell), P(C.c_int64)]),
        "edb_pack_weights": (C.c_int32, [P(Cell), P(P(C.c_float)), vp, vp]),
        "edb_prepare": (C.c_int32, [vp, vp, vp, P(Cell), C.c_int32, P(vp)]),
        "edb_execute": (C.c_int32, [vp, P(vp), vp, vp, vp, vp]),
        "edb_graph_stats": (C.c_int32, [P(C.c_int64), P(C.c_int64)]),
        "edb_exec_launches": (C.c_int32, [vp, P(C.c_int32)]),
        "edb_exec_launch_info": (C.c_int32, [vp, C.c_int32, P(LaunchInfo)]),
        "edb_exec_launch_times": (C.c_int32, [vp, P(C.c_float), C.c_int32]),
        "edb_exec_check": (C.c_int32, [vp, vp]),
        "edb_exec_validate": (C.c_int32, [vp, C.c_int32, P(C.c_int64)]),
        "edb_exec_free": (None, [vp]),
        "edb_forward": (C.c_int32, [C.c_int32, C.c_int32, P(C.c_int32), P(C.c_int64), P(C.c_int32), P(C.c_int32),
                                    P(Policy), P(OperandShape), C.c_int32, P(Cell), C.c_int32, P(vp), vp, vp, vp,
                                    C.c_int64, vp, P(C.c_int32), P(vp)]),
        "edb_stream_release": (C.c_int32, [vp]),
        "edb_forward_noalloc": (C.c_int32, [C.c_int32, C.c_int32, P(C.c_int32), P(C.c_int64), P(C.c_int32),
                                            P(C.c_int32), P(Policy), P(OperandShape), C.c_int32, P(Cell),
                                            C.c_int32, P(vp), vp, vp, vp, C.c_int64, vp, P(C.c_int32)]),
        "edb_split_phase_bytes": (C.c_int32, [vp, P(C.c_int64)]),
        "edb_split_phase": (C.c_int32, [vp, vp, vp, vp, vp, C.c_int64, vp, P(C.c_float), C.c_int32]),
        "edb_probe_mfma": (C.c_int32, [C.c_int32, C.c_int32, C.c_int32, P(C.c_float), vp, P(C.c_float)]),
        "edb_probe_copy": (C.c_int32, [vp, vp, C.c_int64, C.c_int32, vp, P(C.c_float)]),
    }
    for name, (res, args) in sig.items():
        f = getattr(lib, name)
        f.restype = res
        f.argtypes = args
    _lib = lib
    return lib


def check(status, what=""):
    if status != EDB_OK:
        msg = load().edb_last_error().decode()
        raise EdbError(status, f"{what}: {msg}" if what else msg)
