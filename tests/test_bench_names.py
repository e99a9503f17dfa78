"""The benchmark's kernel names: the symbol a launch's kernel has in a
rocprofv3 trace (which the profile summaries and the traffic counters are
looked up by) and its readable name, per tile family."""
import os
import sys

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))

import bench  # noqa: E402
from paper_2302_03851_amd import _lib as L  # noqa: E402


def test_kernel_symbols_per_tile_family():
    assert bench.kernel_symbol(2, "f32", 11, 0) == "edbk::stream_kernel<2, float, 1, 4>"
    assert bench.kernel_symbol(5, "bf16", 4, 0) == "edbk::cell_kernel<5, __bf16, 1, 1, 8>"
    assert bench.kernel_symbol(1, "f32", 15, 0) == "edbk::big_kernel<1, float, 3>"
    # child-sum batches on the large tile: forget GEMM (part 2), sums (part 1), parents (part 0)
    assert bench.kernel_symbol(5, "bf16", 10, 2) == "edbk::big_kernel<15, __bf16, 2>"
    assert bench.kernel_symbol(5, "bf16", 10, 1) == "edbk::child_reduce_kernel"
    assert bench.kernel_symbol(5, "bf16", 16, 0) == "edbk::big_kernel<16, __bf16, 4>"
    assert bench.kernel_symbol(4, "bf16", L.WS_VARIANT, 0) == "edbk::ws_kernel<4>"
    assert bench.kernel_symbol(12, "f32", 3, 1) == "edbk::mv_matvec_kernel"


def test_kernel_names_per_tile_family():
    assert bench.kernel_name(2, 11, 0, "f32") == "stream_kernel<NARY_INTERNAL, f32, variant 11>"
    assert bench.kernel_name(4, L.WS_VARIANT, 0, "bf16") == "ws_kernel<CS_LEAF, bf16>"
    assert bench.kernel_name(5, 10, 2, "bf16") == "big_kernel<CS_FORGET, bf16, size class 2>"
    assert bench.kernel_name(5, 16, 0, "bf16") == "big_kernel<CS_PARENT, bf16, size class 4>"
    assert bench.kernel_name(5, 4, 0, "bf16") == "cell_kernel<CS_INTERNAL, bf16, variant 4>"
    assert bench.kernel_name(5, 10, 1, "bf16") == "child_reduce_kernel"


def test_launch_work_of_split_batches():
    """A child-sum batch on the large tile counts its forget GEMM in part 2,
    nothing in part 1 and the parents' GEMM in part 0; an unsplit batch counts
    both."""
    work = {0: (100.0, 40.0, 0.0), 1: (10.0, 4.0, 0.0)}
    split = {0}
    assert bench.launch_work({"batch": 0, "part": 2, "kind": 5}, work, split) == 40.0
    assert bench.launch_work({"batch": 0, "part": 1, "kind": 5}, work, split) == 0
    assert bench.launch_work({"batch": 0, "part": 0, "kind": 5}, work, split) == 100.0
    assert bench.launch_work({"batch": 1, "part": 0, "kind": 5}, work, split) == 14.0
