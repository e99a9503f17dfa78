"""The instance-by-instance evaluation that the full-size GPU tests use
gives bitwise the oracle's whole-graph result (CPU only)."""
import numpy as np
import pytest

from oracle.evaluate import evaluate_workload
from oracle_instances import components, evaluate_by_instance
from paper_2302_03851_amd import workloads as WL


@pytest.mark.parametrize("k,inst", [(1, 8), (2, 5), (3, 4), (4, 2), (5, 3), (6, 5), (7, 5)])
def test_instances_equal_whole_graph(k, inst):
    w = WL.make_config(k, instances=inst)
    assert len(np.unique(components(w))) == inst
    h, c = evaluate_workload(w)
    for workers in (1, 3):
        hi, ci = evaluate_by_instance(w, workers=workers)
        np.testing.assert_array_equal(hi, h)
        np.testing.assert_array_equal(ci, c)
