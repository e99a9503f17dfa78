"""Host-side validation of the uploaded descriptors (edb_exec_validate) on
dry-run executors of all nine workloads, in every layout and tile mode, and
of the dataflow launches' descriptors and ticket protocol (built on the host
only: the dataflow launch is switched off on the GPU).  CPU only."""
import pytest

from paper_2302_03851_amd import _lib as L
from paper_2302_03851_amd import edb
from paper_2302_03851_amd import workloads as WL

INSTANCES = {1: None, 2: None, 3: None, 4: None, 5: 64, 6: None, 7: None, 8: 16, 9: None}
MODES = [dict(flags=L.DRYRUN), dict(flags=L.DRYRUN | L.FLOW_DRYRUN), dict(flags=L.DRYRUN | L.TILE_LARGE),
         dict(flags=L.DRYRUN | L.FORCE_GATHER | L.X_DIRECT), dict(flags=L.DRYRUN, plan_mode=L.PLAN_IDENTITY),
         dict(flags=L.DRYRUN | L.FLOW_DRYRUN, plan_mode=L.PLAN_PQ)]


@pytest.mark.parametrize("k", sorted(INSTANCES))
def test_descriptors_validate(k):
    w = WL.make_config(k, instances=INSTANCES[k])
    for kw in MODES:
        if kw.get("plan_mode") == L.PLAN_PQ and k in (8, 9):
            continue   # the PQ-tree layout takes the tree and lattice workloads of configs 1-7
        f = edb.Forward(w, **kw)
        n = f.exec.validate(n_workers=64)
        assert n >= f.sched.n_batches, (k, kw, n)
        if kw["flags"] & L.FLOW_DRYRUN:
            flows = [f.exec.launch_info(i) for i in range(f.exec.launches())
                     if f.exec.launch_info(i)["variant"] == L.FLOW_VARIANT]
            # runs of consecutive small batches exist in the tree, chain, grid and lattice schedules
            if k in (1, 2, 3, 4, 5, 6, 7):
                assert flows, (k, kw)
            for W in (1, 3, 512):
                f.exec.validate(n_workers=W)


def test_flow_dryrun_needs_dryrun():
    w = WL.make_config(1)
    with pytest.raises(L.EdbError) as ei:
        edb.Forward(w, flags=L.FLOW_DRYRUN)
    assert ei.value.status == L.EDB_ERR_INVALID
