"""Host-side guard of the GPU instance coverage (no GPU): the kernel instances
the planner picks for the benchmark's calls are exactly those listed in
tests/golden/sweep_instances.json, which tests/test_gpu_instances.py runs
one by one against the oracle.  A planner change that brings in an instance
the GPU suite has never run fails here until the list is regenerated
(tests/golden/make_sweep_instances.py) and the GPU suite is run on it."""
import json
import os
import sys

import pytest

import paper_2405_15013_amd as ks

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.join(HERE, "golden"))
import make_sweep_instances as msi  # noqa: E402

with open(msi.OUT) as _fh:
    LISTED = json.load(_fh)


def test_listed_instances_are_the_planned_ones():
    planned = msi.instances()
    listed = {r["kernel"] for r in LISTED}
    missing = sorted(set(planned) - listed)
    assert not missing, "planned kernel instances with no GPU parity case: %s" % missing[:10]
    stale = sorted(listed - set(planned))
    assert not stale, "listed instances the planner no longer picks: %s" % stale[:10]


@pytest.mark.parametrize("row", LISTED, ids=[r["kernel"] for r in LISTED])
def test_representative_call_runs_its_instance(row):
    """The listed call still runs the listed instance, and the host replay of
    its launch at that full batch stays in bounds and writes every output
    once."""
    assert msi.kernel_of(tuple(row["pattern"]), row["batch"], row["dtype"], row["layout"]) == row["kernel"]
    st, rep = ks.ks_plan_verify(*row["pattern"], row["batch"], row["layout"], row["dtype"])
    assert st == 0, rep
