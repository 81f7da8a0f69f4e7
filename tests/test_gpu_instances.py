"""GPU parity of every kernel instance the planner picks for the benchmark's
calls (tests/golden/sweep_instances.json; the list is kept equal to the
planner's choices by tests/test_instance_coverage.py on the CPU).

Each instance runs once, at its representative call (the real pattern, batch,
layout and storage type of one of its benchmark calls), through the C ABI
into a NaN-prefilled output, and the whole output is compared with the fp64
oracle on the same seeded inputs."""
import json
import os

import pytest

from parity_util import TOL, rel_err
from test_gpu_parity import run_gpu
import oracle
from paper_2405_15013_amd import inputs
import paper_2405_15013_amd as ks

pytestmark = pytest.mark.gpu

HERE = os.path.dirname(os.path.abspath(__file__))
with open(os.path.join(HERE, "golden", "sweep_instances.json")) as _fh:
    LISTED = json.load(_fh)


@pytest.mark.parametrize("row", LISTED, ids=[r["kernel"] for r in LISTED])
def test_instance_against_oracle(row):
    import numpy as np
    pattern, batch, dtype, layout = tuple(row["pattern"]), row["batch"], row["dtype"], row["layout"]
    desc = ks.ks_plan_describe(*pattern, batch, layout, dtype)
    assert ("kernel=" + row["kernel"]) in desc, desc
    print("instance %s: %s B=%d %s %s" % (row["kernel"], pattern, batch, dtype, layout), flush=True)
    if dtype == "fp8":
        from test_gpu_fp8 import run_fp8
        run_fp8(pattern, batch, layout)  # E4M3 inputs, whole bf16 output against the oracle
        return
    x = inputs.make_x(21, pattern, batch, dtype)
    kv = inputs.make_kv(21, pattern, batch, dtype, dist="normal")
    y = run_gpu(pattern, x, kv, batch, dtype, layout)
    assert np.all(np.isfinite(y)), "unwritten (NaN) outputs"
    y64 = oracle.matmul(pattern, inputs.to_f64(kv, dtype), inputs.to_f64(x, dtype), batch, "bsf")
    err = rel_err(y, y64)
    assert err <= TOL[dtype], "%s: rel err %.3e" % (row["kernel"], err)
