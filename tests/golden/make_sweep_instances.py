"""Write sweep_instances.json: every distinct kernel instance the library's
planner picks for the benchmark's calls (tests/shapes.py bench_points), each
with one of its own calls as the representative GPU parity case (the call with
the fewest X + Y bytes; ties go to the earlier call).

    python tests/golden/make_sweep_instances.py

Host-only: it asks the planner (ks_plan_describe) which kernel each call runs;
nothing is launched and no expected value is stored.  Re-run it whenever the
planner changes, then run the GPU suite: tests/test_instance_coverage.py
fails on the CPU until the file matches the planner.
"""
import json
import os
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(HERE))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

import paper_2405_15013_amd as ks  # noqa: E402
from shapes import bench_points  # noqa: E402

OUT = os.path.join(HERE, "sweep_instances.json")


def kernel_of(pattern, batch, dtype, layout):
    desc = ks.ks_plan_describe(*pattern, batch, layout, dtype)
    return dict(kv.split("=", 1) for kv in desc.split())["kernel"]


def xy_bytes(pattern, batch, dtype):
    a, b, c, d = pattern
    if dtype == "fp8":  # E4M3 X, bf16 Y
        return batch * a * d * (2 * b + c)
    return batch * a * d * (b + c) * (4 if dtype == "f32" else 2)


def instances():
    """{kernel: {"case": representative call, "calls": number of calls}}"""
    out = {}
    for pattern, batch, dtype, layout in bench_points():
        k = kernel_of(pattern, batch, dtype, layout)
        case = {"pattern": list(pattern), "batch": batch, "dtype": dtype, "layout": layout}
        e = out.setdefault(k, {"case": case, "calls": 0})
        e["calls"] += 1
        if xy_bytes(pattern, batch, dtype) < xy_bytes(e["case"]["pattern"], e["case"]["batch"], e["case"]["dtype"]):
            e["case"] = case
    return out


def main():
    inst = instances()
    rows = [dict(kernel=k, calls=v["calls"], **v["case"]) for k, v in sorted(inst.items())]
    with open(OUT, "w") as fh:
        json.dump(rows, fh, indent=0)
        fh.write("\n")
    print("%d kernel instances -> %s" % (len(rows), OUT))


if __name__ == "__main__":
    main()
