"""Host-side pieces of bench.py: the roofline of a point, the profiler
counter parsing and the traffic record lookup (no GPU)."""
import json
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402


def test_sweep_has_700_patterns():
    pats = bench.sweep_patterns()
    assert len(pats) == 700
    assert all(a * b * d <= 8192 and a * c * d <= 8192 for a, b, c, d in pats)


def test_roof_bytes_and_bound():
    # fp32, (1, 64, 64, 1), batch 4096: X, Y 4096*64 each, K 64*64 (paper Section 4.3 traffic).
    nbytes, flops, t, bound = bench.roof((1, 64, 64, 1), 4096, "f32")
    assert nbytes == (4096 * 64 * 2 + 64 * 64) * 4
    assert flops == 2.0 * 4096 * 64 * 64
    assert bound == "hbm" and abs(t - nbytes / bench.HBM_BW) < 1e-15
    # bf16 with large b*c stays HBM-bound on the MFMA peak.
    assert bench.roof((1, 128, 128, 64), 25088, "bf16")[3] == "hbm"


def _write_counter_csv(path, rows):
    with open(path, "w") as fh:
        fh.write('"Dispatch_Id","Kernel_Name","Counter_Name","Counter_Value"\n')
        for did, name, ctr, val in rows:
            fh.write('%d,"%s","%s",%s\n' % (did, name, ctr, val))


def test_counter_per_dispatch_sums_instances_and_filters(tmp_path):
    p = tmp_path / "c.csv"
    _write_counter_csv(p, [
        (1, "void ks::ks_staged_kernel<float, 0, 4, true, 2, 1>(ks::Problem, ks::StagedTile)", "FETCH_SIZE", 10),
        (1, "void ks::ks_staged_kernel<float, 0, 4, true, 2, 1>(ks::Problem, ks::StagedTile)", "FETCH_SIZE", 5),
        (2, "void ks::ks_staged_kernel<float, 0, 4, true, 1, 1>(ks::Problem, ks::StagedTile)", "FETCH_SIZE", 7),
        (3, "__amd_rocclr_copyBuffer", "FETCH_SIZE", 3),
    ])
    per, names = bench.counter_per_dispatch(str(p), "FETCH_SIZE", "ks_staged_kernel<float,0,4,true,2,1>")
    assert per == {"1": 15.0}
    per, _ = bench.counter_per_dispatch(str(p), "FETCH_SIZE", "copy")
    assert per == {"3": 3.0}
    assert len(bench.counter_per_dispatch(str(p), "FETCH_SIZE")[0]) == 3


def test_pmc_summary_scales_by_copy_calibration(tmp_path):
    k = "ks_staged_kernel<float,0,4,true,2,1>"
    kname = "void ks::ks_staged_kernel<float, 0, 4, true, 2, 1>(ks::Problem, ks::StagedTile)"
    fill = "void at::native::vectorized_elementwise_kernel<16, FillFunctor>"
    cal_kib = 64 * 1024  # 64 MiB
    _write_counter_csv(tmp_path / "copy_fetch.csv", [(i, "__amd_rocclr_copyBuffer", "FETCH_SIZE", cal_kib / 2)
                                                     for i in range(5)] + [(9 + i, fill, "FETCH_SIZE", 0)
                                                                           for i in range(8)])
    _write_counter_csv(tmp_path / "copy_write.csv", [(i, "__amd_rocclr_copyBuffer", "WRITE_SIZE", cal_kib)
                                                     for i in range(5)])
    # Two dispatches, 1000 and 3000 KiB fetched (counter) -> mean 2000 KiB x2 scale.
    _write_counter_csv(tmp_path / "fetch.csv", [(1, kname, "FETCH_SIZE", 600), (1, kname, "FETCH_SIZE", 400),
                                                (2, kname, "FETCH_SIZE", 3000)])
    _write_counter_csv(tmp_path / "write.csv", [(1, kname, "WRITE_SIZE", 100), (2, kname, "WRITE_SIZE", 300)])
    line = {"config": {"sample_every": 1}, "sources_sha1": "abc",
            "roofline": {"kernel": k, "algorithmic_bytes_per_launch": 4.0e6, "timed_calls": 6, "points": 1}}
    (tmp_path / "bench.json").write_text("[bench] progress\n" + json.dumps(line) + "\n")
    out = tmp_path / "t.md"
    bench.pmc_summary(str(tmp_path), str(out), ["cmd"])
    rec = [json.loads(x[len(bench.TRAFFIC_TAG):]) for x in out.read_text().splitlines()
           if x.startswith(bench.TRAFFIC_TAG)][0]
    assert abs(rec["fetch_scale"] - 2.0) < 1e-12 and abs(rec["write_scale"] - 1.0) < 1e-12
    assert rec["fetch_bytes_per_launch"] == 2000 * 1024 * 2.0
    assert rec["write_bytes_per_launch"] == 200 * 1024
    assert rec["dispatches"] == [2, 2]


def test_traffic_record_needs_current_sources(tmp_path, monkeypatch):
    k = "ks_x_kernel<float>"
    pdir = tmp_path / "profiles"
    pdir.mkdir()
    rec = {"kernel": k, "sources_sha1": bench.kernel_sources_sha1("ks_dma_kernel<float>"), "sample_every": 1,
           "traffic_bytes_per_launch": 123.0}
    (pdir / "a.md").write_text("# x\n" + bench.TRAFFIC_TAG + json.dumps(rec) + "\n")
    stale = dict(rec, kernel="ks_y_kernel<float>", sources_sha1="0" * 40)
    (pdir / "b.md").write_text(bench.TRAFFIC_TAG + json.dumps(stale) + "\n")
    # The records are read from ROOT/profiles; the hash stays the real tree's.
    sha = rec["sources_sha1"]
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    monkeypatch.setattr(bench, "kernel_sources_sha1", lambda kernel=None: sha)
    assert bench.traffic_record(k, 1)["traffic_bytes_per_launch"] == 123.0
    assert bench.traffic_record(k, 2) is None
    assert bench.traffic_record("ks_y_kernel<float>", 1) is None


def test_plan_kernel_names_are_library_symbols():
    """The kernel= field of ks_plan_describe names a kernel instance that the
    library contains (profiler summaries and counter passes select dispatches
    by that name), for every variant the automatic planner picks on a sample
    of the sweep."""
    import shutil
    import subprocess
    import pytest
    import paper_2405_15013_amd as ks
    nm = shutil.which("nm")
    if nm is None or not os.path.exists(ks.library_path()):
        pytest.skip("needs nm and the built library")
    out = subprocess.run([nm, "-C", ks.library_path()], capture_output=True, text=True, check=True).stdout
    syms = {line.split(" ", 2)[2].replace(" ", "").split("(")[0].replace("voidks::", "")
            for line in out.splitlines() if " ks::ks_" in line and "__device_stub" not in line}
    seen = set()
    for p in bench.sweep_patterns()[::9] + [(2, 4, 4, 2), (16, 2, 2, 32), (3, 5, 7, 2)]:
        for layout in ("bsf", "bsl"):
            for dtype in ("f32", "bf16"):
                for batch in (4096, 25088, 100):
                    name = bench.plan_field(ks.ks_plan_describe(*p, batch, layout, dtype), "kernel")
                    seen.add(name)
    missing = sorted(n for n in seen if n not in syms)
    assert not missing, missing[:5]
    assert any(n.startswith("ks_dma_kernel<") for n in seen) and any(n.startswith("ks_direct_c_kernel<") for n in seen)


def test_copy_floor_frac_interpolates_in_log_bytes():
    rows = [{"bytes": 1 << 20, "us": 2.0}, {"bytes": 4 << 20, "us": 4.0}]
    # at the measured sizes: bytes / 8 TB/s / time
    assert abs(bench.copy_floor_frac(rows, 1 << 20) - (1 << 20) / 8e12 / 2e-6) < 1e-12
    # halfway in log(bytes) between 1 and 4 MiB: time halfway, 3 us
    assert abs(bench.copy_floor_frac(rows, 2 << 20) - (2 << 20) / 8e12 / 3e-6) < 1e-12
    # beyond the largest size: the largest size's rate
    assert abs(bench.copy_floor_frac(rows, 8 << 20) - bench.copy_floor_frac(rows, 4 << 20)) < 1e-12


def test_points_summary_tables(tmp_path):
    pats = bench.sweep_patterns()
    recs = []
    for i, p in enumerate(pats[:40]):
        for dtype in ("f32", "bf16"):
            recs.append({"pattern": list(p), "batch": 4096, "dtype": dtype, "layout": "bsl", "us": 5.0,
                         "epilogue": None, "gbps": 1000.0 + i, "frac": 0.01 * (i + 1), "bound": "hbm",
                         "bytes": 1 << 20, "kernel": "k%d" % i})
    recs.append(dict(recs[0], pattern=[2, 2, 2, 512]))  # a family point: not a sweep pattern
    pts = tmp_path / "points.jsonl"
    pts.write_text("\n".join(json.dumps(r) for r in recs) + "\n")
    floor = tmp_path / "floor.json"
    floor.write_text(json.dumps({"copy_floor": [{"bytes": 1 << 20, "us": 2.0, "frac": 0.06}]}))
    out = tmp_path / "summary.md"
    bench.points_summary(str(pts), str(out), ["cmd"], str(floor), lowest=5)
    text = out.read_text()
    assert "| f32 BSL B=4096 | 40 |" in text and "| bf16 BSL B=4096 | 40 |" in text
    assert "(2, 2, 2, 512)" not in text
    assert text.count("`k0`") == 2 and "0.010" in text  # the lowest point of each dtype listed


def test_kernel_family_hash_covers_its_sources_only():
    """The traffic record of a kernel family is keyed on the sources that build
    it (its translation units, their headers, its planners): another family's
    source does not change it, a shared header does."""
    dma = bench.kernel_sources_sha1("ks_dma_kernel<float,4,true,1,4,4,2>")
    assert dma == bench.kernel_sources_sha1("ks_dma_kernel<unsignedshort,1,false,1,8,2,4>")
    assert dma != bench.kernel_sources_sha1("ks_fp8_kernel<0,8>")
    files = [os.path.basename(p) for p in bench._include_closure(
        [os.path.join(bench.ROOT, "paper_2405_15013_amd", "csrc", "ks_dma_f32_v1.hip")])]
    assert "ks_dma.h" in files and "ks_direct.h" in files and "ks_fp8.hip" not in files


def test_chain_summary_tables(tmp_path):
    stats = tmp_path / "stats.csv"
    stats.write_text('"Name","Calls","TotalDurationNs","AverageNs","Percentage","MinNs","MaxNs","StdDev"\n'
                     '"void ks::(anonymous namespace)::ks_chain_bfly_kernel<float, 1, true, 5, 5>(ks::FusedChain)",'
                     '20,200000,10000.0,50.0,9000,11000,100.0\n'
                     '"void ks::(anonymous namespace)::ks_dma_kernel<float, 4, true, 1, 4, 4, 2>(ks::Problem)",'
                     '5,100,20.0,1.0,10,30,1.0\n')
    recs = tmp_path / "chains.jsonl"
    recs.write_text(json.dumps({"chain": [[1, 2, 2, 1]] * 10, "batch": 4096, "dtype": "f32", "layout": "bsl",
                                "path": "fused-bfly", "us": 11.9, "launch_us_median": 14.0,
                                "fused_lower_bound_us": 4.2, "frac_fused_bound": 0.353}) + "\n")
    out = tmp_path / "out.md"
    bench.chain_summary(str(stats), str(recs), str(out), ["python3 bench.py --chains chains.jsonl"])
    text = out.read_text()
    assert "| butterfly 10 | 4096 | f32 | BSL | fused-bfly | 11.90 | 14.00 | 4.20 | 0.353 |" in text
    assert "`void ks::ks_chain_bfly_kernel<float, 1, true, 5, 5>(ks::FusedChain)` | 20 | 10.00 | 9.00 | 11.00 |" in text
    assert "ks_dma_kernel" not in text
