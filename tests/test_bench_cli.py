"""Host logic of bench.py that runs without a GPU: the one-GPU contract, the
visit ceiling it prices the walks against, and the staleness rule of the
committed HBM-traffic counters."""
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402


@pytest.mark.parametrize("gpus", [2, 8])
def test_more_than_one_gpu_is_refused(gpus):
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", str(gpus)],
                       capture_output=True, text=True, timeout=120, cwd=ROOT)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout.strip() == ""  # no JSON line for an unsupported run


def test_visit_ceiling_from_unit_counts():
    # 256 CUs at 2.4 GHz: LDS 256 B/clk/CU over 12 B per visit, VALU 128
    # lanes/clk/CU over the 5 instructions per visit counted on the walks
    # (SQ_INSTS_VALU per wave-visit 5.01 / 5.27); the lower one is the peak.
    lds = 256 * 256 * 2.4e9 / 12
    valu = 256 * 128 * 2.4e9 / 5
    assert bench.VISIT_PEAK_LDS == pytest.approx(lds)
    assert bench.VISIT_PEAK_VALU == pytest.approx(valu)
    assert bench.VISIT_PEAK_VALU == pytest.approx(15.72864e12)
    assert bench.VISIT_PEAK_PER_S == pytest.approx(min(lds, valu))
    assert bench.VISIT_PEAK_PER_S == pytest.approx(13.1072e12)


def test_probe_shape_is_the_perf_walk_shape():
    # the walk-loop ceiling is taken at the 16M pool's perf walk shape:
    # depth 8, four trees per lane, two lanes per candidate, eight waves,
    # 128 features
    import gen
    w = gen.WORKLOADS["roofline"]
    d, g, s, waves, f = bench.PERF_WALK_SHAPE["roofline"]
    assert d == w.p_depth and f == w.F and (g, s, waves) == (4, 2, 8)
    # the other shapes: depth and the columns P reads of their workloads
    for name, (d, g, s, waves, f) in bench.PERF_WALK_SHAPE.items():
        w = gen.WORKLOADS[name]
        assert d == w.p_depth and f == (w.K if w.visible_only else w.F)
    # the validity walk's: V's depth and the columns V reads
    assert set(bench.VALIDITY_WALK_SHAPE) == set(bench.PERF_WALK_SHAPE)
    for name, (d, g, s, waves, f) in bench.VALIDITY_WALK_SHAPE.items():
        w = gen.WORKLOADS[name]
        assert d == w.v_depth and f == (w.K if w.visible_only else w.F)


def test_mall_flush_applies_to_pools_below_the_cache():
    import gen
    small = [n for n, w in gen.WORKLOADS.items() if 4.0 * w.F * w.n < bench.MALL_BYTES]
    assert sorted(small) == ["medium", "tiny"]


def test_traffic_only_for_the_profiled_source(tmp_path, monkeypatch):
    sha = bench._kernel_sha()
    f = tmp_path / "traffic.json"
    f.write_text(json.dumps({"kernel_source_sha256": sha,
                             "launches": {"roofline": {"bytes_per_launch": 123.0}}}))
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(f))
    assert bench._traffic(sha, "roofline") == 123.0
    assert bench._traffic(sha, "hbm") is None  # no counters for that workload
    assert bench._traffic("0" * 64, "roofline") is None  # counters taken on other source
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(tmp_path / "missing.json"))
    assert bench._traffic(sha, "roofline") is None


def test_committed_traffic_matches_current_source():
    """The committed counters were taken on the walk kernels as they stand;
    a kernel change makes bench.py report traffic as null until the
    counters are taken again."""
    with open(bench.TRAFFIC_FILE) as fh:
        t = json.load(fh)
    if t["kernel_source_sha256"] != bench._kernel_sha():
        pytest.skip("walk kernels changed since the counters were taken (traffic reported null)")
    copy = t["copy_probe"]
    assert set(t["launches"]) == {"roofline", "hbm"}
    for launch in t["launches"].values():
        want = (launch["fetch_size_kib"] * 1024 / copy["fetch_factor"]
                + launch["write_size_kib"] * 1024 / copy["write_factor"])
        assert launch["bytes_per_launch"] == pytest.approx(want, rel=1e-9)
