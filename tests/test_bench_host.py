"""bench.py's host-side bookkeeping (no GPU): ideal and algorithmic bytes, and
the lookup of committed counter records."""
import json

import bench


def test_ideal_bytes():
    B, N, P, C, s = 4, 65536, 65536, 128, 2
    xy = B * N * C * s
    assert bench.ideal_bytes("forward", B, N, P, C, s) == 2 * xy + 4 * P * C
    assert bench.ideal_bytes("separable", B, N, P, C, s) == 2 * xy + 4 * (P + C)
    assert bench.ideal_bytes("module", B, N, P, C, s) == 2 * xy + 4 * P * C + 2 * C * C * s
    assert bench.ideal_bytes("backward", B, N, P, C, s) == 3 * xy + 8 * P * C


def test_module_algorithmic_bytes_and_flops():
    names = ["module_outer_fwd", "middle", "module_outer_inv"]
    b, f = bench.module_algorithmic(names, 4, 65536, 65536, 128, 2, 4 * 65536 * 128)
    L = 65536 * 128
    assert b == [4 * L * 2 + 4 * L * 4 + 128 * 128 * 2, 4 * L * 8 + 4 * L, 4 * L * 4 + 4 * L * 2 + 128 * 128 * 2]
    assert f == [2 * 4 * 65536 * 128 * 128, 0, 2 * 4 * 65536 * 128 * 128]
    assert bench.module_kernels("three_pass", "mfma") == names
    assert bench.module_kernels("three_pass", "unfused") == ["unfused"]
    assert bench.module_kernels("fused", "mfma") == ["module_fused"]
    assert bench.module_kernels("small", "small") == ["module_small"]


def test_traffic_lookup_tolerates_every_record(tmp_path, monkeypatch):
    """The committed record loads without error, and a record taken on other
    sources (or in an older format) is not reported."""
    assert bench.load_traffic("middle", "stereo64k_bf16", "forward") in (None,) or \
        isinstance(bench.load_traffic("middle", "stereo64k_bf16", "forward"), int)
    assert bench.load_traffic("middle", "stereo64k_bf16", "backward") is None
    path = tmp_path / "traffic.json"
    monkeypatch.setattr(bench, "TRAFFIC_PATH", str(path))
    for rec in [{"source_hash": "abc"}, {"source_hash": {"forward": "x"}}, {}]:
        path.write_text(json.dumps(rec))
        assert bench.load_traffic("middle", "stereo64k_bf16", "forward") is None
    good = {"source_hash": {"forward": bench.kernel_source_hash(bench.FORWARD_SOURCES)},
            "workloads": {"stereo64k_bf16": {"forward": {"middle": {"hbm_bytes_per_launch": 7}}}}}
    path.write_text(json.dumps(good))
    assert bench.load_traffic("middle", "stereo64k_bf16", "forward") == 7
    assert bench.load_traffic("middle", "stereo64k_bf16", "module") is None


def test_input_sets_exceed_twice_the_infinity_cache():
    """Every workload rotates over sets whose footprint is >= 2x the cache
    (the cap only binds below 256 KiB per set)."""
    for fp in (786432, 41943040, 68157440, 167772160, 536870912):
        n = bench.input_sets(fp)
        assert n * fp >= 2 * bench.MALL_BYTES and n >= 2


def test_whole_call_traffic_sums_kernels(tmp_path, monkeypatch):
    path = tmp_path / "traffic.json"
    monkeypatch.setattr(bench, "TRAFFIC_PATH", str(path))
    rec = {"source_hash": {"forward": bench.kernel_source_hash(bench.FORWARD_SOURCES)},
           "workloads": {"w": {"forward": {"outer_fwd": {"hbm_bytes_per_launch": 3},
                                           "middle": {"hbm_bytes_per_launch": 5}}}}}
    path.write_text(json.dumps(rec))
    assert bench.call_traffic(["outer_fwd", "middle"], "w", "forward") == 8
    assert bench.call_traffic(["outer_fwd", "middle", "outer_inv"], "w", "forward") is None


def test_one_launch_design_bytes_are_the_three_passes():
    three = bench.algorithmic_bytes("three_pass", 1, 1024, 64, 4, 4 * 1024 * 64)
    assert bench.algorithmic_bytes("one_launch", 1, 1024, 64, 4, 4 * 1024 * 64) == [sum(three)]
    p = bench.percentiles([1.0, 2.0, 3.0])
    assert p["median_ms"] == 2.0 and p["calls"] == 3


def test_backward_plan_follows_the_library_rule():
    def p(plan, K):
        return {"plan": plan, "log2_slice": K}
    assert bench.backward_plan(p("wave_tiles", 16)) == "three_pass"
    assert bench.backward_plan(p("wave_tiles", 15)) == "fused"
    assert bench.backward_plan(p("one_launch", 13)) == "three_pass"
    assert bench.backward_plan(p("fused", 16)) == "three_pass"
    assert bench.backward_plan(p("fused", 14)) == "fused"
    assert bench.backward_plan(p("three_pass", 23)) == "three_pass"
    assert bench.kernel_names("wave_tiles") == ["wave_pass1", "wave_middle", "wave_pass3"]
