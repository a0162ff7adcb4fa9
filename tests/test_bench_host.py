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
