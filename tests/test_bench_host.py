"""Host logic of bench.py that needs no GPU: the per-workload traffic ratio is
read from the committed counter summary only for the workload that was
measured and only while the forward's sources hash as they did then."""
import os

import pytest

import bench


def test_traffic_ratio_per_workload(tmp_path, monkeypatch):
    h = bench.ffn_source_hash()
    f = tmp_path / "traffic.md"
    f.write_text("# summary\n"
                 f"traffic: config=wide_offload source_hash={h} ratio=1.0571 counted_MB=1 algorithmic_MB=1\n"
                 f"traffic: config=batched_8x64 source_hash={h} ratio=1.1300 counted_MB=1 algorithmic_MB=1\n"
                 "traffic: config=qwen3_30b_a3b source_hash=0000000000000000 ratio=1.0283\n")
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(f))
    assert bench.measured_traffic("wide_offload") == pytest.approx(1.0571)
    assert bench.measured_traffic("batched_8x64") == pytest.approx(1.13)
    assert bench.measured_traffic("qwen3_30b_a3b") is None     # measured on other kernels
    assert bench.measured_traffic("fp32_small") is None        # never measured
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(tmp_path / "missing.md"))
    assert bench.measured_traffic("wide_offload") is None


def test_committed_summary_matches_sources():
    """The committed counter summary covers the three workloads the bench
    line reports, measured on the current forward sources."""
    assert os.path.exists(bench.TRAFFIC_FILE)
    for cfg in ("wide_offload", "qwen3_30b_a3b", "batched_8x64"):
        r = bench.measured_traffic(cfg)
        assert r is not None and 1.0 <= r < 1.5, (cfg, r)


def test_multi_gpu_request_exits(monkeypatch, capsys):
    monkeypatch.setattr("sys.argv", ["bench.py", "--gpus", "2"])
    with pytest.raises(SystemExit) as e:
        bench.main()
    assert e.value.code == 2
    assert "one GPU" in capsys.readouterr().err
