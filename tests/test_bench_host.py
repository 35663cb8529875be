"""Host logic of bench.py (CPU): the one-GPU refusal and the stored traffic
record, which is used only while the kernel sources it was taken on hash to
the recorded value."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_more_than_one_gpu_is_refused_before_any_gpu_work():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU only" in r.stderr
    assert r.stdout == ""


def test_traffic_record_is_used_only_for_the_recorded_sources(monkeypatch, tmp_path):
    src = tmp_path / "kernel.hip"
    src.write_text("// kernel source\n")
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    h = bench.source_hash(["kernel.hip"])
    rec = tmp_path / "pmc_traffic.md"
    rec.write_text("# traffic\n\n```json\n{\"entries\": {\"bwd_loop/wl\": {\"bytes_per_launch\": 123.0, "
                   f"\"sources\": [\"kernel.hip\"], \"source_sha256_16\": \"{h}\"}}}}}}\n```\n")
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(rec))
    assert bench.recorded_traffic("bwd_loop", "wl") == 123.0
    assert bench.recorded_traffic("bwd_loop", "other") is None
    assert bench.recorded_traffic("dw", "wl") is None          # not a loop stage
    src.write_text("// kernel source, changed\n")
    assert bench.recorded_traffic("bwd_loop", "wl") is None    # the kernel changed since


@pytest.mark.parametrize("kernel", ["fwd_loop", "bwd_loop"])
def test_committed_record_names_existing_sources(kernel):
    """Every entry of the committed record names sources that exist."""
    import json
    text = open(bench.TRAFFIC_FILE).read()
    rec = json.loads(text.split("```json", 1)[1].split("```", 1)[0])
    ents = [v for k, v in rec["entries"].items() if k.startswith(kernel + "/")]
    assert ents
    for e in ents:
        for rel in e["sources"]:
            assert os.path.exists(os.path.join(ROOT, rel)), rel
