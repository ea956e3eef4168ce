"""Host logic of bench.py (no GPU): the one-GPU guard and the traffic figures'
source check."""
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=300)
    assert r.returncode == 2
    assert "one GPU" in (r.stdout + r.stderr)


@pytest.mark.parametrize("kernel", ["mfma_psi2_grad", "mfma_psi2_fwd"])
def test_committed_traffic_matches_current_source(kernel):
    rec = json.load(open(os.path.join(ROOT, "profiles", f"traffic_{kernel}_large.json")))
    got = bench.traffic_for(kernel, "large")
    # the committed counters are reported only while the kernel source is the one
    # they were taken on
    import hashlib
    cur = hashlib.sha256(open(os.path.join(ROOT, rec["source"]), "rb").read()).hexdigest()
    if cur == rec["source_sha256"]:
        assert got == rec["bytes_per_launch"] and got > 0
    else:
        assert got is None


def test_traffic_is_null_for_a_changed_source(tmp_path, monkeypatch):
    (tmp_path / "profiles").mkdir()
    src = tmp_path / "k.hip"
    src.write_text("kernel v1\n")
    import hashlib
    rec = {"source": "k.hip", "source_sha256": hashlib.sha256(b"kernel v1\n").hexdigest(),
           "bytes_per_launch": 123.0}
    (tmp_path / "profiles" / "traffic_k_w.json").write_text(json.dumps(rec))
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    assert bench.traffic_for("k", "w") == 123.0
    src.write_text("kernel v2\n")
    assert bench.traffic_for("k", "w") is None
    assert bench.traffic_for("missing", "w") is None
