"""Host-side pieces of the benchmark that need no GPU: the refusal of a
multi-GPU run, and the rule that the roofline's HBM traffic is read from a
committed counter summary only while the kernel and planner sources still
hash to the value recorded with it."""

import hashlib
import json
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402


def test_more_than_one_gpu_is_refused_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, cwd=ROOT, timeout=120)
    assert r.returncode == 2
    assert "one GPU only" in r.stderr
    assert r.stdout == ""


def _fake_tree(tmp_path, m, sha, traffic=12345):
    csrc = tmp_path / "paper_2608_28003_amd" / "csrc"
    csrc.mkdir(parents=True)
    for name in ("gemm.hip", "device.h", "kernels.h", "api.hip"):
        (csrc / name).write_text("// %s\n" % name)
    (tmp_path / "profiles").mkdir()
    rec = {"kernel": "k", "m": m, "traffic_bytes": traffic, "source_sha256": sha}
    (tmp_path / "profiles" / ("gate_up_geglu_m%d_hbm_traffic.md" % m)).write_text(
        "# summary\n\n```json\n%s\n```\n" % json.dumps(rec))
    h = hashlib.sha256()
    for name in ("gemm.hip", "device.h", "kernels.h", "api.hip"):
        h.update((csrc / name).read_bytes())
    return h.hexdigest()


def test_traffic_is_read_only_for_the_sources_it_was_measured_on(tmp_path, monkeypatch):
    good = _fake_tree(tmp_path, 2048, sha="0" * 64)
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    assert bench.measured_traffic(2048) is None          # recorded on other sources
    rec_path = tmp_path / "profiles" / "gate_up_geglu_m2048_hbm_traffic.md"
    rec_path.write_text(rec_path.read_text().replace("0" * 64, good))
    assert bench.measured_traffic(2048) == 12345          # same sources: the recorded bytes
    assert bench.measured_traffic(128) is None            # no summary for this M
    (tmp_path / "paper_2608_28003_amd" / "csrc" / "gemm.hip").write_text("// changed\n")
    assert bench.measured_traffic(2048) is None          # a kernel source changed since


def test_committed_summaries_carry_a_machine_read_record():
    for m in (128, 2048):
        path = os.path.join(ROOT, "profiles", "gate_up_geglu_m%d_hbm_traffic.md" % m)
        text = open(path).read()
        start = text.index("```json\n") + len("```json\n")
        rec = json.loads(text[start:text.index("\n```", start)])
        assert rec["m"] == m and rec["traffic_bytes"] > 0 and len(rec["source_sha256"]) == 64
