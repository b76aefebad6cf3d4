"""Host logic of bench.py (no GPU): the one-GPU guard and the lookup of the
measured HBM traffic of the self-attention kernel in its counter summary."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402  (stdlib-only at import time)


@pytest.mark.parametrize("argv,env", [(["--gpus", "2"], {}), (["--gpus", "8"], {}),
                                      ([], {"WORLD_SIZE": "2"})])
def test_more_than_one_gpu_is_refused(argv, env):
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py")] + argv,
                       env={**os.environ, **env}, capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""          # no JSON line for a refused run


def _summary(tmp_path, sha, workload="wan13b_cached", n_branch="1", nbytes="7522578237"):
    p = tmp_path / "traffic.md"
    p.write_text("# traffic\n\nsome text: not a field\n\n"
                 f"- workload: `{workload}`\n- n_branch: {n_branch}\n"
                 f"- kernel_source_sha256: {sha}\n- bytes_per_launch: {nbytes}\n")
    return str(p)


def test_measured_traffic_follows_the_kernel_sources(tmp_path, monkeypatch):
    sha = bench.attn_source_hash()
    assert len(sha) == 16 and int(sha, 16) >= 0
    monkeypatch.setattr(bench, "TRAFFIC_PROFILE", _summary(tmp_path, sha))
    assert bench.measured_traffic("wan13b_cached", 1) == 7522578237.0
    # another workload or branch count: the counters do not apply
    assert bench.measured_traffic("wan5b_cached", 1) is None
    assert bench.measured_traffic("wan13b_cached", 2) is None
    # kernel sources changed since the counters were taken
    stale = "0" * 16 if sha != "0" * 16 else "1" * 16
    monkeypatch.setattr(bench, "TRAFFIC_PROFILE", _summary(tmp_path, stale))
    assert bench.measured_traffic("wan13b_cached", 1) is None
    # unreadable value, missing file
    monkeypatch.setattr(bench, "TRAFFIC_PROFILE", _summary(tmp_path, sha, nbytes="n/a"))
    assert bench.measured_traffic("wan13b_cached", 1) is None
    monkeypatch.setattr(bench, "TRAFFIC_PROFILE", str(tmp_path / "absent.md"))
    assert bench.measured_traffic("wan13b_cached", 1) is None


def test_committed_traffic_summary_is_well_formed():
    """The committed summary names the default workload and a positive byte
    count; its hash is either current (the bench reports the traffic) or
    stale (the bench reports null), never unparsable."""
    txt = open(bench.TRAFFIC_PROFILE).read()
    fields = dict(l.split(":", 1) for l in txt.splitlines() if l.startswith("- ") and ":" in l)
    assert fields["- workload"].strip().strip("`") == "wan13b_cached"
    assert fields["- n_branch"].strip() == "1"
    assert float(fields["- bytes_per_launch"]) > 0
    v = bench.measured_traffic("wan13b_cached", 1)
    current = fields["- kernel_source_sha256"].strip().strip("`") == bench.attn_source_hash()
    assert (v is not None) == current
