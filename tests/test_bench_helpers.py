"""bench.py's host-side helpers (no GPU): the one-GPU refusal, the rule that
stored HBM traffic is used only when it was taken on the current kernel
sources, the affinity formatting, and the committed profile summaries'
shape."""
import glob
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stdout + r.stderr


def _profile(tmp_path, sha, hbm="123456789"):
    d = tmp_path / "profiles"
    d.mkdir(exist_ok=True)
    (d / "k_test_wl.txt").write_text(
        "# rocprofv3 summary: a comment line: with colons\n"
        f"kernel: k_test\nsource_sha: {sha}\nhbm_bytes_per_launch: {hbm}\n")


def test_stored_traffic_only_on_matching_sources(tmp_path, monkeypatch):
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    _profile(tmp_path, "abcdef0123456789")
    assert bench.stored_traffic("wl", "k_test", "abcdef0123456789") == 123456789.0
    assert bench.stored_traffic("wl", "k_test", "0000000000000000") is None  # kernel changed since
    assert bench.stored_traffic("other", "k_test", "abcdef0123456789") is None  # no summary
    _profile(tmp_path, "abcdef0123456789", hbm="n/a")
    assert bench.stored_traffic("wl", "k_test", "abcdef0123456789") is None


def test_kernel_source_sha_shape():
    sha = bench.kernel_source_sha()
    assert len(sha) == 16 and int(sha, 16) >= 0
    assert bench.kernel_source_sha() == sha


@pytest.mark.parametrize("cpus,text", [([0], "0"), ([0, 1, 2, 3], "0-3"), ([3, 1, 2, 0, 8, 9, 11], "0-3,8-9,11")])
def test_cpu_ranges(cpus, text):
    assert bench._cpu_ranges(cpus) == text


def test_committed_profiles_are_complete():
    """Every summary names its kernel, the sources it was taken on, and the
    per-launch byte figures the bench line uses; all were taken together."""
    files = sorted(glob.glob(os.path.join(ROOT, "profiles", "*.txt")))
    assert files
    shas = set()
    for f in files:
        kv = {}
        for line in open(f):
            if ":" in line and not line.lstrip().startswith("#"):
                k, v = line.split(":", 1)
                kv.setdefault(k.strip(), v.strip())
        name = os.path.basename(f)[:-4]
        assert name.startswith(kv["kernel"] + "_"), f
        assert name[len(kv["kernel"]) + 1:] in bench.WORKLOAD_LABEL, f
        assert float(kv["hbm_bytes_per_launch"]) > 0, f
        assert int(kv["algorithmic_bytes_per_launch"]) > 0, f
        shas.add(kv["source_sha"])
    assert len(shas) == 1
