"""Host logic of bench.py (CPU only): the kernel-source hash that decides
whether committed counter runs still describe a kernel, the traffic lookup
built on it, and the refusal of more than one GPU."""
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def _tree(tmp_path, kernel_src, header_src):
    csrc = tmp_path / "paper_2308_15152_amd" / "csrc"
    csrc.mkdir(parents=True)
    (tmp_path / "include").mkdir()
    (csrc / "k.hip").write_text(kernel_src)
    (tmp_path / "include" / "h.hpp").write_text(header_src)
    return tmp_path


KERNEL = '#include "h.hpp"\n__global__ void k(float* p) { p[0] = 1.0f; }  // store\n'
HEADER = "inline int f() { return 3; }\n"


@pytest.fixture
def fake_tree(tmp_path, monkeypatch):
    root = _tree(tmp_path, KERNEL, HEADER)
    monkeypatch.setattr(bench, "ROOT", str(root))
    monkeypatch.setitem(bench.KERNEL_SOURCES, "k", "k.hip")
    return root


def test_hash_ignores_comments_and_layout(fake_tree):
    h0 = bench.kernel_source_hash("k")
    src = fake_tree / "paper_2308_15152_amd" / "csrc" / "k.hip"
    src.write_text('#include "h.hpp"\n/* a new comment */\n__global__ void k(float* p)\n'
                   '{\n    p[0] = 1.0f;   // other words\n}\n')
    assert bench.kernel_source_hash("k") == h0


def test_hash_changes_with_code_and_with_included_headers(fake_tree):
    h0 = bench.kernel_source_hash("k")
    src = fake_tree / "paper_2308_15152_amd" / "csrc" / "k.hip"
    src.write_text(KERNEL.replace("1.0f", "2.0f"))
    h1 = bench.kernel_source_hash("k")
    assert h1 != h0
    (fake_tree / "include" / "h.hpp").write_text(HEADER.replace("3", "4"))
    assert bench.kernel_source_hash("k") != h1


def test_traffic_lookup(fake_tree, tmp_path, monkeypatch):
    table = tmp_path / "traffic.json"
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(table))
    entry = {"kernel": "k", "source_sha256": bench.kernel_source_hash("k"),
             "fetch_kib": 100.0, "fetch_scale": 2.0, "write_kib": 50.0, "write_scale": 1.0}
    table.write_text(json.dumps({"w": entry}))
    assert bench.measured_traffic("w", "k") == (100 * 2 + 50) * 1024
    assert bench.measured_traffic("other", "k") is None
    assert bench.measured_traffic("w", "another_kernel") is None
    # counters taken on different sources are not reported
    table.write_text(json.dumps({"w": dict(entry, source_sha256="0" * 64)}))
    assert bench.measured_traffic("w", "k") is None
    table.write_text("not json")
    assert bench.measured_traffic("w", "k") is None


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=300)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_committed_traffic_describes_the_committed_kernels():
    """Every counter run in profiles/traffic.json was taken on the kernel
    sources as they stand, so the benchmark line can report its traffic; a
    kernel or header change needs its counter runs taken again."""
    with open(bench.TRAFFIC_FILE) as fh:
        table = json.load(fh)
    stale = [key for key, e in table.items()
             if e["source_sha256"] != bench.kernel_source_hash(e["kernel"])]
    assert not stale, f"counter runs older than their kernel sources: {stale}"
    for key, e in table.items():
        assert os.path.exists(os.path.join(ROOT, e["summary"])), key
