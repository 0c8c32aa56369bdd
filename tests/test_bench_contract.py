"""Host-side parts of bench.py's contract, on the CPU: the one-GPU refusal,
the comment-insensitive kernel source hash, and the reading of committed
HBM traffic (null once the kernel source differs from the profiled one)."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def _hash_of(tmp_path, monkeypatch, texts):
    paths = []
    for k, t in enumerate(texts):
        p = tmp_path / f"src{k}.h"
        p.write_text(t)
        paths.append(str(p))
    monkeypatch.setattr(bench, "KERNEL_SOURCES", paths)
    return bench.kernel_source_hash()


def test_kernel_hash_ignores_comments_and_spacing(tmp_path, monkeypatch):
    base = _hash_of(tmp_path, monkeypatch, ["int f(int x) { return x + 1; }\n", "// a\nint g;\n"])
    same = _hash_of(tmp_path, monkeypatch, ["/* doc */ int f(int x)   {\n  return x + 1;  // inc\n}\n",
                                            "int g;   /* b */\n"])
    other = _hash_of(tmp_path, monkeypatch, ["int f(int x) { return x + 2; }\n", "int g;\n"])
    assert base == same and base != other and len(base) == 16


def test_committed_traffic_follows_the_kernel_hash(tmp_path, monkeypatch):
    monkeypatch.setattr(bench, "PROFILES", str(tmp_path))
    monkeypatch.setattr(bench, "kernel_source_hash", lambda: "0123456789abcdef")
    assert bench.committed_traffic("w") is None                       # no summary
    (tmp_path / "sig_chunk_w_hbm_traffic.md").write_text(
        "traffic_bytes_per_launch: `1.25e+11`\nkernel_source_sha256_16: `0123456789abcdef`\n")
    assert bench.committed_traffic("w") == 1.25e11
    assert bench.committed_traffic("w", fused=True) is None            # other file
    (tmp_path / "sig_chunk_w_hbm_traffic.md").write_text(
        "traffic_bytes_per_launch: `1.25e+11`\nkernel_source_sha256_16: `fedcba9876543210`\n")
    assert bench.committed_traffic("w") is None                       # profiled another kernel
