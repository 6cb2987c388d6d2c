"""Host-side checks of bench.py's contract pieces that need no GPU: the
profiled-traffic lookup (reported only while the kernel's code is the
profiled one) and the refusal of more than one GPU."""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def make_tree(tmp_path, fwd_text):
    csrc = tmp_path / "paper_2609_33591_amd" / "csrc"
    csrc.mkdir(parents=True)
    for name in ("kia_device.hpp", "kia_kernels.hpp", "kia_bwd.hip", "kia_bf16.hip"):
        shutil.copy(os.path.join(ROOT, "paper_2609_33591_amd", "csrc", name), csrc / name)
    (csrc / "kia_fwd.hip").write_text(fwd_text)
    (tmp_path / "profiles").mkdir()
    return tmp_path


def test_traffic_follows_the_code_hash(tmp_path, monkeypatch):
    src = open(os.path.join(ROOT, "paper_2609_33591_amd", "csrc", "kia_fwd.hip")).read()
    root = make_tree(tmp_path, src)
    monkeypatch.setattr(bench, "ROOT", str(root))
    h = bench.source_hash("kia_fwd")
    traffic = root / "profiles" / "t.md"
    traffic.write_text('x\n```json\n{"kia_fwd": {"bytes_per_launch": 1234, '
                       f'"source_sha256_16": "{h}"}}}}\n```\n')
    monkeypatch.setattr(bench, "TRAFFIC", {False: str(traffic), True: str(traffic)})
    assert bench.profiled_traffic("kia_fwd") == 1234
    # the bf16-input kernels hash their own source file
    assert bench.source_hash("kia_fwd", True) != h
    assert bench.profiled_traffic("kia_fwd", True) is None
    assert bench.profiled_traffic("kia_bwd_main") is None     # not in the table
    # a comment or whitespace edit keeps the figure ...
    (root / "paper_2609_33591_amd" / "csrc" / "kia_fwd.hip").write_text(
        "// note\n" + src.replace("\n", "\n  "))
    assert bench.profiled_traffic("kia_fwd") == 1234
    # ... a code edit drops it
    (root / "paper_2609_33591_amd" / "csrc" / "kia_fwd.hip").write_text(src + "\nint x;\n")
    assert bench.profiled_traffic("kia_fwd") is None


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
