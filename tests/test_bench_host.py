"""Host logic of bench.py (no GPU): the algorithmic bytes behind the reported
bandwidth, the source hash that decides whether a committed profile still
describes the library, and the one-GPU guard."""

import os
import subprocess
import sys

import pytest
import torch

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_algorithmic_bytes_by_hand():
    """Counters per tree are (rows consulted, residual passes, accepted leaf,
    tests). A consulted node costs both of its rows, a residual pass both rows
    again, an accepted leaf its target row; trees with an error status are
    left out."""
    V, w, n1 = 1000, 2, 5
    counters = torch.tensor([[3, 2, 0, 4],      # 3 rows, 2 passes
                             [1, 0, 1, 1],      # 1 row, accepted leaf
                             [7, 7, 1, 9]],     # an error tree: excluded
                            dtype=torch.int32)
    status = torch.tensor([0, 0, 2], dtype=torch.int32)
    got = bench.algorithmic_bytes(counters, V, w, n1, status)
    row = V * w
    assert got["compulsory"] == 2 * row * (3 + 1) + row * 1
    assert got["rescan"] == 2 * row * 2
    assert got["small"] == 2 * n1 * (4 + 4 + 4 + 1 + 4) + 2 * 4 * (4 + bench.TV_NUM_COUNTERS)
    assert got["total"] == got["compulsory"] + got["rescan"] + got["small"]
    # without a status every tree counts
    all_trees = bench.algorithmic_bytes(counters, V, w, n1)
    assert all_trees["rescan"] == 2 * row * (2 + 0 + 7)


def test_kernel_hash_covers_every_source_and_the_header(tmp_path, monkeypatch):
    csrc = tmp_path / "csrc"
    csrc.mkdir()
    (csrc / "a.hip").write_text("kernel a")
    (csrc / "b.h").write_text("launch constants")
    header = tmp_path / "tv.h"
    header.write_text("declarations")
    monkeypatch.setattr(bench, "CSRC", str(csrc))
    monkeypatch.setattr(bench, "HEADER", str(header))
    h0 = bench.kernel_hash()
    (csrc / "b.h").write_text("launch constants changed")
    h1 = bench.kernel_hash()
    header.write_text("declarations changed")
    h2 = bench.kernel_hash()
    (csrc / "c.cpp").write_text("a new source")
    h3 = bench.kernel_hash()
    assert len({h0, h1, h2, h3}) == 4


def test_profile_values_only_for_the_current_sources(tmp_path, monkeypatch):
    monkeypatch.setattr(bench, "kernel_hash", lambda: "0123456789abcdef")
    good = tmp_path / "good.md"
    good.write_text("    kernel_source_sha256_16: 0123456789abcdef\n"
                    "    hbm_bytes_per_launch: 1.806e+09\n")
    stale = tmp_path / "stale.md"
    stale.write_text("    kernel_source_sha256_16: fedcba9876543210\n"
                     "    hbm_bytes_per_launch: 1.806e+09\n")
    assert bench._profile_value(str(good), "hbm_bytes_per_launch") == pytest.approx(1.806e9)
    assert bench._profile_value(str(stale), "hbm_bytes_per_launch") is None
    assert bench._profile_value(str(tmp_path / "missing.md"), "hbm_bytes_per_launch") is None


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "only --gpus 1 is supported" in r.stderr
