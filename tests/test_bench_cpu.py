"""Host-side checks of bench.py (no GPU): the one-GPU refusal, the
algorithmic byte counts the roofline divides by, and the lookup of the
committed HBM-counter profiles."""

import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from paper_2608_00814_amd import workload as wl  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode != 0
    assert "one GPU" in (r.stdout + r.stderr)


def test_algorithmic_bytes_at_the_qwen3_8b_shape():
    cfg = wl.CONFIGS["qwen3-8b"]
    N = 64
    # K and V of 8 KV heads over the 4096 prefix rows and 64 node rows, plus
    # Q and O of 64 nodes x 32 heads, all head_dim 128 in bf16
    assert bench.attention_bytes(cfg, N) == 2 * 8 * (4096 + 64) * 128 * 2 + 2 * 64 * 32 * 128 * 2 == 18087936
    # the LM-head weight, the 64 hidden rows, and an id and a max logit per node
    assert bench.lmhead_bytes(cfg, N) == 151936 * 4096 * 2 + 64 * 4096 * 2 + 64 * 8 == 1245184512


def test_recorded_traffic_follows_the_sources(tmp_path, monkeypatch):
    """A counter profile counts only while the kernel sources it names are
    unchanged (comments aside)."""
    src = "paper_2608_00814_amd/csrc/tree_attn.hip"
    os.makedirs(tmp_path / "profiles")
    os.makedirs(tmp_path / os.path.dirname(src))
    (tmp_path / src).write_text(open(os.path.join(ROOT, src)).read())
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    rec = {"workload": "w", "ooo_tree_attn": {"bytes_per_launch": 123456, "sources": {src: bench._source_digest(src)}}}
    (tmp_path / "profiles" / "hbm_traffic_w.json").write_text(json.dumps(rec))
    assert bench.recorded_traffic("w", "ooo_tree_attn") == 123456
    assert bench.recorded_traffic("no-such-workload", "ooo_tree_attn") is None
    assert bench.recorded_traffic("w", "no-such-entry") is None
    # a kernel source that changed since the counters were taken voids them
    (tmp_path / src).write_text(open(os.path.join(ROOT, src)).read() + "\nint x;\n")
    assert bench.recorded_traffic("w", "ooo_tree_attn") is None


@pytest.mark.parametrize("path", ["paper_2608_00814_amd/csrc/tree_attn.hip"])
def test_source_digest_ignores_comments_and_layout(tmp_path, monkeypatch, path):
    text = open(os.path.join(ROOT, path)).read()
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    (tmp_path / "a.hip").write_text(text)
    (tmp_path / "b.hip").write_text("// a new comment\n" + text.replace("\n", "\n\n") + "\n/* trailing */\n")
    (tmp_path / "c.hip").write_text(text + "\nint x;\n")
    assert bench._source_digest("a.hip") == bench._source_digest("b.hip")
    assert bench._source_digest("a.hip") != bench._source_digest("c.hip")
