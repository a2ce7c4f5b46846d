"""Host logic of bench.py (CPU, no GPU): the one-GPU guard, the algorithmic
byte counts the roofline divides by, and the source hash that decides
whether a committed counter record still describes the kernels."""
import json
import os
import shutil
import subprocess
import sys

import numpy as np

import bench
from workloads import make_workload

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_algorithmic_bytes_of_the_single_image_workload():
    """608 fp32 tokens of 1,024 channels: rows once plus 16 B of statistics per
    token for the scoring pass; 1 B of flag per token and 4 B per kept index
    for the selection; a segment keeping every row is written by the scoring
    pass, the others by the gather."""
    w = make_workload(1)
    assert [s.n_tokens for s in w.segments] == [576, 32] and all(s.hidden == 1024 for s in w.segments)
    kept = np.array([288, 32])
    score, select, gather = bench.algorithmic_bytes(w, kept, compact=True)
    row = 1024 * 4
    assert score == 608 * row + 16 * 608 + 32 * row       # the 32 text rows kept whole
    assert select == 608 + 4 * 320
    assert gather == 288 * row
    score0, select0, gather0 = bench.algorithmic_bytes(w, kept, compact=False)
    assert (score0, select0, gather0) == (608 * row + 16 * 608, select, 0)


def test_video_tokens_count_their_temporal_outputs():
    w = make_workload(3, n_requests=1)
    n = w.n_tokens
    score, _, _ = bench.algorithmic_bytes(w, np.array([2458]), compact=False)
    assert score == w.input_bytes + 24 * n


def test_stale_counter_record_reads_as_none(tmp_path, monkeypatch):
    """A record is used only while the hash of its kernel source, the shared
    device headers and the host planner matches; any edit makes it None."""
    csrc = tmp_path / "paper_2604_02945_amd" / "csrc"
    csrc.mkdir(parents=True)
    for f in ("msao_entropy.hip",) + bench.TRAFFIC_SOURCES:
        shutil.copy(os.path.join(ROOT, "paper_2604_02945_amd", "csrc", f), csrc / f)
    (tmp_path / "profiles").mkdir()
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    rec = {"kernel_source_sha256": bench.source_hash("msao_entropy.hip"), "traffic_bytes_per_launch": 123.0}
    (tmp_path / "profiles" / "k_entropy_draft_logits_traffic.json").write_text(json.dumps(rec))
    assert bench.committed_entropy_traffic() == 123.0
    with open(csrc / "msao_host.cpp", "a") as f:
        f.write("\n// planner edited\n")
    assert bench.committed_entropy_traffic() is None
    assert bench.committed_traffic(4) is None             # no record in this tree at all
