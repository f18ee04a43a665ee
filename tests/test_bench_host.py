"""Host logic of bench.py (no GPU): the roofline's algorithmic operation and
byte counts against hand counts on a tiny problem, the keying of the measured
HBM traffic to the kernel sources, and the refusal of more than one GPU."""
import os
import subprocess
import sys

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from paper_2302_11665_amd.workload.problems import Problem  # noqa: E402


def _tiny():
    # 2 models, one placement of 3 groups at S = 2: model 0 on groups 0 and 2
    # (H = 2), model 1 on group 1 (H = 1), model 2 on no group; 3 + 2 + 1
    # requests; 2 SLO scales
    t = np.array([0.0, 0.1, 0.2, 0.3, 0.4, 0.5])
    model = np.array([0, 1, 0, 2, 1, 0], np.int32)
    d = np.array([0.2, 0.3, 0.4])
    L = np.full((3, 1, 2), 0.1)
    gcfg = np.zeros((1, 3), np.int32)
    masks = np.array([[0b101, 0b010, 0]], np.uint64)
    return Problem("tiny", t, model, d, np.zeros(3, np.int64), np.array([2], np.int32), np.ones(1, np.int32), L,
                   gcfg, masks, np.array([1.0, 5.0]), np.array([1], np.int32))


def test_algorithmic_ops_hand_count():
    pb = _tiny()
    # per request of a hosted model: (H - 1) dispatch compares, S max + S add,
    # the deadline add and the admission compare; an unhosted model costs
    # nothing; plus one SLO multiply per (placement, model); per scale
    per_scale = 3 * ((2 - 1) + 2 * 2 + 2) + 2 * ((1 - 1) + 2 * 2 + 2) + 0 + 1 * 3
    assert bench.algorithmic_ops(pb) == 2 * per_scale


def test_algorithmic_bytes_hand_count():
    pb = _tiny()
    N, J = 6, 2
    expect = (12 * N + pb.group_cfg.nbytes + pb.host_mask.nbytes + pb.stage_lat.nbytes
              + J * (8 + 8 + 16) + 8 * N * 1)
    assert bench.algorithmic_bytes(pb) == expect == 72 + 12 + 24 + 48 + 64 + 48


def test_measured_traffic_follows_the_sources(monkeypatch):
    m = dict(bench.MEASURED_TRAFFIC)
    m["sources_sha256"] = "0" * 64
    monkeypatch.setattr(bench, "sources_sha256", lambda: "0" * 64)
    got = bench.measured_traffic(m, True)
    assert got == round((m["fetch_kib"] * m["fetch_scale"] + m["write_kib"] * m["write_scale"]) * 1024.0)
    # another workload than the one measured, or other kernel sources: none
    assert bench.measured_traffic(m, False) is None
    monkeypatch.setattr(bench, "sources_sha256", lambda: "1" * 64)
    assert bench.measured_traffic(m, True) is None


def test_sources_hash_covers_every_kernel_source():
    for f in bench.KERNEL_SOURCES:
        assert os.path.exists(os.path.join(ROOT, f)), f
    assert len(bench.sources_sha256()) == 64


@pytest.mark.parametrize("argv,env", [(["--gpus", "2"], {}), ([], {"WORLD_SIZE": "2"})])
def test_more_than_one_gpu_is_refused(argv, env):
    e = dict(os.environ, **env)
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py")] + argv, capture_output=True, text=True,
                       env=e, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stdout


def test_sweep_algorithmic_bytes_hand_count():
    from types import SimpleNamespace
    # 3 segments of 4, 0 and 5 requests, 4 jobs, 2 output rows of stride 5
    sp = SimpleNamespace(t=np.zeros(9), seg_offsets=np.array([0, 4, 4, 9], np.int64),
                         job_segment=np.array([0, 1, 2, 2], np.int32))
    # every request read once (12 B), the offsets, a 16-byte job record and
    # 32 bytes of outputs per job, and the output rows
    assert bench.sweep_algorithmic_bytes(sp, 2, 5) == 12 * 9 + 4 * 8 + 16 * 4 + 32 * 4 + 8 * 2 * 5
