"""Host-side pieces of the benchmark (CPU): the one-GPU contract, the
selection statistics it reports, and the rule that a counter-derived
traffic figure is only reported for the kernel source it was measured on."""
import hashlib
import itertools
import os

import numpy as np
import pytest

import bench


def test_more_than_one_gpu_exits_with_a_message(capsys):
    assert bench.main(["--gpus", "2"]) == 2
    assert "one GPU only" in capsys.readouterr().err


def test_world_size_above_one_exits(monkeypatch, capsys):
    monkeypatch.setenv("WORLD_SIZE", "4")
    assert bench.main([]) == 2
    assert "WORLD_SIZE 4" in capsys.readouterr().err


def _bits(words):
    return [64 * w + b for w, v in enumerate(words) for b in range(64) if (int(v) >> b) & 1]


@pytest.mark.parametrize("words", [1, 2, 4])
def test_popcounts_and_union_sizes_match_brute_force(words):
    rng = np.random.default_rng(words)
    steps, B = 5, 7
    raw = rng.integers(0, 2**63, size=(steps, B, words), dtype=np.int64).astype(np.uint64)
    raw |= (rng.integers(0, 2, size=raw.shape).astype(np.uint64) << np.uint64(63))   # the top bit too
    masks = raw[..., 0] if words == 1 else raw
    k = bench.popcounts(masks, words)
    U = bench.union_sizes(masks, words)
    for s, b in itertools.product(range(steps), range(B)):
        assert k[s, b] == len(_bits(raw[s, b]))
    for s in range(steps):
        assert U[s] == len(set().union(*(_bits(raw[s, b]) for b in range(B))))


def test_traffic_is_reported_only_for_the_measured_source_and_run(tmp_path, monkeypatch):
    src_dir = tmp_path / "paper_2609_33614_amd" / "csrc"
    src_dir.mkdir(parents=True)
    (tmp_path / "profiles").mkdir()
    src = src_dir / "expert.hip"
    src.write_bytes(b"kernel v1")
    sha = hashlib.sha1(b"kernel v1").hexdigest()
    for steps, warm, val in ((20, 5, 1234), (256, 16, 999)):
        (tmp_path / "profiles" / f"k_s{steps}.traffic.txt").write_text(
            f"kernel: x\nsource_sha1: {sha}\nbatch: 64\nsteps: {steps}\nwarmup: {warm}\n"
            f"traffic_bytes_per_launch: {val}\n")
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    assert bench.measured_traffic("k", 64, 20, 5) == 1234.0
    assert bench.measured_traffic("k", 64, 256, 16) == 999.0
    assert bench.measured_traffic("k", 64, 20, 16) is None       # a run the counters were not taken on
    assert bench.measured_traffic("k", 32, 20, 5) is None
    assert bench.measured_traffic("missing", 64, 20, 5) is None
    src.write_bytes(b"kernel v2")                      # the kernel changed since the counters were taken
    assert bench.measured_traffic("k", 64, 20, 5) is None


def test_routing_stats_and_trajectory():
    B, E, K = 4, 8, 2
    masks = np.array([[0b11, 0b11, 0b101, 0b111], [0b11, 0b11, 0b11, 0b11]], dtype=np.uint64)
    res = {"k": bench.popcounts(masks), "masks": masks, "words": 1, "E": E, "U": bench.union_sizes(masks),
           "step_ms": np.array([2.0, 1.0])}
    st = bench.routing_stats(res, K)
    assert st["k_histogram"] == {"2": 7, "3": 1}
    assert st["tokens_above_cap"] == 1
    assert st["expert_load_share"][:3] == [round(8 / 17, 4), round(7 / 17, 4), round(2 / 17, 4)]
    assert st["experts_touched_min_mean_max"] == [2, 2.5, 3]
    tr = bench.trajectory(res, B, first=1, settle=1)
    assert tr["experts_touched_per_step"] == [3, 2]
    assert tr["first_1_steps"]["tokens_per_s"] == round(B / 2e-3, 1)
    assert tr["steps_1_to_2"]["tokens_per_s"] == round(B / 1e-3, 1)
