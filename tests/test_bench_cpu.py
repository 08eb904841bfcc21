"""The benchmark's host logic (no GPU): the stratified frame sample reproduces the
stream's mean context, and the multi-GPU request is refused with a message."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


@pytest.mark.parametrize("steps", [1, 5, 20, 37, 100, 999])
def test_stratified_frames_cover_the_stream(steps):
    t = bench.stratified(1000, steps)
    assert len(t) == steps == len(set(t)) and t == sorted(t)
    assert 0 <= t[0] and t[-1] < 1000
    # one frame from the middle of each of `steps` equal stretches
    for i, x in enumerate(t):
        assert i * 1000 // steps <= x < (i + 1) * 1000 // steps + 1
    # memory t * 10 rows: the sample's mean context is the stream's (1041 + 4995), within half a stretch
    mean_ctx = 1041 + 10 * sum(t) / steps
    assert abs(mean_ctx - 6036) <= 10 * 500 / steps + 1e-9


def test_whole_stream_when_steps_equal_its_length():
    assert bench.stratified(1000, 1000) == list(range(1000))
    from paper_2609_23286_amd import synth
    cfg = synth.CONFIGS["vitl_stack_1000"]
    assert bench.workload_key(cfg, 1000, 1000, []) == "vitl_stack_1000"
    assert bench.workload_key(cfg, 1000, 20, []) == "vitl_stack_1000__20of1000"
    assert bench.workload_key(cfg, 1000, 20, ["gamma 0.02"]) is None


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2 and "one GPU" in r.stderr
