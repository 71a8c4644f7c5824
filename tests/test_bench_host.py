"""Host-side parts of bench.py: the CPU baseline leg and the one-GPU limit."""
import os
import subprocess
import sys

import bench
from paper_2601_01310_amd import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_cpu_baseline_takes_the_whole_batch_when_it_is_smaller_than_the_sample():
    # A batch of 64 tokens (a decode-sized batch) with the default sample of
    # 1536 tokens: the sample is the whole batch.
    wl = synth.make("tiny", device="cpu")
    r = bench.cpu_baseline(wl)
    assert r["kind"] == "oracle" and r["unit"] == "routed pairs/s"
    assert r["value"] > 0 and r["cores"] >= 1
    assert r["sample"].startswith(f"{wl.T} seeded tokens")


def test_more_than_one_gpu_is_refused_with_a_message():
    p = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120, cwd=ROOT)
    assert p.returncode != 0
    assert "one GPU" in (p.stdout + p.stderr)
