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
    assert r["host_cores"] >= r["cores"] and r["blas_threads"] >= 1 and r["cpu_model"]
    assert r["sample"].startswith(f"{wl.T} seeded tokens")


def test_more_than_one_gpu_is_refused_with_a_message():
    p = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120, cwd=ROOT)
    assert p.returncode != 0
    assert "one GPU" in (p.stdout + p.stderr)


def test_quantiles_and_compact_summary():
    assert bench._pct([3, 1, 2, 4, 5], 0.5) == 3
    assert bench._pct([1, 2, 3, 4], 0.25) == 2 and bench._pct([1, 2, 3, 4], 0.75) == 3
    wl = synth.make("dsv3_decode", device="cpu", with_weights=False)
    r = {"routed_pairs": 116, "touched_slots": 31, "pairs_per_s": 2.4e5, "step_ms_p50": 0.49,
         "ms_per_step": 0.5, "stages_ms": {"gate": 0.01}, "failover": None,
         "roofline": {"bound": "hbm", "frac": 0.76}, "step_hbm_frac": 0.72, "step_flop_frac": 0.0}
    c = bench.compact(wl, r)
    assert c["step_hbm_frac"] == 0.72 and "step_flop_frac" not in c and "failover" not in c


def test_kernel_source_hash_ignores_comments_but_not_code(tmp_path):
    a = tmp_path / "a.hip"
    a.write_text("// header\nint f(int x) {\n  return x + 1;  // add one\n}\n/* block\n comment */\n")
    h0 = bench.kernel_source_hash([str(a)])
    a.write_text("// another header\n\nint f(int x) {\n  return x + 1;\n}\n")
    assert bench.kernel_source_hash([str(a)]) == h0
    a.write_text("int f(int x) {\n  return x + 2;\n}\n")
    assert bench.kernel_source_hash([str(a)]) != h0
