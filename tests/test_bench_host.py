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


def test_gateup_roofline_picks_the_bound_by_arithmetic_intensity():
    """The mixtral batch (8192 pairs, 8 touched slots) is past the ridge
    point and is reported against the bf16 MFMA peak; the decode batch (116
    pairs over 32 touched slots) streams weights and is reported against HBM,
    with the algorithmic bytes written out by hand."""
    r = bench.gateup_roofline(4096, 14336, 8192, 8, 1.5e-3)
    flop = 4.0 * 4096 * 14336 * 8192
    assert r["bound"] == "mfma" and r["unit"] == "TFLOP/s"
    assert abs(r["achieved"] - flop / 1.5e-3 / 1e12) < 1e-9
    assert abs(r["frac"] - r["achieved"] / 2500.0) < 1e-12
    d, I, P, touched = 7168, 2048, 116, 32
    r = bench.gateup_roofline(d, I, P, touched, 305e-6)
    weights = 32 * 4096 * 7168 * 2          # W1 and W3 of every touched slot
    rows = 116 * 7168 * 2 + 116 * 2048 * 2  # routed rows of x read, of h written
    assert r["bound"] == "hbm" and r["unit"] == "GB/s"
    assert abs(r["achieved"] - (weights + rows) / 305e-6 / 1e9) < 1e-6
    assert abs(r["frac"] - r["achieved"] / 8000.0) < 1e-12
